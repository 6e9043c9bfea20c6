/*
 * mivision — the vision-specific operators of detection post-processing on
 * AMD Instinct MI355X (gfx950), part of libmiconv: the three-stage prefix sum
 * (paper Sec. 3.1.1, "Prefix sum", Fig. 3), segmented argsort (Sec. 3.1.1,
 * "Sorting", Fig. 2) and box_nms (Sec. 3.1.1, "Other vision-specific
 * operators"; its evaluation in Sec. 4.3 describes the output convention).
 *
 * Conventions (as in miconv.h)
 *  - Tensor pointers are DEVICE pointers owned by the caller; the library
 *    never frees them.  `stream` is a hipStream_t passed as void* (NULL = the
 *    default stream).  Calls validate their scalar arguments, enqueue kernels
 *    and return; they never allocate, free or synchronise, so every call can
 *    be captured into a HIP graph.  Scratch memory comes from a caller-owned
 *    workspace (`ws`, at least the bytes the matching *_workspace_bytes call
 *    reports, 256-byte aligned; it may be NULL when that is 0).
 *  - Return 0 (MICONV_OK) or a negative miconv_status (miconv.h); on a
 *    validation error nothing is enqueued.  Device-side data (segment
 *    offsets, scores, boxes) is not validated: the kernels clamp every index
 *    they derive from it, so bad data gives wrong results, never an access
 *    outside the buffers.
 *  - Results are deterministic: integer and index outputs are unique (ties
 *    are broken by position), and box_nms copies input rows bit for bit.
 */
#ifndef MIVISION_H
#define MIVISION_H

#include <stddef.h>
#include <stdint.h>

#pragma GCC visibility push(default)

#ifdef __cplusplus
extern "C" {
#endif

/* Prefix sum of `rows` independent rows of n int32 values each (x and y
 * [rows][n], row-major; y may be x).  Inclusive: y[r][i] = x[r][0] + ... +
 * x[r][i]; exclusive (exclusive != 0): y[r][0] = 0, y[r][i] = x[r][0] + ... +
 * x[r][i-1].  Sums wrap modulo 2^32 (two's complement).  Computed in the
 * three stages of Sec. 3.1.1 / Fig. 3: up-sweep (each thread scans a block
 * of consecutive values sequentially in registers), a Hillis-Steele scan of
 * the block totals, down-sweep (each block adds the scanned total of the
 * blocks before it).  Many rows, or short ones, take one work-group per row
 * (the stages inside the work-group, no synchronisation across
 * work-groups); a few long rows take the stages across work-groups, one
 * launch each, with the tile totals in the workspace.
 * Errors: MICONV_ERR_NULL (x or y NULL), MICONV_ERR_SHAPE (rows < 1,
 * n < 1), MICONV_ERR_TOO_LARGE (rows * n >= 2^31), MICONV_ERR_WORKSPACE. */
long vision_scan_workspace_bytes(int rows, long n);
int vision_scan_i32(int rows, long n, const int32_t *x, int32_t *y, int exclusive, void *ws, size_t ws_bytes,
                    void *stream);

/* Segmented argsort (Sec. 3.1.1 / Fig. 2).  keys: fp32 [n], flattened
 * segments; offsets: int32 [segments + 1] on the device, offsets[0] = 0,
 * non-decreasing, offsets[segments] = n (segment s is keys[offsets[s] ..
 * offsets[s+1])).  out: int32 [n]; out[offsets[s] + r] is the index, local
 * to segment s, of the element of rank r in segment s (descending != 0:
 * largest key first).  Equal keys keep their order (stable); -0 and +0 are
 * equal; NaN keys come last in either order.  Positions at or past
 * offsets[segments] belong to no segment and get -1.
 * The flattened array is cut into equal blocks of 2048 elements, each block
 * is sorted in LDS by (segment, key, position), then sorted runs are merged
 * pairwise, doubling the run length per pass, each work-group producing
 * 2048 outputs of a merge at the split points of its merge path; a pair
 * whose two runs meet at a segment boundary is already in order and is
 * copied.  Errors: MICONV_ERR_NULL, MICONV_ERR_SHAPE (n < 1, segments < 1),
 * MICONV_ERR_TOO_LARGE (n >= 2^31 or segments >= 2^21 - 1),
 * MICONV_ERR_WORKSPACE. */
long vision_argsort_workspace_bytes(long n, int segments);
int vision_segmented_argsort(long n, int segments, const float *keys, const int32_t *offsets, int descending,
                             int32_t *out, void *ws, size_t ws_bytes, void *stream);

/* Largest number of candidates box_nms compares per image. */
#define MIVISION_NMS_MAX_CANDIDATES 4096

/* box_nms: greedy non-maximum suppression per image of detection rows.
 * data, out: fp32 [batch][num][width] (must not overlap); a row holds a
 * score at score_index, a corner-encoded box (x1, y1, x2, y2) at
 * coord_start .. coord_start + 3 and, when id_index >= 0, a class id.
 * Candidates are the rows with score > valid_thresh, ranked by score
 * (highest first, equal scores by row order); the first topk of them take
 * part (all when topk < 0).  In rank order a candidate is kept unless a kept
 * candidate of the same class (any class when force_suppress != 0 or
 * id_index < 0) overlaps it with IoU > overlap_thresh, where IoU =
 * intersection / union of the boxes (widths and heights max(0, .), fp32,
 * each operation rounded, no fused multiply-add; 0 when the union is 0).
 * Kept rows are copied to out[b][0 ..], in rank order; every other value of
 * out is -1 (the output is first set invalid as a whole, Sec. 4.3).
 * Pipeline: a fill kernel sets out to -1; a three-stage scan of the
 * candidate flags gives each candidate its slot; the candidates' scores are
 * compacted per image and ranked by segmented argsort; a kernel grid over
 * (candidate block, candidate block, image) computes which later candidate
 * each candidate suppresses as 64-bit masks (the innermost loop on threads,
 * the loop above it on work-groups, images on the grid); one wavefront per
 * image then walks the candidates in rank order, OR-ing the mask rows of
 * the kept ones, and copies the kept rows.
 * Errors: MICONV_ERR_NULL, MICONV_ERR_SHAPE (batch, num or width < 1, an
 * index outside the row),
 * MICONV_ERR_UNSUPPORTED (more than MIVISION_NMS_MAX_CANDIDATES candidates
 * per image possible: min(topk, num), or num when topk < 0),
 * MICONV_ERR_TOO_LARGE (batch * num * width >= 2^31, batch >= 2^21 - 1),
 * MICONV_ERR_WORKSPACE. */
long vision_box_nms_workspace_bytes(int batch, int num, int width, int topk);
int vision_box_nms(int batch, int num, int width, const float *data, float *out, float overlap_thresh,
                   float valid_thresh, int topk, int id_index, int score_index, int coord_start,
                   int force_suppress, void *ws, size_t ws_bytes, void *stream);

#ifdef __cplusplus
}
#endif

#pragma GCC visibility pop

#endif /* MIVISION_H */
