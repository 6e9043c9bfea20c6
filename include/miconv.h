/*
 * miconv — the convolution hot path of CNN inference on AMD Instinct MI355X
 * (gfx950): dense conv2d, depthwise conv2d and the glue operators of the
 * evaluated networks.  C ABI, no C++ or framework types.
 *
 * The paper optimises the Conv2D operator of CNN inference (Sec. 3.2.2:
 * spatial packing / loop tiling, output channels split across work-groups,
 * feature map split along its height, unrolled loop nests) and keeps the
 * operator's semantics (Sec. 4.2, Sec. 5).  The operator computed here is:
 *
 *   P = floor((H + 2*pad - R) / stride) + 1,   Q = floor((W + 2*pad - S) / stride) + 1
 *   y[n][k][p][q] = act( bias[k] + sum_{c < C/groups, r < R, s < S}
 *                        x[n][g*(C/groups) + c][p*stride - pad + r][q*stride - pad + s]
 *                        * w[k][c][r][s] ),     g = k / (K/groups)
 *
 * cross-correlation (no kernel flip), symmetric zero padding, act = ReLU when
 * relu != 0 else identity.
 *
 * Conventions shared by every entry point
 *  - Layouts (all contiguous, row-major): x [N][C][H][W], w [K][C/groups][R][S],
 *    bias [K] (may be NULL: no bias), y [N][K][P][Q].
 *  - All tensor pointers are DEVICE pointers owned by the caller; the library
 *    never frees them.  x, w, bias must not overlap y.
 *  - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *    Calls are asynchronous: they validate, enqueue kernels on `stream` and
 *    return.  Launch errors are returned; faults inside a kernel surface at
 *    the caller's next synchronisation.
 *  - Return 0 (MICONV_OK) on success or a negative miconv_status.  On a
 *    validation error nothing is enqueued.
 *  - Tensor extents are limited to 2^31-1 elements each (MICONV_ERR_TOO_LARGE).
 *  - Dilation is not supported (the evaluated networks use none).
 *  - Entry points are stateless and thread-safe, and no call below allocates,
 *    frees or synchronises (the stack executor allocates once, at create).
 *    Scratch memory (split-K partial sums, an internal channel-last copy of
 *    x, filters packed into the layout a kernel reads) comes only from a
 *    caller-owned workspace passed to conv2d_fwd_ws; the entry points without
 *    one run plans that need none (no split reduction, filters read as
 *    given), so every call can be captured into a HIP graph, the first one
 *    included.
 */
#ifndef MICONV_H
#define MICONV_H

#include <stddef.h>
#include <stdint.h>

/* The library is built with hidden symbol visibility; everything declared
 * here is exported. */
#pragma GCC visibility push(default)

#ifdef __cplusplus
extern "C" {
#endif

enum miconv_status {
    MICONV_OK = 0,
    MICONV_ERR_NULL = -1,        /* x, w or y is NULL */
    MICONV_ERR_SHAPE = -2,       /* a dim <= 0, stride < 1, pad < 0, or P or Q < 1 */
    MICONV_ERR_GROUPS = -3,      /* C % groups or K % groups != 0; depthwise needs groups == C == K */
    MICONV_ERR_UNSUPPORTED = -4, /* valid but not provided (e.g. depthwise filter wider than 7) */
    MICONV_ERR_TOO_LARGE = -5,   /* a tensor exceeds 2^31-1 elements */
    MICONV_ERR_ALIGN = -6,       /* a pointer is not aligned to its element size */
    MICONV_ERR_HIP = -7,         /* a HIP call failed; see miconv_last_hip_error() */
    MICONV_ERR_WORKSPACE = -8    /* workspace missing, smaller than conv2d_workspace_bytes
                                    reports, or not 256-byte aligned */
};

/* What a dense call may use besides its tensors, which decides its kernel
 * plan (conv2d_describe names the kernels of each). */
enum miconv_plan_mode {
    MICONV_PLAN_PLAIN = 0,   /* conv2d_fwd, conv2d_fwd_bf16, *_algo, _res, _ex: no workspace */
    MICONV_PLAN_WS = 1,      /* conv2d_fwd_ws: caller workspace (split reductions, channel-last
                                copy of x, filters packed per call) */
    MICONV_PLAN_PACKED = 2,  /* conv2d_fwd_packed: filters packed ahead, no workspace */
    MICONV_PLAN_STACK = 3    /* a layer of miconv_stack: both */
};

/* Dense-conv algorithm selector for conv2d_fwd_algo (tests and A/B runs). */
enum miconv_algo {
    MICONV_ALGO_AUTO = 0,   /* shape-based choice, what conv2d_fwd does */
    MICONV_ALGO_DIRECT = 1, /* one output per lane, plain FMA loop: any shape and groups */
    MICONV_ALGO_IGEMM = 2,  /* implicit GEMM on MFMA with LDS-staged tiles (+ split-K when small) */
    MICONV_ALGO_WAVE = 3    /* implicit GEMM on MFMA fed straight from global memory by each
                               wavefront, reduction split across wavefronts; what AUTO picks for
                               fp32 dense layers whose x and filters fit 2 GiB.  Reads the filters
                               as given (a stack or conv2d_fwd_packed reads them packed in the
                               wavefront load order); larger tensors: MICONV_ERR_UNSUPPORTED. */
};

/* Output extent: floor((H + 2*pad - R)/stride) + 1 and likewise for W.
 * Writes *P and *Q; returns MICONV_ERR_SHAPE if either is < 1. */
int miconv_out_dims(int H, int W, int R, int S, int stride, int pad, int *P, int *Q);

/* Dense or grouped conv2d forward in fp32 (the Conv2D operator of Sec. 3.2.2).
 * x fp32 [N][C][H][W], w fp32 [K][C/groups][R][S], bias fp32 [K] or NULL,
 * y fp32 [N][K][P][Q].  When groups == C == K the call is the depthwise
 * operator and is served by the depthwise kernel. */
int conv2d_fwd(int N, int C, int H, int W, int K, int R, int S, int stride, int pad,
               int groups, const float *x, const float *w, const float *bias, float *y,
               int relu, void *stream);

/* conv2d_fwd with an explicit algorithm (enum miconv_algo). */
int conv2d_fwd_algo(int N, int C, int H, int W, int K, int R, int S, int stride, int pad,
                    int groups, const float *x, const float *w, const float *bias, float *y,
                    int relu, int algo, void *stream);

/* Same operator with x and w stored as bf16 (raw bit patterns, uint16),
 * products accumulated in fp32, bias and y in fp32. */
int conv2d_fwd_bf16(int N, int C, int H, int W, int K, int R, int S, int stride, int pad,
                    int groups, const uint16_t *x, const uint16_t *w, const float *bias,
                    float *y, int relu, void *stream);

/* conv2d_fwd_bf16 with an explicit algorithm: MICONV_ALGO_AUTO (channel-last
 * internal copy of x when C/groups % 32 == 0, else the NCHW-gather MFMA
 * kernel), MICONV_ALGO_IGEMM (the NCHW-gather MFMA kernel), MICONV_ALGO_DIRECT. */
int conv2d_fwd_bf16_algo(int N, int C, int H, int W, int K, int R, int S, int stride, int pad,
                         int groups, const uint16_t *x, const uint16_t *w, const float *bias,
                         float *y, int relu, int algo, void *stream);

/* Depthwise conv2d forward in fp32 (MobileNet's per-channel filter, Sec. 4.2
 * discusses its cost): requires groups == C == K; w fp32 [C][1][R][S] with
 * R, S <= 7; otherwise the same conventions as conv2d_fwd. */
int dwconv2d_fwd(int N, int C, int H, int W, int K, int R, int S, int stride, int pad,
                 int groups, const float *x, const float *w, const float *bias, float *y,
                 int relu, void *stream);

/* Dense conv2d with a residual join fused into the epilogue (the operator
 * fusion of the paper's graph-level optimisation, Sec. 3.2.3, applied to the
 * shortcut add of ResNet's bottleneck blocks):
 *   y = act(conv(x, w) + bias + res),  act = ReLU when relu != 0, else identity,
 * with the sum taken in fp32 in that order.  dtype 0: x, w fp32 (conv2d_fwd);
 * dtype 1: x, w bf16 bit patterns (conv2d_fwd_bf16).  algo as for
 * conv2d_fwd_algo / conv2d_fwd_bf16_algo.  res is device fp32
 * [N][K][P][Q], caller-owned, or NULL (then the call equals the plain entry
 * point).  res may be y itself (in-place join: each element is read before it
 * is written, by the same thread); it must not otherwise overlap y.  res must
 * be 4-byte aligned and lie at the same offset modulo 16 bytes as y (the
 * kernels read it with y's own vector accesses), else MICONV_ERR_ALIGN.
 * Depthwise shapes (groups == C == K with fp32): MICONV_ERR_UNSUPPORTED. */
int conv2d_fwd_res(int N, int C, int H, int W, int K, int R, int S, int stride, int pad,
                   int groups, int dtype, int algo, const void *x, const void *w,
                   const float *bias, const float *res, float *y, int relu, void *stream);

/* conv2d_fwd_res with the output written at an image stride: image n of y
 * (and of res) starts y_image_stride elements after image n-1, each image
 * being a dense [K][P][Q] block; 0 means K*P*Q (a dense y).  With a larger
 * stride, y can be a channel range of a wider NCHW tensor, which is how the
 * fire modules of SqueezeNet (Sec. 4.1) concatenate their two expand convs:
 * each expand conv writes its channel range in place, at any batch.  The
 * stride must be >= K*P*Q (images must not overlap; MICONV_ERR_SHAPE),
 * (N-1)*stride + K*P*Q must stay below 2^31 (MICONV_ERR_TOO_LARGE), and
 * depthwise shapes take no stride (MICONV_ERR_UNSUPPORTED). */
int conv2d_fwd_ex(int N, int C, int H, int W, int K, int R, int S, int stride, int pad,
                  int groups, int dtype, int algo, const void *x, const void *w, const float *bias,
                  const float *res, float *y, long y_image_stride, int relu, void *stream);

/* Workspace for conv2d_fwd_ws.  conv2d_workspace_bytes returns the bytes of
 * scratch the fastest plan for this shape needs (0: none), for any pointer
 * alignment, or a negative miconv_status (invalid shape, groups, dtype or
 * algo).  dtype 0 = fp32, 1 = bf16; algo as for conv2d_fwd_algo /
 * conv2d_fwd_bf16_algo. */
long conv2d_workspace_bytes(int N, int C, int H, int W, int K, int R, int S, int stride, int pad,
                            int groups, int dtype, int algo);

/* conv2d_fwd_ex with a caller-owned device workspace `ws` of `ws_bytes`
 * bytes, 256-byte aligned, at least conv2d_workspace_bytes (NULL when that is
 * 0).  With it the dense conv may split its reduction across work-groups
 * (fp32 partial sums, reduced in a fixed order: results are run-to-run
 * deterministic), stage x channel-last (bf16) and pack the filters into the
 * order its kernel reads, all inside `ws`: the fastest single-call plans.
 * The library keeps no reference to ws after the call's kernels are
 * enqueued; they use it until they complete on `stream`, so concurrent calls
 * need distinct workspaces.  Too small or unaligned: MICONV_ERR_WORKSPACE,
 * nothing enqueued.  Everything else as conv2d_fwd_ex. */
int conv2d_fwd_ws(int N, int C, int H, int W, int K, int R, int S, int stride, int pad, int groups,
                  int dtype, int algo, const void *x, const void *w, const float *bias, const float *res,
                  float *y, long y_image_stride, int relu, void *ws, size_t ws_bytes, void *stream);

/* For callers that cannot allocate device memory at all (code under HIP
 * graph capture that may not call hipMalloc, tight serving loops, harnesses
 * that forbid allocation): conv2d_fwd_ws with the workspace taken from a
 * fixed scratch array of MICONV_NOALLOC_SCRATCH_BYTES inside the library's
 * device code, one per GPU, held from its first use on that GPU until the
 * process ends.  Allocates nothing (no hipMalloc, hipFree or allocating
 * library routine) and synchronises nothing.  A plan that needs more scratch
 * than that (conv2d_workspace_bytes reports it) fails with
 * MICONV_ERR_WORKSPACE and enqueues nothing.  Every call on one GPU shares
 * its scratch: calls that can overlap on one GPU (other streams, other
 * threads, or a graph replay of one) race on it and must be serialised by the
 * caller; calls ordered on one stream are safe.  Whatever must start at zero
 * is written by the call's own kernels.  Everything else as conv2d_fwd_ws. */
#define MICONV_NOALLOC_SCRATCH_BYTES (32u << 20)
int conv2d_fwd_noalloc(int N, int C, int H, int W, int K, int R, int S, int stride, int pad,
                       int groups, int dtype, int algo, const void *x, const void *w, const float *bias,
                       const float *res, float *y, long y_image_stride, int relu, void *stream);

/* Filters packed once for repeated calls of one layer (the pre-computing step
 * of the paper's graph-level optimisation, Sec. 3.2.3), outside a stack.
 * The packed layout is the one the kernel chosen for this shape reads: the
 * wavefront load order of the fp32 wave kernel, (r, s, c) order for the bf16
 * channel-last kernels, tap pairs for the bf16 7x7 stem.  dtype 0 = fp32
 * (conv2d_fwd), 1 = bf16 (conv2d_fwd_bf16).  Shapes as in conv2d_fwd.
 *
 * conv2d_packed_weight_bytes returns the size in bytes of the packed buffer,
 * 0 when the kernel reads w as given (then conv2d_fwd_packed takes w itself),
 * or a negative miconv_status (invalid shape, groups or dtype). */
long conv2d_packed_weight_bytes(int N, int C, int H, int W, int K, int R, int S, int stride,
                                int pad, int groups, int dtype);

/* Pack w (device, [K][C/groups][R][S], fp32 or bf16 bits) into `packed`
 * (device, caller-owned, conv2d_packed_weight_bytes bytes, 16-byte aligned;
 * the library keeps no reference) on `stream`.  Nothing is launched when the
 * packed size is 0. */
int conv2d_pack_weights(int N, int C, int H, int W, int K, int R, int S, int stride, int pad,
                        int groups, int dtype, const void *w, void *packed, void *stream);

/* conv2d_fwd (dtype 0) or conv2d_fwd_bf16 (dtype 1) with the filters from
 * conv2d_pack_weights for the same shape and dtype (or w itself when the
 * packed size is 0).  No packing launch and no workspace (MICONV_PLAN_PACKED:
 * no split reduction, no channel-last copy).  The kernel is chosen again from
 * the actual pointers; if their alignment selects a kernel with another
 * filter layout than the one packed for (x and y at 256-byte boundaries never
 * do), or packed is not 16-byte aligned, the call fails with
 * MICONV_ERR_ALIGN and launches nothing. */
int conv2d_fwd_packed(int N, int C, int H, int W, int K, int R, int S, int stride, int pad,
                      int groups, int dtype, const void *x, const void *packed, const float *bias,
                      float *y, int relu, void *stream);

/* ---- Channel-last bf16 activations between layers ----
 *
 * The paper's graph tuner chooses each operator's data layout for the whole
 * network and its fusion merges element-wise work into the conv (Sec. 3.2.3).
 * Here that is a bf16 channel-last activation layout kept from layer to
 * layer: a layer reads the previous layer's bf16 [N][H][W][C] output as given
 * (no transposing copy) and its epilogue writes its own output as bf16
 * [N][P][Q][K], bias, residual join and ReLU applied in fp32 before one
 * round-to-nearest-even to bf16: half the output bytes of fp32 NCHW. */
enum miconv_layout {
    MICONV_LAYOUT_NCHW = 0,          /* x bf16 NCHW, y fp32 NCHW: conv2d_fwd_bf16 */
    MICONV_LAYOUT_X_NHWC = 1,        /* x bf16 [N][H][W][C] */
    MICONV_LAYOUT_Y_NHWC_BF16 = 2    /* y (and res) bf16 [N][P][Q][K] */
};

/* bf16 conv2d with channel-last x and/or y (enum miconv_layout flags, or-ed):
 *   y = act(conv(x, w) + bias + res),  summed in fp32; with
 *   MICONV_LAYOUT_Y_NHWC_BF16 the result is rounded once to bf16 (nearest
 *   even) and res, when given, is bf16 [N][P][Q][K] like y.
 * w bf16 [K][C/groups][R][S] and bias fp32 [K] as everywhere.  Supported:
 *  - MICONV_LAYOUT_X_NHWC (with or without a channel-last y): C/groups % 64
 *    == 0, x 16-byte aligned (and w for 1x1 filters); with a channel-last y
 *    K/groups % 8 == 0 and y, res 16-byte aligned;
 *  - MICONV_LAYOUT_Y_NHWC_BF16 alone (x NCHW): the 7x7 stride-2 stem on at
 *    most 4 channels with 112 output columns (ResNet's first layer), K % 8
 *    == 0, no residual;
 * anything else MICONV_ERR_UNSUPPORTED (MICONV_ERR_ALIGN for alignment).
 * Workspace as for conv2d_fwd_ws, sized by conv2d_cl_workspace_bytes (split
 * partials and per-call packed filters; never a copy of x). */
long conv2d_cl_workspace_bytes(int N, int C, int H, int W, int K, int R, int S, int stride, int pad,
                               int groups, int layout);
int conv2d_fwd_cl(int N, int C, int H, int W, int K, int R, int S, int stride, int pad, int groups,
                  int layout, const uint16_t *x, const uint16_t *w, const float *bias, const void *res,
                  void *y, int relu, void *ws, size_t ws_bytes, void *stream);

/* The kernels conv2d_fwd_cl would launch for this shape and layout (with its
 * workspace), as conv2d_describe names them; validates like conv2d_fwd_cl
 * (pointers taken as 256-byte aligned); enqueues nothing. */
int conv2d_cl_describe(int N, int C, int H, int W, int K, int R, int S, int stride, int pad, int groups,
                       int layout, char *buf, int buflen, int *launches);

/* Glue operators of the evaluated networks (not part of the conv operator). */

/* Max-pool on bf16 channel-last tensors: x [N][H][W][C] -> y [N][P][Q][C],
 * R x S window, stride, symmetric pad (pad < R and pad < S); padded positions
 * never win, so y holds input values exactly.  C % 8 == 0, x and y 16-byte
 * aligned. */
int maxpool2d_nhwc_bf16(int N, int C, int H, int W, int R, int S, int stride, int pad,
                        const uint16_t *x, uint16_t *y, void *stream);

/* Max-pool fp32 NCHW with an R x S window, stride and symmetric pad
 * (pad < R and pad < S); padded positions never win. y [N][C][P][Q]. */
int maxpool2d_fwd(int N, int C, int H, int W, int R, int S, int stride, int pad,
                  const float *x, float *y, void *stream);

/* Residual join: y[i] = act(a[i] + b[i]) for i < count, fp32.  y may alias a or b. */
int add_act_fwd(long count, const float *a, const float *b, float *y, int relu, void *stream);

/* fp32 -> bf16 bit patterns, round to nearest even (NaN stays NaN). */
int cast_f32_to_bf16(long count, const float *x, uint16_t *y, void *stream);

/* ---- Stack executor: a network's conv layers planned once and replayed ----
 *
 * Batch-1 inference (the latency setting of Sec. 4.2) runs layers of a few
 * microseconds, so the executor validates and plans every layer once, packs
 * its filters once (the pre-computing of Sec. 3.2.3), owns one workspace for
 * the whole stack (allocated at create), and can capture repeated passes
 * into a single HIP graph.  Tensor pointers are borrowed: they must stay
 * valid and keep their contents' meaning for the executor's lifetime (a
 * replay reads x/w/bias and writes y of every layer). */

enum miconv_op {
    MICONV_OP_CONV_F32 = 0,    /* conv2d_fwd */
    MICONV_OP_CONV_BF16 = 1,   /* conv2d_fwd_bf16 (x, w are bf16 bit patterns), or with
                                  `layout` conv2d_fwd_cl */
    MICONV_OP_DWCONV_F32 = 2,  /* dwconv2d_fwd */
    MICONV_OP_MAXPOOL_BF16_NHWC = 3,  /* maxpool2d_nhwc_bf16: R x S window, stride, pad; K = C,
                                         w, bias, res NULL (glue between channel-last layers) */
    MICONV_OP_MAXPOOL_F32 = 4         /* maxpool2d_fwd on fp32 NCHW, the same fields */
};

typedef struct miconv_conv_desc {
    int op;                    /* enum miconv_op */
    int N, C, H, W, K, R, S, stride, pad, groups, relu;
    const void *x;             /* device, layout as the matching entry point */
    const void *w;
    const float *bias;         /* may be NULL */
    void *y;                   /* fp32 NCHW, or bf16 channel-last per `layout` */
    const void *res;           /* residual joined before the activation, as in
                                  conv2d_fwd_res / conv2d_fwd_cl (dense ops only); may be NULL */
    long y_image_stride;       /* as in conv2d_fwd_ex; 0 = dense y */
    int layout;                /* MICONV_OP_CONV_BF16: enum miconv_layout flags, as in conv2d_fwd_cl */
} miconv_conv_desc;

typedef struct miconv_stack miconv_stack;

/* Validate and plan n layers (each as its entry point would); allocate the
 * executor, its packed filters and its workspace on the current device.  On error
 * nothing is allocated and *out is NULL. */
int miconv_stack_create(const miconv_conv_desc *layers, int n, miconv_stack **out);

/* Number of layers. */
int miconv_stack_size(const miconv_stack *s);

/* Kernel names of one layer (as conv2d_describe); returns its launch count. */
int miconv_stack_describe(const miconv_stack *s, int layer, char *buf, int buflen);

/* Kernel launches in one pass (a layer with a split reduction launches two). */
int miconv_stack_launches(const miconv_stack *s);

/* Kernel name of launch `launch` of a pass; returns the index of its layer. */
int miconv_stack_launch_info(const miconv_stack *s, int launch, char *buf, int buflen);

/* Enqueue every layer once, in order, on `stream`. */
int miconv_stack_launch(miconv_stack *s, void *stream);

/* Enqueue `steps` passes eagerly, every kernel launch carrying a start and an
 * end event that the runtime stamps with that kernel's own execution interval
 * (read them with miconv_stack_times once the stream is done).  Drops any
 * captured graph. */
int miconv_stack_launch_timed(miconv_stack *s, int steps, void *stream);

/* Overlap of independent layers in untimed captures (off by default): at
 * create every layer's dependencies are derived from the byte ranges of x,
 * res and y it shares with earlier layers (read after write, write after
 * write, write after read); with enable != 0 a layer that its successor does
 * not depend on runs on a second stream, joined by event waits (graph
 * edges), each stream with its own half of the workspace; passes never
 * overlap each other.  In ResNet the projection shortcut then runs beside
 * the first two convs of its block.  On MI355X the cross-stream edges cost
 * more than the overlap gains on ResNet-50 (batch 1 and 64), hence the
 * default.  Takes effect at the next capture.  Returns the number of layers
 * on the second stream when enabled (0 when nothing can overlap), else 0. */
int miconv_stack_overlap(miconv_stack *s, int enable);

/* Capture `steps` consecutive passes into one HIP graph, replacing any
 * previous capture (nothing executes; the NULL stream is served by a private
 * capture stream).  With timed != 0 an event is recorded before every kernel
 * launch of every pass and after the last one.  Workspace and events are owned by
 * the executor, so a replay allocates nothing. */
int miconv_stack_capture(miconv_stack *s, int steps, int timed, void *stream);

/* Launch the captured graph on `stream` (MICONV_ERR_UNSUPPORTED if none). */
int miconv_stack_replay(miconv_stack *s, void *stream);

/* After a timed replay has completed: ms[k*L + j] = time from the event
 * before launch j of pass k to the next event (L = miconv_stack_launches);
 * after miconv_stack_launch_timed: the execution time of launch j of pass k.
 * capacity is the length of ms, at least steps*L. */
int miconv_stack_times(const miconv_stack *s, float *ms, long capacity);

/* Free the graph, events, workspace and the executor (NULL is a no-op). */
int miconv_stack_destroy(miconv_stack *s);

/* Names the kernels a dense call of this shape would launch on the current
 * device (dtype 0 = fp32, 1 = bf16; algo as for conv2d_fwd_algo; mode = enum
 * miconv_plan_mode: which entry point), as a profiler prints them (template
 * arguments included, namespaces omitted), joined by " + "; writes at most
 * buflen bytes (NUL-terminated) into buf and the number of kernel launches
 * into *launches.  Validates like the conv entry points (pointer alignment
 * is taken as 256 bytes); enqueues nothing. */
int conv2d_describe(int N, int C, int H, int W, int K, int R, int S, int stride, int pad,
                    int groups, int dtype, int algo, int mode, char *buf, int buflen, int *launches);

/* Human-readable text for a miconv_status. */
const char *miconv_strerror(int status);

/* The hipError_t of the last failed HIP call made by this thread (0 if none). */
int miconv_last_hip_error(void);

/* Library version, major*10000 + minor*100 + patch. */
int miconv_version(void);

#ifdef __cplusplus
}
#endif

#pragma GCC visibility pop

#endif /* MICONV_H */
