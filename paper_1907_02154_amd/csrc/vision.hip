// Vision operators of detection post-processing (paper Sec. 3.1.1): the
// three-stage prefix sum (Fig. 3), segmented argsort (Fig. 2) and box_nms,
// with their C ABI (include/mivision.h).
//
// The paper's designs target integrated GPUs; what carries over to gfx950 is
// the structure: the scan's register blocking with a Hillis-Steele scan of
// block totals, the sort's equal-block local sorts followed by cooperative
// merges that only move segments spanning a merge interface, and NMS's
// mapping of the innermost loop onto threads with the output set invalid as a
// whole first.  On a 64-wide wavefront the Hillis-Steele passes are lane
// shuffles, the merge path of a work-group is found by a 64-way search (one
// dependent memory round trip per factor of 64), and NMS's suppression test
// becomes 64-bit masks, so that the one sequential walk per image is a
// broadcast and an OR per candidate.
#include "internal.h"
#include "../../include/miconv.h"
#include "../../include/mivision.h"

#include <climits>

namespace miconv {
namespace {

// ----------------------------------------------------------------- scan

constexpr int kScanThreads = 256;                     // work-groups across a row
constexpr int kScanItems = 16;                        // values per thread (register block)
constexpr int kScanTile = kScanThreads * kScanItems;  // 4096 values per tile
constexpr int kScanWide = 1024;                       // a work-group owning one of few rows

// One spare LDS word per 16: thread t's values t*16 .. t*16+15 start in
// distinct banks.
__device__ __forceinline__ int pad16(int i) { return i + (i >> 4); }

// Hillis-Steele inclusive scan of one value per thread over a work-group of
// NT threads: in pass d every thread adds the value held by the thread 2^d
// before it.  Within a wavefront the passes are lane shuffles; the NT/64
// wavefront totals are scanned the same way by the first wavefront, through
// LDS.  Returns the thread's inclusive prefix; *total gets the work-group sum.
template <int NT>
__device__ int wg_scan_incl(int v, int *wsum, int *total)
{
    constexpr int NW = NT / 64;
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const int u = __shfl_up(v, d);
        if (lane >= d) v += u;
    }
    if (lane == 63) wsum[wid] = v;
    __syncthreads();
    if (wid == 0) {
        int w = lane < NW ? wsum[lane] : 0;
#pragma unroll
        for (int d = 1; d < NW; d <<= 1) {
            const int u = __shfl_up(w, d);
            if (lane >= d) w += u;
        }
        if (lane < NW) wsum[lane] = w;
    }
    __syncthreads();
    const int r = v + (wid ? wsum[wid - 1] : 0);
    *total = wsum[NW - 1];
    __syncthreads();   // wsum is free for the next call
    return r;
}

// Sources of scanned values: an int32 array, or the candidate flag of a
// detection row (score > threshold).
// SrcI32 can also be read four values per 16-byte load where aligned.
struct SrcI32 {
    static constexpr bool kVec = true;
    const int32_t *x;
    __device__ int operator()(long i) const { return x[i]; }
    __device__ bool aligned(long i) const { return (((uintptr_t)(x + i)) & 15) == 0; }
    __device__ int4 vec(long i) const { return *reinterpret_cast<const int4 *>(x + i); }
};
struct SrcScore {
    static constexpr bool kVec = false;
    const float *data;
    int width, score_index;
    float thresh;
    __device__ int operator()(long i) const { return data[i * width + score_index] > thresh ? 1 : 0; }
    __device__ bool aligned(long) const { return false; }
    __device__ int4 vec(long) const { return int4{}; }
};

// The three stages on one tile [base, base + len) (len <= NT * kScanItems),
// carry = sum of everything before the tile.  Up-sweep: thread t scans its
// kScanItems consecutive values sequentially in registers; scan: Hillis-
// Steele over the thread totals; down-sweep: each value gets the scanned
// total of the threads before its own.  Loads and stores are striped over
// the threads (coalesced) and transposed through LDS; NTS: whole tiles are
// stored non-temporally.  Returns carry + the tile's sum.
template <int NT, class Src, bool NTS = false>
__device__ int scan_tile(const Src &src, long base, int len, int32_t *y, int carry, bool exclusive, int *tile,
                         int *wsum)
{
    const int t = threadIdx.x;
    if (Src::kVec && len == NT * kScanItems && src.aligned(base)) {
        // whole aligned tile: 16-byte loads, four values each (a group of
        // four never straddles a pad word)
#pragma unroll
        for (int j = 0; j < kScanItems / 4; ++j) {
            const int i4 = j * NT + t;
            const int4 q = src.vec(base + 4L * i4);
            const int o = pad16(4 * i4);
            tile[o] = q.x;
            tile[o + 1] = q.y;
            tile[o + 2] = q.z;
            tile[o + 3] = q.w;
        }
    } else {
#pragma unroll
        for (int j = 0; j < kScanItems; ++j) {
            const int i = j * NT + t;
            tile[pad16(i)] = i < len ? src(base + i) : 0;
        }
    }
    __syncthreads();
    int x0[kScanItems], v[kScanItems];
    int run = 0;
#pragma unroll
    for (int k = 0; k < kScanItems; ++k) {
        x0[k] = tile[pad16(t * kScanItems + k)];
        run += x0[k];
        v[k] = run;
    }
    int total;
    const int incl = wg_scan_incl<NT>(run, wsum, &total);
    const int before = incl - run + carry;
#pragma unroll
    for (int k = 0; k < kScanItems; ++k)
        tile[pad16(t * kScanItems + k)] = before + (exclusive ? v[k] - x0[k] : v[k]);
    __syncthreads();
    if (len == NT * kScanItems && (((uintptr_t)(y + base)) & 15) == 0) {
#pragma unroll
        for (int j = 0; j < kScanItems / 4; ++j) {
            const int i4 = j * NT + t;
            const int o = pad16(4 * i4);
            typedef int i32x4 __attribute__((ext_vector_type(4)));
            const i32x4 q = {tile[o], tile[o + 1], tile[o + 2], tile[o + 3]};
            if constexpr (NTS)
                __builtin_nontemporal_store(q, reinterpret_cast<i32x4 *>(y + base + 4L * i4));
            else
                *reinterpret_cast<i32x4 *>(y + base + 4L * i4) = q;
        }
    } else {
#pragma unroll
        for (int j = 0; j < kScanItems; ++j) {
            const int i = j * NT + t;
            if (i < len) y[base + i] = tile[pad16(i)];
        }
    }
    __syncthreads();   // the tile buffer is free
    return carry + total;
}

// One work-group per row, its tiles in order with a running carry: the three
// stages inside the work-group, nothing shared across work-groups.  Row r is
// elements [r*n, r*n + n).  row_totals[r] (if given) gets the row's sum.
// NT = 1024 when the rows are few (a tile of 16384 values per round trip).
template <int NT, class Src>
__global__ __launch_bounds__(NT) void scan_rows_kernel(Src src, long n, int32_t *y, int exclusive,
                                                       int32_t *row_totals)
{
    constexpr int TILE = NT * kScanItems;
    __shared__ int tile[TILE + TILE / 16];
    __shared__ int wsum[NT / 64];
    const long row = blockIdx.x;
    int carry = 0;
    for (long b = 0; b < n; b += TILE)
        carry = scan_tile<NT>(src, row * n + b, (int)(n - b < TILE ? n - b : TILE), y, carry, exclusive != 0,
                              tile, wsum);
    if (row_totals && threadIdx.x == 0) row_totals[row] = carry;
}

// The stages across work-groups (a few long rows).  Up-sweep: the sum of
// every tile (grid: tiles x rows).
template <class Src>
__global__ __launch_bounds__(kScanThreads) void scan_upsweep_kernel(Src src, long n, int32_t *tile_sums)
{
    __shared__ int wsum[kScanThreads / 64];
    const long base = (long)blockIdx.y * n + (long)blockIdx.x * kScanTile;
    const long rem = n - (long)blockIdx.x * kScanTile;
    const int len = (int)(rem < kScanTile ? rem : kScanTile);
    int s = 0;
    if (Src::kVec && len == kScanTile && src.aligned(base)) {
#pragma unroll
        for (int j = 0; j < kScanItems / 4; ++j) {
            const int4 q = src.vec(base + 4L * (j * kScanThreads + threadIdx.x));
            s += q.x + q.y + q.z + q.w;
        }
    } else {
#pragma unroll
        for (int j = 0; j < kScanItems; ++j) {
            const int i = j * kScanThreads + threadIdx.x;
            if (i < len) s += src(base + i);
        }
    }
    int total;
    wg_scan_incl<kScanThreads>(s, wsum, &total);
    if (threadIdx.x == 0) tile_sums[(long)blockIdx.y * gridDim.x + blockIdx.x] = total;
}

// Scan: the tile sums of each row become exclusive prefixes, in place (one
// 1024-thread work-group per row, the same three stages over chunks of 16384
// sums: a 2^26-value row in one pass).
__global__ __launch_bounds__(kScanWide) void scan_tile_sums_kernel(int32_t *tile_sums, int tiles)
{
    constexpr int kChunk = kScanWide * kScanItems;
    __shared__ int tile[kChunk + kChunk / 16];
    __shared__ int wsum[kScanWide / 64];
    const long row = blockIdx.x;
    int carry = 0;
    for (int b = 0; b < tiles; b += kChunk)
        carry = scan_tile<kScanWide>(SrcI32{tile_sums}, row * tiles + b, tiles - b < kChunk ? tiles - b : kChunk,
                                     tile_sums, carry, true, tile, wsum);
}

// Down-sweep: each tile scanned again with the prefix of the tiles before it.
// The tiles are taken last first: the up-sweep has just read them in order,
// so the last ones are still in the last-level cache; y is stored
// non-temporally so that it does not evict them (2^26 values: 158 -> 134 us).
template <class Src>
__global__ __launch_bounds__(kScanThreads) void scan_downsweep_kernel(Src src, long n, const int32_t *tile_prefix,
                                                                      int32_t *y, int exclusive)
{
    __shared__ int tile[kScanTile + kScanTile / 16];
    __shared__ int wsum[kScanThreads / 64];
    const long bx = gridDim.x - 1 - blockIdx.x;
    const long base = (long)blockIdx.y * n + bx * kScanTile;
    const long rem = n - bx * kScanTile;
    scan_tile<kScanThreads, Src, true>(src, base, (int)(rem < kScanTile ? rem : kScanTile), y,
                                       tile_prefix[(long)blockIdx.y * gridDim.x + bx], exclusive != 0, tile, wsum);
}

// Rows this long or more, fewer than this many of them, go across work-groups.
constexpr long kScanLongRow = 4L * kScanTile;
constexpr int kScanFewRows = 64;

bool scan_across(int rows, long n) { return rows < kScanFewRows && n > kScanLongRow; }

long scan_ws_bytes(int rows, long n)
{
    if (!scan_across(rows, n)) return 0;
    return ((long)rows * ((n + kScanTile - 1) / kScanTile) * 4 + 255) / 256 * 256;
}

template <class Src>
hipError_t launch_scan(const Src &src, int rows, long n, int32_t *y, bool exclusive, int32_t *row_totals,
                       void *ws, hipStream_t st)
{
    if (!scan_across(rows, n) || row_totals) {
        if (rows < 256 && n > kScanTile)
            launch_kernel(scan_rows_kernel<kScanWide, Src>, dim3((unsigned)rows), dim3(kScanWide), 0, st, src, n, y,
                          exclusive ? 1 : 0, row_totals);
        else
            launch_kernel(scan_rows_kernel<kScanThreads, Src>, dim3((unsigned)rows), dim3(kScanThreads), 0, st, src,
                          n, y, exclusive ? 1 : 0, row_totals);
        return hipGetLastError();
    }
    const int tiles = (int)((n + kScanTile - 1) / kScanTile);
    int32_t *sums = static_cast<int32_t *>(ws);
    launch_kernel(scan_upsweep_kernel<Src>, dim3((unsigned)tiles, (unsigned)rows), dim3(kScanThreads), 0, st, src,
                  n, sums);
    launch_kernel(scan_tile_sums_kernel, dim3((unsigned)rows), dim3(kScanWide), 0, st, sums, tiles);
    launch_kernel(scan_downsweep_kernel<Src>, dim3((unsigned)tiles, (unsigned)rows), dim3(kScanThreads), 0, st,
                  src, n, static_cast<const int32_t *>(sums), y, exclusive ? 1 : 0);
    return hipGetLastError();
}

// ----------------------------------------------------------------- argsort

constexpr int kSortThreads = 256;
constexpr int kSortItems = 8;
constexpr int kSortTile = kSortThreads * kSortItems;   // 2048: block size and merge output per work-group
constexpr uint64_t kPadKey = ~0ull;                    // sorts after every element of every segment

// Order-preserving image of an fp32 key: ascending (or, descending != 0,
// descending) float order becomes ascending unsigned order; -0 maps with +0,
// and every NaN to the largest value, so NaNs come last in either order.
__device__ __forceinline__ uint32_t key_bits(float f, int descending)
{
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) == 0) u = 0;
    if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) return 0xffffffffu;
    u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
    return descending ? ~u : u;   // never 0xffffffff for a number
}

// Offset s of the segment table, clamped to [0, limit].
__device__ __forceinline__ long seg_at(const int32_t *off, int s, long limit)
{
    const long o = off[s];
    return o < 0 ? 0 : (o > limit ? limit : o);
}

// Segment of position i: the last s < S with offsets[s] <= i (binary search;
// any offsets give some s in [0, S-1]).
__device__ int find_segment(const int32_t *off, int S, long n, long i)
{
    int lo = 0, hi = S - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (seg_at(off, mid, n) <= i) lo = mid;
        else hi = mid - 1;
    }
    return lo;
}

// Elements are ordered by (composite key, position): all distinct.
__device__ __forceinline__ bool elem_less(uint64_t ka, int va, uint64_t kb, int vb)
{
    return ka < kb || (ka == kb && va < vb);
}

// The answer for one sorted element: its position local to its segment, or
// -1 past the last segment.
__device__ __forceinline__ int32_t local_index(uint64_t k, int v, const int32_t *off, long n)
{
    if (k == kPadKey) return -1;
    const int s = (int)(k >> 32);
    return (int32_t)(v - seg_at(off, s, n));
}

// The same search by a whole wavefront for a uniform i: 64 probes per round,
// so a table of S offsets costs about log64(S) dependent round trips.
__device__ int find_segment_wave(const int32_t *off, int S, long n, long i)
{
    const int lane = threadIdx.x & 63;
    int lo = 0, hi = S - 1;   // the answer is in [lo, hi]
    while (lo < hi) {
        const int span = hi - lo;                   // probes lo + 1 .. hi
        const int step = (span + 63) / 64;
        const int m = lo + 1 + lane * step;
        const bool f = m <= hi && seg_at(off, m, n) <= i;   // true ... true false ... false
        const uint64_t bal = __ballot(f);
        if (!bal) {
            hi = lo;                                // no probe at or below i: the answer is lo
        } else {
            const int l = 63 - __clzll((long long)bal);   // last true probe
            const int ml = lo + 1 + l * step;
            lo = ml;
            const int next = ml + step;             // the first false probe (if any) bounds hi
            hi = next - 1 < hi ? next - 1 : hi;
        }
    }
    return lo;
}

__device__ __forceinline__ uint64_t shfl_xor64(uint64_t v, int d)
{
    const int lo = __shfl_xor((int)(uint32_t)v, d), hi = __shfl_xor((int)(uint32_t)(v >> 32), d);
    return ((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo;
}

// One step of the bitonic network between elements J apart (J < 8) held by
// one thread (elements 8t .. 8t+7 in x): the pair is put in ascending order
// where bit k of its index is clear, descending where it is set.
template <int J>
__device__ __forceinline__ void bitonic_regs(uint64_t (&x)[kSortItems], int t, int k)
{
#pragma unroll
    for (int r = 0; r < kSortItems; ++r) {
        if ((r & J) == 0) {
            const bool up = ((kSortItems * t + r) & k) == 0;
            const uint64_t p = x[r], q = x[r + J];
            if ((p > q) == up) {
                x[r] = q;
                x[r + J] = p;
            }
        }
    }
}

// Equal blocks sorted locally: block b of the flattened array (kSortTile
// positions) is sorted by a bitonic network over one 64-bit word per element,
// (segment: 21 bits | key bits: 32 | position in the block: 11), which orders
// by segment, key, position and is unique; positions past the last segment
// get segment 2^21 - 1 and all-ones key bits, so they sort last.  Segments
// stay in order, each segment's part of the block is sorted.
//   Thread t holds elements 8t .. 8t+7 in registers: network steps between
// elements less than 8 apart stay in registers, steps up to 511 apart are
// lane shuffles within the wavefront, and only the three steps of 512 and
// 1024 go through LDS.  The segments overlapping the block are found once
// (two wavefront searches) and their offsets staged in LDS, where each
// element looks up its own.  The result leaves as (segment << 32 | key bits,
// position) for the merge passes, or, with a single block, as the answers.
constexpr uint64_t kPackPadSeg = 0x1FFFFFull;

__global__ __launch_bounds__(kSortThreads) void segsort_block_kernel(const float *keys, const int32_t *off, int S,
                                                                     long n, int descending, uint64_t *K, int32_t *V,
                                                                     int32_t *out)
{
    __shared__ uint64_t sk[kSortTile];
    __shared__ long soff[kSortTile + 1];
    __shared__ int seg_lo, seg_cnt;
    const int t = threadIdx.x, lane = t & 63, wid = t >> 6;
    const long base = (long)blockIdx.x * kSortTile;
    const long end = seg_at(off, S, n);   // positions >= end belong to no segment
    const long last = (base + kSortTile < end ? base + kSortTile : end) - 1;
    if (wid == 0 && base <= last) {
        const int lo = find_segment_wave(off, S, n, base);
        const int hi = find_segment_wave(off, S, n, last);
        const int cnt = hi - lo + 1;
        if (lane == 0) {
            seg_lo = lo;
            seg_cnt = cnt;
        }
        if (cnt <= kSortTile)
            for (int q = lane; q < cnt; q += 64) soff[q] = seg_at(off, lo + q, n);
    }
    __syncthreads();
    uint64_t x[kSortItems];
#pragma unroll
    for (int r = 0; r < kSortItems; ++r) {
        const int e = kSortItems * t + r;
        const long g = base + e;
        x[r] = (kPackPadSeg << 43) | (0xFFFFFFFFull << 11) | (uint64_t)e;
        if (g < end) {
            int sg;
            if (seg_cnt <= kSortTile) {      // last q with soff[q] <= g
                int lo = 0, hi = seg_cnt - 1;
                while (lo < hi) {
                    const int mid = (lo + hi + 1) >> 1;
                    if (soff[mid] <= g) lo = mid;
                    else hi = mid - 1;
                }
                sg = seg_lo + lo;
            } else {
                sg = find_segment(off, S, n, g);
            }
            x[r] = ((uint64_t)sg << 43) | ((uint64_t)key_bits(keys[g], descending) << 11) | (uint64_t)e;
        }
    }
    for (int k = 2; k <= kSortTile; k <<= 1) {
        for (int j = k >> 1; j >= kSortItems; j >>= 1) {
            // partner of element e = 8t + r is e ^ j = 8(t ^ (j/8)) + r
            const bool up = ((kSortItems * t) & k) == 0;
            const bool lower = ((kSortItems * t) & j) == 0;
            uint64_t y[kSortItems];
            if (j < 64 * kSortItems) {
#pragma unroll
                for (int r = 0; r < kSortItems; ++r) y[r] = shfl_xor64(x[r], j / kSortItems);
            } else {
                __syncthreads();   // everyone is done reading the previous LDS step
#pragma unroll
                for (int r = 0; r < kSortItems; ++r) sk[kSortItems * t + r] = x[r];
                __syncthreads();
#pragma unroll
                for (int r = 0; r < kSortItems; ++r) y[r] = sk[(kSortItems * t + r) ^ j];
            }
#pragma unroll
            for (int r = 0; r < kSortItems; ++r) {
                const bool keep_min = lower == up;
                const uint64_t mn = x[r] < y[r] ? x[r] : y[r], mx = x[r] < y[r] ? y[r] : x[r];
                x[r] = keep_min ? mn : mx;
            }
        }
        // steps between a thread's own elements
        if (k > 4) bitonic_regs<4>(x, t, k);
        if (k > 2) bitonic_regs<2>(x, t, k);
        bitonic_regs<1>(x, t, k);
    }
#pragma unroll
    for (int r = 0; r < kSortItems; ++r) {
        const long g = base + kSortItems * t + r;
        if (g >= n) continue;
        const uint64_t w = x[r];
        const bool pad = (w >> 43) == kPackPadSeg;
        const uint64_t key = pad ? kPadKey : ((w >> 43) << 32) | ((w >> 11) & 0xFFFFFFFFull);
        const int32_t v = (int32_t)(base + (long)(w & 0x7FF));
        if (out) out[g] = local_index(key, v, off, n);
        else {
            K[g] = key;
            V[g] = v;
        }
    }
}

// One merge pass: runs of length L (sorted) merged pairwise into runs of 2L.
// Work-group w writes outputs [w*C, w*C + C) (C = kSortTile) of the pair
// containing them.  Where that pair's two runs meet at a segment boundary
// (the last element of A in an earlier segment than the first of B) the pair
// is already in order and the chunk is copied: only segments that span the
// interface between two runs are reordered.  Otherwise the first two
// wavefronts find where diagonals d0 and d1 of the merge path cross (how many
// of the first d outputs come from A), each by a 64-way search (64 probes
// per round), the work-group stages the A and B elements between the two
// crossings in LDS, every thread finds its own crossing there by bisection
// and merges kSortItems outputs sequentially.  The last pass writes the
// answers (out) instead of keys.
__global__ __launch_bounds__(kSortThreads) void segsort_merge_kernel(const uint64_t *Ki, const int32_t *Vi,
                                                                     uint64_t *Ko, int32_t *Vo, long n, long L,
                                                                     const int32_t *off, int32_t *out)
{
    constexpr int C = kSortTile;
    __shared__ uint64_t sk[C];
    __shared__ int32_t sv[C];
    __shared__ long split[2];
    const int t = threadIdx.x, lane = t & 63, wid = t >> 6;
    const long o0 = (long)blockIdx.x * C;
    const long p0 = o0 / (2 * L) * (2 * L);
    const long na = n - p0 < L ? n - p0 : L;
    const long nbr = n - p0 - L;
    const long nb = nbr <= 0 ? 0 : (nbr < L ? nbr : L);
    const long d0 = o0 - p0;
    const long d1 = d0 + C < na + nb ? d0 + C : na + nb;
    const int cnt = (int)(d1 - d0);
    const uint64_t *KA = Ki + p0, *KB = Ki + p0 + L;
    const int32_t *VA = Vi + p0, *VB = Vi + p0 + L;

    // already in order: no B, or A's last element precedes B's first (in
    // particular when A ends in an earlier segment than B starts)
    const bool concat = nb == 0 || elem_less(KA[na - 1], VA[na - 1], KB[0], VB[0]);
    if (concat) {
        for (int i = t; i < cnt; i += kSortThreads) {
            const long g = o0 + i;
            const uint64_t k = Ki[g];
            const int32_t v = Vi[g];
            if (out) out[g] = local_index(k, v, off, n);
            else {
                Ko[g] = k;
                Vo[g] = v;
            }
        }
        return;
    }

    if (wid < 2) {
        const long d = wid ? d1 : d0;
        long lo = d - nb > 0 ? d - nb : 0, hi = d < na ? d : na;
        // f(m) = "A[m] is not among the first d outputs" = B[d-1-m] < A[m]:
        // false below the crossing, true from it on
        while (hi > lo) {
            const long span = hi - lo;
            const long step = (span + 63) / 64;
            const long m = lo + (long)lane * step;
            bool f = false;
            if (m < hi) f = elem_less(KB[d - 1 - m], VB[d - 1 - m], KA[m], VA[m]);
            const uint64_t bal = __ballot(f);
            if (bal) {
                const int l = __ffsll((unsigned long long)bal) - 1;
                const long ml = lo + (long)l * step;
                lo = l ? lo + (long)(l - 1) * step + 1 : lo;
                hi = ml;
            } else {
                const long last = (span - 1) / step < 63 ? (span - 1) / step : 63;
                lo = lo + last * step + 1;
            }
        }
        if (lane == 0) split[wid] = lo;
    }
    __syncthreads();
    const long a0 = split[0], a1 = split[1] > split[0] ? split[1] : split[0];
    const int ca = (int)(a1 - a0 < cnt ? a1 - a0 : cnt);   // crossings are monotone: 0 <= ca <= cnt
    const long b0 = d0 - a0;
    for (int i = t; i < cnt; i += kSortThreads) {
        if (i < ca) {
            sk[i] = KA[a0 + i];
            sv[i] = VA[a0 + i];
        } else {
            sk[i] = KB[b0 + (i - ca)];
            sv[i] = VB[b0 + (i - ca)];
        }
    }
    __syncthreads();
    const int cb = cnt - ca;
    const int dt = t * kSortItems < cnt ? t * kSortItems : cnt;
    int lo = dt - cb > 0 ? dt - cb : 0, hi = dt < ca ? dt : ca;
    while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (elem_less(sk[ca + dt - 1 - mid], sv[ca + dt - 1 - mid], sk[mid], sv[mid])) hi = mid;
        else lo = mid + 1;
    }
    int ia = lo, ib = dt - lo;
    uint64_t rk[kSortItems];
    int32_t rv[kSortItems];
#pragma unroll
    for (int k = 0; k < kSortItems; ++k) {
        rk[k] = kPadKey;
        rv[k] = INT_MAX;
        if (dt + k >= cnt) continue;
        const bool take_a = ib >= cb || (ia < ca && elem_less(sk[ia], sv[ia], sk[ca + ib], sv[ca + ib]));
        const int src = take_a ? ia++ : ca + ib++;
        rk[k] = sk[src];
        rv[k] = sv[src];
    }
    __syncthreads();   // every thread has read its inputs
#pragma unroll
    for (int k = 0; k < kSortItems; ++k)
        if (dt + k < cnt) {
            sk[dt + k] = rk[k];
            sv[dt + k] = rv[k];
        }
    __syncthreads();
    for (int i = t; i < cnt; i += kSortThreads) {
        const long g = o0 + i;
        if (out) out[g] = local_index(sk[i], sv[i], off, n);
        else {
            Ko[g] = sk[i];
            Vo[g] = sv[i];
        }
    }
}

long align256(long b) { return (b + 255) / 256 * 256; }

long argsort_ws_bytes(long n) { return n <= kSortTile ? 0 : 2 * align256(n * 8) + 2 * align256(n * 4); }

// The whole sort: local block sorts, then merge passes L = 2048, 4096, ...
// ping-ponging between two key/position buffers; the last pass (or the block
// sort, for one block) writes the answers.
hipError_t launch_segsort(const float *keys, const int32_t *off, int S, long n, int descending, int32_t *out,
                          void *ws, hipStream_t st)
{
    const unsigned blocks = (unsigned)((n + kSortTile - 1) / kSortTile);
    if (n <= kSortTile) {
        launch_kernel(segsort_block_kernel, dim3(blocks), dim3(kSortThreads), 0, st, keys, off, S, n, descending,
                      (uint64_t *)nullptr, (int32_t *)nullptr, out);
        return hipGetLastError();
    }
    char *p = static_cast<char *>(ws);
    uint64_t *K[2] = {reinterpret_cast<uint64_t *>(p), reinterpret_cast<uint64_t *>(p + align256(n * 8))};
    p += 2 * align256(n * 8);
    int32_t *V[2] = {reinterpret_cast<int32_t *>(p), reinterpret_cast<int32_t *>(p + align256(n * 4))};
    launch_kernel(segsort_block_kernel, dim3(blocks), dim3(kSortThreads), 0, st, keys, off, S, n, descending, K[0],
                  V[0], (int32_t *)nullptr);
    int cur = 0;
    for (long L = kSortTile; L < n; L *= 2) {
        const bool last = 2 * L >= n;
        launch_kernel(segsort_merge_kernel, dim3(blocks), dim3(kSortThreads), 0, st,
                      static_cast<const uint64_t *>(K[cur]), static_cast<const int32_t *>(V[cur]), K[cur ^ 1],
                      V[cur ^ 1], n, L, off, last ? out : (int32_t *)nullptr);
        cur ^= 1;
    }
    return hipGetLastError();
}

// ----------------------------------------------------------------- box_nms

constexpr int kNmsMax = MIVISION_NMS_MAX_CANDIDATES;

struct NmsArgs {
    const float *data;
    float *out;
    int B, N, width;
    int cand_max;      // candidates compared per image at most: min(topk, N), or N
    int capw;          // 64-bit mask words per candidate row: ceil(cand_max / 64)
    int mrows;         // mask rows per image: 64 * capw
    float overlap, valid;
    int id_index, score_index, coord_start, force;
    const int32_t *pos;       // [B][N] exclusive scan of the candidate flags
    const int32_t *seg_off;   // [B + 1] first compacted slot of each image; seg_off[B] = all candidates
    float *ckey;              // [B*N] compacted scores
    int32_t *corig;           // [B*N] compacted row index within the image
    int32_t *rank;            // [B*N] segmented argsort of ckey: rank r of image b -> local slot
    float4 *cbox;             // [B][mrows] box of the candidate of rank r
    float *ccls;              // [B][mrows] its class
    int32_t *crow;            // [B][mrows] its input row
    uint64_t *mask;           // [B][mrows][capw]
};

// Every value of out is set invalid first (Sec. 4.3): no per-row decision.
__global__ __launch_bounds__(256) void nms_fill_kernel(float *out, long count)
{
    const long i0 = ((long)blockIdx.x * 256 + threadIdx.x) * 4;
    if (((uintptr_t)out & 15) == 0 && i0 + 3 < count) {
        *reinterpret_cast<float4 *>(out + i0) = make_float4(-1.f, -1.f, -1.f, -1.f);
        return;
    }
    for (long i = i0; i < i0 + 4 && i < count; ++i) out[i] = -1.f;
}

// Candidate rows move to their compacted slots, image after image.
__global__ __launch_bounds__(256) void nms_compact_kernel(NmsArgs a)
{
    const long g = (long)blockIdx.x * 256 + threadIdx.x;
    if (g >= (long)a.B * a.N) return;
    const int b = (int)(g / a.N), i = (int)(g - (long)b * a.N);
    const float s = a.data[g * a.width + a.score_index];
    if (!(s > a.valid)) return;
    const long total = (long)a.B * a.N;
    long slot = (long)a.seg_off[b] + a.pos[g];
    if (slot < 0 || slot >= total) return;
    a.ckey[slot] = s;
    a.corig[slot] = i;
}

// Candidates of image b: count, and the input row of rank r.
__device__ __forceinline__ int nms_count(const NmsArgs &a, int b)
{
    const long total = (long)a.B * a.N;
    long s0 = a.seg_off[b], s1 = a.seg_off[b + 1];
    s0 = s0 < 0 ? 0 : (s0 > total ? total : s0);
    s1 = s1 < s0 ? s0 : (s1 > total ? total : s1);
    long c = s1 - s0;
    c = c < a.N ? c : a.N;   // an image has at most N candidates
    return (int)(c < a.cand_max ? c : a.cand_max);
}

__device__ __forceinline__ int nms_row(const NmsArgs &a, int b, int r)
{
    const long total = (long)a.B * a.N;
    long s0 = a.seg_off[b];
    s0 = s0 < 0 ? 0 : (s0 > total ? total : s0);
    long li = a.rank[s0 + r];                     // r < count: s0 + r < total
    li = li < 0 ? 0 : li;
    long slot = s0 + li;
    slot = slot < total ? slot : total - 1;
    const int i = a.corig[slot];
    return i < 0 ? 0 : (i >= a.N ? a.N - 1 : i);
}

// IoU of two corner-encoded boxes, each operation rounded to fp32 in the
// order of the definition.  Contraction into fused multiply-adds is switched
// off here: the compiler would otherwise fold the area products into the
// union's sums, whose single rounding moves the IoU by an ulp and flips
// comparisons at the threshold.
__device__ __forceinline__ float box_iou(float4 p, float4 q)
{
#pragma clang fp contract(off)
    const float iw = fmaxf(0.f, fminf(p.z, q.z) - fmaxf(p.x, q.x));
    const float ih = fmaxf(0.f, fminf(p.w, q.w) - fmaxf(p.y, q.y));
    const float inter = iw * ih;
    const float ap = fmaxf(0.f, p.z - p.x) * fmaxf(0.f, p.w - p.y);
    const float aq = fmaxf(0.f, q.z - q.x) * fmaxf(0.f, q.w - q.y);
    const float uni = (ap + aq) - inter;
    return uni <= 0.f ? 0.f : inter / uni;
}

__device__ __forceinline__ float4 load_box(const NmsArgs &a, int b, int i, float *cls)
{
    const float *row = a.data + ((long)b * a.N + i) * a.width;
    *cls = a.id_index >= 0 ? row[a.id_index] : 0.f;
    const float *c = row + a.coord_start;
    return make_float4(c[0], c[1], c[2], c[3]);
}

// The compared candidates in rank order: box, class and input row of rank r
// of image b (r < the image's candidate count), gathered once so that the
// mask and walk kernels read them with one request each.
__global__ __launch_bounds__(256) void nms_gather_kernel(NmsArgs a)
{
    const int b = blockIdx.y;
    const int r = blockIdx.x * 256 + threadIdx.x;
    if (r >= nms_count(a, b)) return;
    const int i = nms_row(a, b, r);
    float c;
    const long k = (long)b * a.mrows + r;
    a.cbox[k] = load_box(a, b, i, &c);
    a.ccls[k] = c;
    a.crow[k] = i;
}

// Suppression masks: work-group (column block cb, row block rb, image b),
// four wavefronts.  Lane t of wavefront q takes candidate i = 64*rb + t (the
// loop above the innermost one, on work-groups and lanes) and tests it
// against the 16 candidates j = 64*cb + 16*q .. + 15 staged in LDS (the
// innermost loop): bit j - 64*cb of mask[b][i][cb] is set when j comes later
// and i, once kept, suppresses it.  Each wavefront writes its 16 bits of the
// word.  Blocks below the diagonal are never read and not computed.
__global__ __launch_bounds__(256) void nms_mask_kernel(NmsArgs a)
{
    __shared__ float4 cbox[64];
    __shared__ float ccls[64];
    const int cb = blockIdx.x, rb = blockIdx.y, b = blockIdx.z;
    if (cb < rb) return;
    const int count = nms_count(a, b);
    if (rb * 64 >= count) return;
    const int t = threadIdx.x & 63, q = threadIdx.x >> 6;
    const long base = (long)b * a.mrows;
    if (threadIdx.x < 64) {
        const int j = cb * 64 + t;
        if (j < count) {
            cbox[t] = a.cbox[base + j];
            ccls[t] = a.ccls[base + j];
        }
    }
    __syncthreads();
    const int i = rb * 64 + t;
    if (i >= count) return;
    const float4 bi = a.cbox[base + i];
    const float ci = a.ccls[base + i];
    const bool any_class = a.force || a.id_index < 0;
    uint32_t bits = 0;
    const int j0 = cb * 64 + 16 * q;
    const int jn = count - j0 < 16 ? count - j0 : 16;
    for (int jj = 0; jj < jn; ++jj) {
        const int jg = j0 + jj;
        if (jg <= i) continue;
        if (!any_class && !(ccls[16 * q + jj] == ci)) continue;
        if (box_iou(bi, cbox[16 * q + jj]) > a.overlap) bits |= 1u << jj;
    }
    // bits 16q .. 16q+15 of the 64-bit word (little-endian halves of halves)
    reinterpret_cast<uint16_t *>(a.mask)[((base + i) * a.capw + cb) * 4 + q] = (uint16_t)bits;
}

// The greedy walk, one work-group per image.  The mask rows of the image's
// candidates are staged in LDS by all 256 threads at once (as many rows as
// fit; all requests in flight together), then the first wavefront walks:
// lane w holds word w of the removed set, candidate i (rank order) is kept
// unless its bit is set (the word is read from its lane with readlane, i
// being uniform), and a kept candidate ORs its mask row (words from its own
// on) into the set.  The kept ranks are listed in LDS, and afterwards all
// threads copy the kept rows, one value each, to the first output rows.
// The 64-bit value v of lane w (uniform w), as a scalar.
__device__ __forceinline__ uint64_t lane_word(uint64_t v, int w)
{
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, w);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), w);
    return ((uint64_t)hi << 32) | lo;
}

constexpr int kSweepThreads = 256;
constexpr int kSweepWords = 6144;   // 48 KB of mask rows per staging round

__global__ __launch_bounds__(kSweepThreads) void nms_sweep_kernel(NmsArgs a)
{
    __shared__ uint64_t rows[kSweepWords];
    __shared__ int kept_rank[kNmsMax];
    __shared__ int kept_n;
    const int b = blockIdx.x, t = threadIdx.x, lane = t & 63;
    const int count = nms_count(a, b);
    const long base = (long)b * a.mrows;
    const int per = kSweepWords / a.capw / 64 * 64;   // rows per staging round: whole words, >= 64
    uint64_t removed = 0;
    int kept = 0;
    for (int r0 = 0; r0 < count; r0 += per) {
        const int nr = count - r0 < per ? count - r0 : per;
        const int words = nr * a.capw;
        __syncthreads();
        for (int e0 = 0; e0 < words; e0 += kSweepThreads * 8) {
            uint64_t v[8];
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                const int e = e0 + k * kSweepThreads + t;
                const int rr = e / a.capw, w = e - rr * a.capw;
                // words left of the row's own block are never written; read as 0
                v[k] = e < words && w >= (r0 + rr) / 64 ? a.mask[(base + r0 + rr) * a.capw + w] : 0;
            }
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                const int e = e0 + k * kSweepThreads + t;
                if (e < words) rows[e] = v[k];
            }
        }
        __syncthreads();
        if (t < 64) {
            // word by word: the next candidate not yet removed is the lowest
            // clear bit above the last one taken, so removed candidates cost
            // nothing and the walk takes one step per kept candidate
            for (int w = r0 >> 6; w * 64 < r0 + nr; ++w) {
                const int valid = r0 + nr - w * 64 < 64 ? r0 + nr - w * 64 : 64;
                const uint64_t live = valid == 64 ? ~0ull : (1ull << valid) - 1;
                uint64_t cur = lane_word(removed, w);
                uint64_t avail = ~cur & live;
                while (avail) {
                    const int bit = __builtin_ctzll(avail);
                    const int i = w * 64 + bit;
                    if (lane == 0) kept_rank[kept] = i;
                    ++kept;
                    if (lane < a.capw) removed |= rows[(i - r0) * a.capw + lane];
                    cur = lane_word(removed, w);
                    avail = ~cur & live & ~((2ull << bit) - 1);   // bits above `bit` (none when bit = 63)
                }
            }
        }
    }
    if (t == 0) kept_n = kept;
    __syncthreads();
    const int nk = kept_n;
    for (int e = t; e < nk * a.width; e += kSweepThreads) {
        const int k = e / a.width, c = e - k * a.width;
        const float *src = a.data + ((long)b * a.N + a.crow[base + kept_rank[k]]) * a.width;
        a.out[((long)b * a.N + k) * a.width + c] = src[c];
    }
}

struct NmsLayout {
    long pos, seg_off, ckey, corig, rank, sort, cbox, ccls, crow, mask, total;
};

NmsLayout nms_layout(int B, int N, int cap)
{
    const long n = (long)B * N;
    const int capw = (cap + 63) / 64;
    NmsLayout l{};
    long o = 0;
    l.pos = o;
    o += align256(n * 4);
    l.seg_off = o;
    o += align256((long)(B + 1) * 4);
    l.ckey = o;
    o += align256(n * 4);
    l.corig = o;
    o += align256(n * 4);
    l.rank = o;
    o += align256(n * 4);
    l.sort = o;
    o += align256(argsort_ws_bytes(n));
    const long mrows = (long)B * capw * 64;
    l.cbox = o;
    o += align256(mrows * 16);
    l.ccls = o;
    o += align256(mrows * 4);
    l.crow = o;
    o += align256(mrows * 4);
    l.mask = o;
    o += align256(mrows * capw * 8);
    l.total = o;
    return l;
}

int nms_cap(int N, int topk) { return topk < 0 ? N : (topk < N ? topk : N); }

bool ws_ok(void *ws, size_t bytes, long need)
{
    if (need == 0) return true;
    return ws && ((uintptr_t)ws & 255) == 0 && (long)bytes >= need;
}

}  // namespace
}  // namespace miconv

using namespace miconv;

extern "C" {

long vision_scan_workspace_bytes(int rows, long n)
{
    if (rows < 1 || n < 1) return MICONV_ERR_SHAPE;
    if ((long)rows * n >= (1L << 31)) return MICONV_ERR_TOO_LARGE;
    return scan_ws_bytes(rows, n);
}

int vision_scan_i32(int rows, long n, const int32_t *x, int32_t *y, int exclusive, void *ws, size_t ws_bytes,
                    void *stream)
{
    if (!x || !y) return MICONV_ERR_NULL;
    const long need = vision_scan_workspace_bytes(rows, n);
    if (need < 0) return (int)need;
    if (!ws_ok(ws, ws_bytes, need)) return MICONV_ERR_WORKSPACE;
    const hipError_t e = launch_scan(SrcI32{x}, rows, n, y, exclusive != 0, (int32_t *)nullptr, ws,
                                     static_cast<hipStream_t>(stream));
    return e == hipSuccess ? MICONV_OK : set_hip_error(e);
}

long vision_argsort_workspace_bytes(long n, int segments)
{
    if (n < 1 || segments < 1) return MICONV_ERR_SHAPE;
    if (n >= (1L << 31) || segments >= (1 << 21) - 1) return MICONV_ERR_TOO_LARGE;
    return argsort_ws_bytes(n);
}

int vision_segmented_argsort(long n, int segments, const float *keys, const int32_t *offsets, int descending,
                             int32_t *out, void *ws, size_t ws_bytes, void *stream)
{
    if (!keys || !offsets || !out) return MICONV_ERR_NULL;
    const long need = vision_argsort_workspace_bytes(n, segments);
    if (need < 0) return (int)need;
    if (!ws_ok(ws, ws_bytes, need)) return MICONV_ERR_WORKSPACE;
    const hipError_t e = launch_segsort(keys, offsets, segments, n, descending != 0 ? 1 : 0, out, ws,
                                        static_cast<hipStream_t>(stream));
    return e == hipSuccess ? MICONV_OK : set_hip_error(e);
}

long vision_box_nms_workspace_bytes(int batch, int num, int width, int topk)
{
    if (batch < 1 || num < 1 || width < 1) return MICONV_ERR_SHAPE;
    if ((long)batch * num * width >= (1L << 31) || batch >= (1 << 21) - 1) return MICONV_ERR_TOO_LARGE;
    const int cap = nms_cap(num, topk);
    if (cap > kNmsMax) return MICONV_ERR_UNSUPPORTED;
    return nms_layout(batch, num, cap).total;
}

int vision_box_nms(int batch, int num, int width, const float *data, float *out, float overlap_thresh,
                   float valid_thresh, int topk, int id_index, int score_index, int coord_start,
                   int force_suppress, void *ws, size_t ws_bytes, void *stream)
{
    if (!data || !out) return MICONV_ERR_NULL;
    const long need = vision_box_nms_workspace_bytes(batch, num, width, topk);
    if (need < 0) return (int)need;
    if (score_index < 0 || score_index >= width || coord_start < 0 || coord_start + 4 > width ||
        id_index >= width)
        return MICONV_ERR_SHAPE;
    if (((uintptr_t)data & 3) || ((uintptr_t)out & 3)) return MICONV_ERR_ALIGN;
    if (!ws_ok(ws, ws_bytes, need)) return MICONV_ERR_WORKSPACE;
    const hipStream_t st = static_cast<hipStream_t>(stream);
    const int cap = nms_cap(num, topk);
    const NmsLayout l = nms_layout(batch, num, cap);
    char *w = static_cast<char *>(ws);
    NmsArgs a{};
    a.data = data;
    a.out = out;
    a.B = batch;
    a.N = num;
    a.width = width;
    a.cand_max = cap;
    a.capw = (cap + 63) / 64;
    a.mrows = a.capw * 64;
    a.overlap = overlap_thresh;
    a.valid = valid_thresh;
    a.id_index = id_index < 0 ? -1 : id_index;
    a.score_index = score_index;
    a.coord_start = coord_start;
    a.force = force_suppress != 0;
    a.pos = reinterpret_cast<int32_t *>(w + l.pos);
    a.seg_off = reinterpret_cast<int32_t *>(w + l.seg_off);
    a.ckey = reinterpret_cast<float *>(w + l.ckey);
    a.corig = reinterpret_cast<int32_t *>(w + l.corig);
    a.rank = reinterpret_cast<int32_t *>(w + l.rank);
    a.cbox = reinterpret_cast<float4 *>(w + l.cbox);
    a.ccls = reinterpret_cast<float *>(w + l.ccls);
    a.crow = reinterpret_cast<int32_t *>(w + l.crow);
    a.mask = reinterpret_cast<uint64_t *>(w + l.mask);
    const long n = (long)batch * num;
    const long vals = n * width;
    hipError_t e;
    launch_kernel(nms_fill_kernel, dim3((unsigned)((vals + 1023) / 1024)), dim3(256), 0, st, out, vals);
    // slots of the candidates within each image, and the candidate count per image
    int32_t *pos = reinterpret_cast<int32_t *>(w + l.pos);
    int32_t *seg = reinterpret_cast<int32_t *>(w + l.seg_off);
    if ((e = launch_scan(SrcScore{data, width, score_index, valid_thresh}, batch, (long)num, pos, true, seg + 1,
                         nullptr, st)) != hipSuccess)
        return set_hip_error(e);
    // first slot of each image: exclusive scan of the counts; seg[B] = all
    if ((e = launch_scan(SrcI32{seg + 1}, 1, (long)batch, seg, true, seg + batch, nullptr, st)) != hipSuccess)
        return set_hip_error(e);
    launch_kernel(nms_compact_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, a);
    if ((e = launch_segsort(a.ckey, seg, batch, n, 1, a.rank, w + l.sort, st)) != hipSuccess)
        return set_hip_error(e);
    if (a.capw > 0) {   // topk == 0: no candidate, the output stays invalid
        launch_kernel(nms_gather_kernel, dim3((unsigned)((a.mrows + 255) / 256), (unsigned)batch), dim3(256), 0, st,
                      a);
        launch_kernel(nms_mask_kernel, dim3((unsigned)a.capw, (unsigned)a.capw, (unsigned)batch), dim3(256), 0, st,
                      a);
        launch_kernel(nms_sweep_kernel, dim3((unsigned)batch), dim3(kSweepThreads), 0, st, a);
    }
    e = hipGetLastError();
    return e == hipSuccess ? MICONV_OK : set_hip_error(e);
}

}  // extern "C"
