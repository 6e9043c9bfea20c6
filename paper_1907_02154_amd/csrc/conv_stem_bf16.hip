// bf16 stem: 7x7 stride-2 pad-3 conv on images of at most 4 channels with
// 112-column outputs (ResNet's first layer on 224 x 224 inputs), bf16 inputs,
// fp32 accumulation and output.
//
// The general bf16 paths need the reduction to run over runs of 8 channels;
// with C = 3 every 8-element MFMA operand would be a gather of scattered
// 2-byte values.  Here the reduction is reordered to make each operand one
// aligned 16-byte LDS read:
//  * The input patch a work-group needs (13 input rows for 4 output rows) is
//    staged in LDS channel-interleaved with C padded to 4: one 8-byte entry
//    per input pixel, four zero columns on each side, zero rows outside the
//    image.
//  * The reduction index runs over (r, j, t, c): filter row r, tap pair j
//    (columns s = 2j-1 and 2j, s = -1 having a zero weight), tap t of the
//    pair, channel c.  8 consecutive indices are one pair: two adjacent input
//    pixels x 4 channels, 16 contiguous bytes at an even column, so a lane's
//    MFMA operand is one aligned ds_read_b128, and 32 lanes reading 32
//    consecutive output columns (input stride 2 = 16 bytes) cover every bank
//    once.  7 rows x 4 pairs = 28 pairs = 224 reduction slots = 14 MFMA steps.
//  * Filters are pre-packed in the same order ([K][28][8], zero-padded); the
//    work-group copies its 64 filters into LDS with a row pitch of 29 units
//    of 16 bytes, so 16 consecutive filter rows also hit distinct banks.
// A work-group computes 4 output rows (448 pixels = 14 blocks of 32) x 64
// filters with 7 wavefronts, each 2 pixel blocks x 2 filter blocks of
// v_mfma_f32_32x32x16_bf16 with filters as the A operand and pixels as B, so
// each store instruction writes runs of 32 consecutive output pixels (NCHW
// fp32), or 4 consecutive channels of each of 32 pixels (channel-last bf16).
#include "internal.h"

#include <algorithm>
#include <cstdio>

namespace miconv {
namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int kQ = 112;                 // output columns
constexpr int kRows = 4;                // output rows per work-group
constexpr int kInRows = 2 * kRows + 5;  // input rows of a work-group's patch (13)
constexpr int kCols = 2 * kQ + 8;       // patch columns: input columns -4 .. 2*kQ+3 (232)
constexpr int kPairs = 28;              // 7 filter rows x 4 tap pairs
constexpr int kWPitch = 29;             // filter row pitch in 16-byte units (28 + 1 pad)
constexpr int kWaves = 7;
constexpr int kThreads = 64 * kWaves;
constexpr int kPatchUnits = kInRows * kCols / 2;   // 16-byte units of the patch (1508)

struct StemArgs {
    const uint16_t *x;        // [N][C][H][W] bf16
    const uint16_t *wp;       // [K][28][8] bf16, packed
    const float *bias;
    const float *res;         // [N][K][P][kQ] added before the activation, or nullptr
    long ysn;                 // elements between images of y and res
    float *y;                 // [N][K][P][kQ]
    int N, C, H, W, K, P;
    int relu;
    int vec;                  // W % 8 == 0 and x 16-byte aligned: 16-byte row loads
    int ycl;                  // y bf16 channel-last [N][P][kQ][K] (no residual)
};

constexpr int kOPitch = 68;   // channel-last epilogue: bf16 row pitch of a pixel (64 + 4)
constexpr int kStageUnits = 224 * kOPitch * 2 / 16;   // half an output tile, channel-last (1904)
constexpr int kShared = kPatchUnits > kStageUnits ? kPatchUnits : kStageUnits;
constexpr int kChunks = kQ / 4;                        // 8-pixel chunks of a patch row (28)
constexpr int kTasks = kInRows * kChunks;              // 364: one per thread
constexpr int kWLoads = (64 * kPairs + kThreads - 1) / kThreads;   // filter units per thread (4)
static_assert(kTasks + kInRows * 4 <= kThreads, "one patch task per thread, spare threads for padding");

// A work-group's unit of work is a tile: 4 output rows (448 pixels) x 64
// filters of one image.  Work-groups are persistent (two per CU): each walks
// a contiguous range of tiles, keeps its 64 filters and their bias in LDS
// while the filter block stays the same, and requests the next tile's input
// rows before it runs the current tile's MFMAs and epilogue, so that their
// round trip overlaps the work instead of starting every tile.
__global__ __launch_bounds__(kThreads, 4) void stem7_bf16_kernel(StemArgs a)
{
    // filters, their bias, and one region that holds the input patch during
    // the MFMAs and (channel-last output) half of the output tile after them
    __shared__ __attribute__((aligned(16))) uint4 wl[64 * kWPitch];   // [k][pair] 8 x bf16
    __shared__ __attribute__((aligned(16))) uint4 shared[kShared];
    __shared__ float bias_l[64];
    uint4 *patch = shared;                  // [row][col][4 ch] bf16
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int h = lane >> 5, ll = lane & 31;
    const int groups_p = a.P / kRows;
    const int tiles = groups_p * a.N * ceil_div(a.K, 64);
    const int per = tiles / gridDim.x, extra = tiles % gridDim.x;
    const int t_begin = blockIdx.x * per + min((int)blockIdx.x, extra);
    const int t_end = t_begin + per + ((int)blockIdx.x < extra ? 1 : 0);

    // This thread's patch task: input row pr of the patch, 8-pixel chunk ch.
    const int pr = tid / kChunks, ch = tid - pr * kChunks;
    uint4 xv_ld[4];                         // channel c: 8 pixels
    // Request the input rows of tile t (one 16-byte load per channel row when
    // W % 8 == 0); rows outside the image and channels >= C are zeros.
    auto fetch = [&](int t) {
        const int n = (t / groups_p) % a.N;
        const int ih = 2 * (t % groups_p) * kRows - 3 + pr;
        const bool row_ok = tid < kTasks && (unsigned)ih < (unsigned)a.H;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            xv_ld[c] = make_uint4(0, 0, 0, 0);
            if (!row_ok || c >= a.C) continue;
            const uint16_t *src = a.x + (((long)n * a.C + c) * a.H + ih) * a.W + 8 * ch;
            if (a.vec) {
                if (8 * ch < a.W) xv_ld[c] = *reinterpret_cast<const uint4 *>(src);
            } else {
                uint16_t v[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) v[e] = 8 * ch + e < a.W ? src[e] : 0;
                xv_ld[c] = make_uint4(v[0] | (uint32_t)v[1] << 16, v[2] | (uint32_t)v[3] << 16,
                                      v[4] | (uint32_t)v[5] << 16, v[6] | (uint32_t)v[7] << 16);
            }
        }
    };
    // Filters and bias of filter block kt into LDS (all requests first).
    auto load_filters = [&](int kt) {
        const int k0 = kt * 64;
        uint4 wv_ld[kWLoads];
#pragma unroll
        for (int j = 0; j < kWLoads; ++j) {
            const int i = tid + j * kThreads;
            const int k = i / kPairs, u = i - k * kPairs;
            wv_ld[j] = make_uint4(0, 0, 0, 0);
            if (i < 64 * kPairs && k0 + k < a.K) wv_ld[j] = reinterpret_cast<const uint4 *>(a.wp)[(long)(k0 + k) * kPairs + u];
        }
        const float bv = tid < 64 && a.bias && k0 + tid < a.K ? a.bias[k0 + tid] : 0.f;
#pragma unroll
        for (int j = 0; j < kWLoads; ++j) {
            const int i = tid + j * kThreads;
            const int k = i / kPairs, u = i - k * kPairs;
            if (i < 64 * kPairs) wl[k * kWPitch + u] = wv_ld[j];
        }
        if (tid < 64) bias_l[tid] = bv;
    };

    int pbase[2];                           // patch unit of (row 2*pr, column 2q - 4) for this lane's pixel
#pragma unroll
    for (int b = 0; b < 2; ++b) {
        const int m = 32 * (2 * wave + b) + ll;       // pixel within the 4 x 112 tile
        const int rr = m / kQ, q = m - rr * kQ;
        pbase[b] = (2 * rr * kCols + 2 * q) / 2;      // 16-byte units (columns are 8 bytes)
    }

    int kt_loaded = -1;
    if (t_begin < t_end) fetch(t_begin);
    for (int t = t_begin; t < t_end; ++t) {
        const int pg = t % groups_p;
        const int n = (t / groups_p) % a.N;
        const int kt = t / (groups_p * a.N);
        const int p0 = pg * kRows;
        const int k0 = kt * 64;
        __syncthreads();                    // the previous tile's LDS reads are done
        if (kt != kt_loaded) {
            load_filters(kt);
            kt_loaded = kt;
        }
        // The patch, channel-interleaved: 16-byte unit e of the chunk holds
        // pixels 2e, 2e+1, 4 channels each (input column iw at patch column
        // iw + 4); spare threads zero the 4 padding columns on each side.
        if (tid < kTasks) {
            const uint32_t *q0 = reinterpret_cast<const uint32_t *>(&xv_ld[0]);
            const uint32_t *q1 = reinterpret_cast<const uint32_t *>(&xv_ld[1]);
            const uint32_t *q2 = reinterpret_cast<const uint32_t *>(&xv_ld[2]);
            const uint32_t *q3 = reinterpret_cast<const uint32_t *>(&xv_ld[3]);
            uint4 *dst = patch + pr * (kCols / 2) + 4 * ch + 2;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                // word e of a channel holds pixels 2e (low half) and 2e+1 (high half)
                const uint32_t a0 = q0[e], a1 = q1[e], a2 = q2[e], a3 = q3[e];
                dst[e] = make_uint4((a0 & 0xFFFFu) | (a1 << 16), (a2 & 0xFFFFu) | (a3 << 16),
                                    (a0 >> 16) | (a1 & 0xFFFF0000u), (a2 >> 16) | (a3 & 0xFFFF0000u));
            }
        } else if (tid < kTasks + kInRows * 4) {
            const int z = tid - kTasks;
            const int zr = z >> 2, zu = z & 3;
            patch[zr * (kCols / 2) + (zu < 2 ? zu : kCols / 2 - 4 + zu)] = make_uint4(0, 0, 0, 0);
        }
        __syncthreads();

        // MFMA: wavefront w takes pixel blocks 2w, 2w+1 and both filter blocks
        floatx16 acc[2][2];
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
            for (int f = 0; f < 2; ++f)
#pragma unroll
                for (int v = 0; v < 16; ++v) acc[b][f][v] = 0.f;
#pragma unroll
        for (int ks = 0; ks < kPairs / 2; ++ks) {
            const int pi = 2 * ks + h;                     // this half's tap pair
            const int r = pi >> 2, j = pi & 3;
            const int off = (r * kCols + 2 * j) / 2;       // units
            bf16x8 xv[2], wv[2];
#pragma unroll
            for (int b = 0; b < 2; ++b) xv[b] = *reinterpret_cast<const bf16x8 *>(&patch[pbase[b] + off]);
#pragma unroll
            for (int f = 0; f < 2; ++f)
                wv[f] = *reinterpret_cast<const bf16x8 *>(&wl[(f * 32 + ll) * kWPitch + pi]);
#pragma unroll
            for (int b = 0; b < 2; ++b)
#pragma unroll
                for (int f = 0; f < 2; ++f)
                    acc[b][f] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wv[f], xv[b], acc[b][f], 0, 0, 0);
        }
        // the next tile's input rows, in flight during this tile's epilogue
        // (requested here rather than before the MFMAs, whose operands leave
        // no registers for them)
        if (t + 1 < t_end) fetch(t + 1);

        // Epilogue: filters are the MFMA rows and pixels its columns, so
        // register v of lane l is filter 8*(v/4) + 4*h + v%4 of the filter
        // block and pixel l%32 of the pixel block.
        if (a.ycl) {
            // Channel-last bf16: register group v/4 of lane l holds 4
            // consecutive channels of pixel l%32.  The tile goes out in two
            // halves (pixel block b of every wavefront): bias, activation and
            // the bf16 rounding in registers, the half staged pixel-major in
            // LDS ([224][64 + 4] bf16: the pitch spreads a store's 32 pixels
            // over the banks), then every lane writes 16 bytes = 8 channels of
            // one pixel, so a wavefront's stores are 1 KB of contiguous y.
            uint16_t *y = reinterpret_cast<uint16_t *>(a.y);
            uint16_t *ot = reinterpret_cast<uint16_t *>(shared);
            const int kn = min(64, a.K - k0);              // channels of this filter tile (% 8 == 0)
            const long pix0 = ((long)n * a.P + p0) * kQ;   // first pixel of the 4-row tile
#pragma unroll
            for (int b = 0; b < 2; ++b) {
                __syncthreads();                            // LDS free (the patch, or the last half)
#pragma unroll
                for (int f = 0; f < 2; ++f)
#pragma unroll
                    for (int q4 = 0; q4 < 4; ++q4) {
                        const float4 bq = *reinterpret_cast<const float4 *>(&bias_l[f * 32 + 8 * q4 + 4 * h]);
                        const float bb[4] = {bq.x, bq.y, bq.z, bq.w};
                        uint32_t d[2];
#pragma unroll
                        for (int e = 0; e < 2; ++e) {
                            float v0 = acc[b][f][4 * q4 + 2 * e] + bb[2 * e];
                            float v1 = acc[b][f][4 * q4 + 2 * e + 1] + bb[2 * e + 1];
                            if (a.relu) {
                                v0 = fmaxf(v0, 0.f);
                                v1 = fmaxf(v1, 0.f);
                            }
                            d[e] = pack_bf16x2(v0, v1);
                        }
                        const int row = 32 * wave + ll;     // pixel 32*(2*wave + b) + ll of the tile
                        *reinterpret_cast<uint2 *>(ot + row * kOPitch + f * 32 + 8 * q4 + 4 * h) =
                            make_uint2(d[0], d[1]);
                    }
                __syncthreads();
                for (int u = tid; u < 224 * 8; u += kThreads) {
                    const int row = u >> 3, o = u & 7;
                    if (8 * o >= kn) continue;
                    const int px = 32 * (2 * (row >> 5) + b) + (row & 31);
                    const uint2 lo = *reinterpret_cast<const uint2 *>(ot + row * kOPitch + 8 * o);
                    const uint2 hi = *reinterpret_cast<const uint2 *>(ot + row * kOPitch + 8 * o + 4);
                    *reinterpret_cast<uint4 *>(y + (pix0 + px) * a.K + k0 + 8 * o) =
                        make_uint4(lo.x, lo.y, hi.x, hi.y);
                }
            }
            continue;
        }
        // NCHW fp32: each store instruction writes 32 consecutive pixels
        // (128 bytes) of two filter planes.  Non-temporal: at batch 64 the
        // output (205 MB) nearly fills the last-level cache, and written
        // normally its dirty lines are written back during the following
        // kernels, slowing them.
        const long plane = (long)a.P * kQ;
#pragma unroll
        for (int f = 0; f < 2; ++f) {
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int kl = f * 32 + 8 * (v >> 2) + 4 * h + (v & 3);
                const int k = k0 + kl;
                if (k >= a.K) continue;
                const float bv = bias_l[kl];
                const long yo = (long)n * a.ysn + (long)k * plane + (long)p0 * kQ;
#pragma unroll
                for (int b = 0; b < 2; ++b) {
                    const long o = yo + 32 * (2 * wave + b) + ll;
                    float val = acc[b][f][v] + bv;
                    if (a.res) val += a.res[o];
                    __builtin_nontemporal_store(a.relu ? fmaxf(val, 0.f) : val, &a.y[o]);
                }
            }
        }
    }
}

// w [K][C][7][7] -> wp [K][28][8]: slot ((r*4 + j)*2 + t)*4 + c holds
// w[k][c][r][2j - 1 + t], zero for s = -1 and for c >= C.
__global__ __launch_bounds__(256) void pack_stem_kernel(const uint16_t *__restrict__ w,
                                                        uint16_t *__restrict__ wp, int K, int C)
{
    const int total = K * kPairs * 8;
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < total; i += gridDim.x * blockDim.x) {
        const int c = i & 3, t = (i >> 2) & 1;
        const int pi = (i >> 3) % kPairs;
        const int k = i / (kPairs * 8);
        const int r = pi >> 2, s = 2 * (pi & 3) - 1 + t;
        uint16_t v = 0;
        if (s >= 0 && c < C) v = w[(((long)k * C + c) * 7 + r) * 7 + s];
        wp[i] = v;
    }
}

}  // namespace

bool stem_bf16_eligible(const ConvProblem &p, const void *y)
{
    return p.groups == 1 && p.C <= 4 && p.R == 7 && p.S == 7 && p.stride == 2 && p.pad == 3 &&
           p.Q == kQ && p.P % kRows == 0 && p.W <= 2 * kQ && (uintptr_t)y % 16 == 0;
}

size_t stem_packed_bytes(const ConvProblem &p) { return (size_t)p.K * kPairs * 8 * sizeof(uint16_t); }

hipError_t launch_pack_stem(const ConvProblem &p, const uint16_t *w, uint16_t *packed, hipStream_t st)
{
    const int total = p.K * kPairs * 8;
    launch_kernel(pack_stem_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, st, w, packed,
                  p.K, p.C);
    return hipGetLastError();
}

void describe_stem_bf16(char *buf, int len, int *launches)
{
    snprintf(buf, len, "stem7_bf16_kernel");
    *launches = 1;
}

hipError_t launch_stem_bf16(const ConvProblem &p, const uint16_t *x, const uint16_t *wpacked,
                            const float *bias, float *y, hipStream_t st)
{
    StemArgs a{};
    a.x = x;
    a.wp = wpacked;
    a.bias = bias;
    a.res = p.res;
    a.ysn = p.ysn;
    a.y = y;
    a.N = p.N;
    a.C = p.C;
    a.H = p.H;
    a.W = p.W;
    a.K = p.K;
    a.P = p.P;
    a.relu = p.relu;
    a.vec = p.W % 8 == 0 && (uintptr_t)x % 16 == 0;
    a.ycl = p.ycl;
    if (p.ycl && (p.res || p.K % 8 || (uintptr_t)y % 16)) return hipErrorInvalidValue;
    const long tiles = (long)(p.P / kRows) * p.N * ceil_div(p.K, 64);
    if (tiles >= (1L << 31)) return hipErrorInvalidValue;
    // two persistent work-groups per CU (LDS and registers allow two)
    const long wgs = std::min(tiles, 2L * cu_count());
    launch_kernel(stem7_bf16_kernel, dim3((unsigned)wgs), dim3(kThreads), 0, st, a);
    return hipGetLastError();
}

}  // namespace miconv
