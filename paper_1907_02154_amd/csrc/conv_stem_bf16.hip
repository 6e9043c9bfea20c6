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

__global__ __launch_bounds__(kThreads) void stem7_bf16_kernel(StemArgs a)
{
    // one LDS block: the input patch and the filters during the MFMAs, then
    // (channel-last output) half of the output tile, pixel-major
    __shared__ __attribute__((aligned(16))) uint4 lds[kPatchUnits + 64 * kWPitch];
    static_assert(224 * kOPitch * 2 <= (kPatchUnits + 64 * kWPitch) * 16, "epilogue tile fits");
    uint4 *patch = lds;                     // [row][col][4 ch] bf16
    uint4 *wl = lds + kPatchUnits;          // [k][pair] 8 x bf16
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int h = lane >> 5, ll = lane & 31;
    const int groups_p = a.P / kRows;
    const int pg = blockIdx.x % groups_p;
    const int n = (blockIdx.x / groups_p) % a.N;
    const int kt = blockIdx.x / (groups_p * a.N);
    const int p0 = pg * kRows;
    const int k0 = kt * 64;
    const int ih0 = 2 * p0 - 3;           // input row of patch row 0

    // 1. zero the patch (padding rows/columns and channel slots >= C stay zero)
    for (int i = tid; i < kPatchUnits; i += kThreads) patch[i] = make_uint4(0, 0, 0, 0);
    // filters: 64 rows x 28 units, straight copies of the packed rows
    for (int i = tid; i < 64 * kPairs; i += kThreads) {
        const int k = i / kPairs, u = i - k * kPairs;
        uint4 v = make_uint4(0, 0, 0, 0);
        if (k0 + k < a.K) v = reinterpret_cast<const uint4 *>(a.wp)[(long)(k0 + k) * kPairs + u];
        wl[k * kWPitch + u] = v;
    }
    __syncthreads();

    // 2. scatter the input rows: a lane moves 8 pixels of one channel row
    uint16_t *pe = reinterpret_cast<uint16_t *>(patch);
    const int chunks = (a.W + 7) / 8;
    const uint16_t *xn = a.x + (long)n * a.C * a.H * a.W;
    for (int i = tid; i < kInRows * a.C * chunks; i += kThreads) {
        const int ch = i % chunks;
        const int rc = i / chunks;
        const int c = rc % a.C, pr = rc / a.C;
        const int ih = ih0 + pr;
        if ((unsigned)ih >= (unsigned)a.H) continue;
        const uint16_t *src = xn + ((long)c * a.H + ih) * a.W + 8 * ch;
        uint16_t v[8];
        if (a.vec) {
            const uint4 q = *reinterpret_cast<const uint4 *>(src);
            const uint16_t *qv = reinterpret_cast<const uint16_t *>(&q);
#pragma unroll
            for (int e = 0; e < 8; ++e) v[e] = qv[e];
        } else {
#pragma unroll
            for (int e = 0; e < 8; ++e) v[e] = 8 * ch + e < a.W ? src[e] : 0;
        }
        uint16_t *dst = pe + ((long)pr * kCols + 8 * ch + 4) * 4 + c;   // column iw + 4
#pragma unroll
        for (int e = 0; e < 8; ++e)
            if (8 * ch + e < a.W) dst[e * 4] = v[e];
    }
    __syncthreads();

    // 3. MFMA: wavefront w takes pixel blocks 2w, 2w+1 and both filter blocks
    floatx16 acc[2][2];
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int f = 0; f < 2; ++f)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[b][f][v] = 0.f;
    int pbase[2];                          // patch unit of (row 2*pr, column 2q - 4) for this lane's pixel
#pragma unroll
    for (int b = 0; b < 2; ++b) {
        const int m = 32 * (2 * wave + b) + ll;       // pixel within the 4 x 112 tile
        const int pr = m / kQ, q = m - pr * kQ;
        pbase[b] = (2 * pr * kCols + 2 * q) / 2;      // 16-byte units (columns are 8 bytes)
    }
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

    // 4. epilogue: filters are the MFMA rows and pixels its columns, so register
    // v of lane l is filter 8*(v/4) + 4*h + v%4 of the filter block and pixel
    // l%32 of the pixel block: each store instruction writes 32 consecutive
    // pixels (128 bytes) of two filter planes.
    if (a.ycl) {
        // Channel-last bf16: register group v/4 of lane l holds 4 consecutive
        // channels of pixel l%32.  The tile goes out in two halves (pixel
        // block b of every wavefront): bias, activation and the bf16 rounding
        // in registers, the half staged pixel-major in LDS ([224][64 + 4]
        // bf16: the pitch spreads a store's 32 pixels over the banks), then
        // every lane writes 16 bytes = 8 channels of one pixel, so a
        // wavefront's stores are 1 KB of contiguous y (64 channels).
        uint16_t *y = reinterpret_cast<uint16_t *>(a.y);
        uint16_t *ot = reinterpret_cast<uint16_t *>(lds);
        const int kn = min(64, a.K - k0);                  // channels of this filter tile (% 4 == 0)
        float bv[2][4][4];
#pragma unroll
        for (int f = 0; f < 2; ++f)
#pragma unroll
            for (int q4 = 0; q4 < 4; ++q4)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int k = k0 + f * 32 + 8 * q4 + 4 * h + e;
                    bv[f][q4][e] = (a.bias && k < a.K) ? a.bias[k] : 0.f;
                }
        const long pix0 = ((long)n * a.P + p0) * kQ;       // first pixel of the 4-row tile
#pragma unroll
        for (int b = 0; b < 2; ++b) {
            __syncthreads();                                // LDS free (MFMA operands, or the last half)
#pragma unroll
            for (int f = 0; f < 2; ++f)
#pragma unroll
                for (int q4 = 0; q4 < 4; ++q4) {
                    uint32_t d[2];
#pragma unroll
                    for (int e = 0; e < 2; ++e) {
                        float v0 = acc[b][f][4 * q4 + 2 * e] + bv[f][q4][2 * e];
                        float v1 = acc[b][f][4 * q4 + 2 * e + 1] + bv[f][q4][2 * e + 1];
                        if (a.relu) {
                            v0 = fmaxf(v0, 0.f);
                            v1 = fmaxf(v1, 0.f);
                        }
                        d[e] = (uint32_t)f32_to_bf16_rne(v0) | ((uint32_t)f32_to_bf16_rne(v1) << 16);
                    }
                    const int row = 32 * wave + ll;         // pixel 32*(2*wave + b) + ll of the tile
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
                *reinterpret_cast<uint4 *>(y + (pix0 + px) * a.K + k0 + 8 * o) = make_uint4(lo.x, lo.y, hi.x, hi.y);
            }
        }
        return;
    }
    const long plane = (long)a.P * kQ;
#pragma unroll
    for (int f = 0; f < 2; ++f) {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const int k = k0 + f * 32 + 8 * (v >> 2) + 4 * h + (v & 3);
            if (k >= a.K) continue;
            const float bv = a.bias ? a.bias[k] : 0.f;
            const long yo = (long)n * a.ysn + (long)k * plane + (long)p0 * kQ;
#pragma unroll
            for (int b = 0; b < 2; ++b) {
                const long o = yo + 32 * (2 * wave + b) + ll;
                float val = acc[b][f][v] + bv;
                if (a.res) val += a.res[o];
                a.y[o] = a.relu ? fmaxf(val, 0.f) : val;
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
    const long wgs = (long)(p.P / kRows) * p.N * ceil_div(p.K, 64);
    launch_kernel(stem7_bf16_kernel, dim3((unsigned)wgs), dim3(kThreads), 0, st, a);
    return hipGetLastError();
}

}  // namespace miconv
