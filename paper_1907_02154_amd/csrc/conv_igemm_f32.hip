// Dense conv2d in fp32 as an implicit GEMM on the gfx950 matrix cores.
//
// GEMM view (per group g): D[k][m] = sum_kr Wg[k][kr] * X[kr][m] with
//   k  = output channel          (GEMM rows,    "output channels divided", Sec. 3.2.2)
//   m  = (n, p, q) output pixel  (GEMM columns, the feature map split across work-groups)
//   kr = (c, r, s) filter tap    (reduction, Kred = C/groups * R * S)
// X is never materialised: each work-group gathers its [KRC x BPX] slice of
// the im2col matrix straight from NCHW x into LDS (the loop tiling / spatial
// packing of Sec. 3.2.2), zero-filling taps that fall in the padding.
//
// Data path per work-group (BKC channels x BPX pixels, 4 wavefronts):
//   HBM/L2 --(coalesced loads along q / along kr)--> VGPR --> LDS (double buffer)
//   LDS --(one fp32 per lane per operand)--> v_mfma_f32_32x32x2_f32 --> AGPR acc
// The next chunk's global loads are issued before the MFMAs on the current
// chunk, so memory latency hides behind matrix work; one barrier per chunk.
//
// MFMA 32x32x2 f32 operand layout (lane l of 64):
//   A[i][kk] with i = l % 32, kk = l / 32   -> output channel i, tap kk
//   B[kk][j] with j = l % 32, kk = l / 32   -> tap kk, pixel j
//   D reg v: i = 8*(v/4) + 4*(l/32) + v%4,  j = l % 32
// Pixels sit on j, so every accumulator store writes 32 consecutive pixels of
// one channel: 128-byte contiguous NCHW segments.
//
// Small layers (batch 1, late stages) do not fill 256 CUs with output tiles;
// there the reduction is split over grid.z, every split writes fp32 partials
// to a workspace, and a second kernel sums them in split order, so results
// are run-to-run deterministic.  (An in-kernel "last work-group reduces"
// scheme needs device-scope fences, which on a multi-XCD part write back and
// invalidate whole L2s and cost far more than a second launch.)
#include "internal.h"

#include <cstdio>

namespace miconv {
namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));

template <int R_, int S_, int BKC, int BPX, int WK, int WP, int KRC>
__global__ __launch_bounds__(64 * WK * WP) void igemm_f32_kernel(ConvArgs a)
{
    constexpr int NT = 64 * WK * WP;
    constexpr int WTK = BKC / WK, WTP = BPX / WP;
    constexpr int BI = WTK / 32, BJ = WTP / 32;
    static_assert(WTK % 32 == 0 && WTP % 32 == 0, "wave tile must be a multiple of 32x32");
    static_assert(NT % BPX == 0 && KRC % (NT / BPX) == 0, "B loader shape");
    static_assert(NT % KRC == 0 && BKC % (NT / KRC) == 0, "A loader shape");
    constexpr int APAD = 4, BPAD = 4;
    constexpr int B_RPP = NT / BPX;          // B rows (taps) per loader pass
    constexpr int B_LOADS = KRC / B_RPP;
    constexpr int A_KPP = NT / KRC;          // A rows (channels) per loader pass
    constexpr int A_LOADS = BKC / A_KPP;

    __shared__ float As[2][KRC][BKC + APAD];
    __shared__ float Bs[2][KRC][BPX + BPAD];

    const float *__restrict__ x = static_cast<const float *>(a.x);
    const float *__restrict__ w = static_cast<const float *>(a.w);
    const int R = R_ ? R_ : a.R;
    const int S = S_ ? S_ : a.S;
    const int RS = R * S;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wid = tid >> 6;
    const int wk = wid / WP, wp = wid % WP;
    const int g = blockIdx.z % a.groups;
    const int split = blockIdx.z / a.groups;
    const int m0 = blockIdx.x * BPX;
    const int k0 = blockIdx.y * BKC;
    const int kr_begin = split * a.kr_per_split;
    const int kr_end = min(a.Kred, kr_begin + a.kr_per_split);

    // B (im2col) loader: this lane always gathers pixel column bcol.
    const int bcol = tid % BPX;
    const int brow0 = tid / BPX;
    const int mB = m0 + bcol;
    const bool mvalid = mB < a.M;
    int ih0 = 0, iw0 = 0, nB = 0;
    if (mvalid) {
        nB = mB / a.PQ;
        const int pq = mB - nB * a.PQ;
        const int p = pq / a.Q;
        const int q = pq - p * a.Q;
        ih0 = p * a.stride - a.pad;
        iw0 = q * a.stride - a.pad;
    }
    const float *xg = x + ((long)nB * a.C + (long)g * a.Cg) * a.HW;

    // A (weights) loader: consecutive lanes walk the reduction axis of one row.
    const int acol = tid % KRC;
    const int arow0 = tid / KRC;
    const float *wg = w + (long)g * a.Kg * a.Kred;

    float breg[B_LOADS], areg[A_LOADS];
    auto gload = [&](int kr0) {
#pragma unroll
        for (int i = 0; i < B_LOADS; ++i) {
            const int kr = kr0 + brow0 + i * B_RPP;
            const int c = kr / RS;
            const int rs = kr - c * RS;
            const int r = rs / S;
            const int s = rs - r * S;
            const int ih = ih0 + r, iw = iw0 + s;
            const bool ok = mvalid && kr < kr_end && (unsigned)ih < (unsigned)a.H &&
                            (unsigned)iw < (unsigned)a.W;
            breg[i] = ok ? xg[(long)c * a.HW + ih * a.W + iw] : 0.f;
        }
#pragma unroll
        for (int i = 0; i < A_LOADS; ++i) {
            const int k = k0 + arow0 + i * A_KPP;
            const int kr = kr0 + acol;
            const bool ok = k < a.Kg && kr < kr_end;
            areg[i] = ok ? wg[(long)k * a.Kred + kr] : 0.f;
        }
    };
    auto sstore = [&](int buf) {
#pragma unroll
        for (int i = 0; i < B_LOADS; ++i) Bs[buf][brow0 + i * B_RPP][bcol] = breg[i];
#pragma unroll
        for (int i = 0; i < A_LOADS; ++i) As[buf][acol][arow0 + i * A_KPP] = areg[i];
    };

    floatx16 acc[BI][BJ];
#pragma unroll
    for (int bi = 0; bi < BI; ++bi)
#pragma unroll
        for (int bj = 0; bj < BJ; ++bj)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[bi][bj][v] = 0.f;

    const int nchunks = kr_end > kr_begin ? ceil_div(kr_end - kr_begin, KRC) : 0;
    if (nchunks > 0) {
        gload(kr_begin);
        sstore(0);
    }
    __syncthreads();
    const int hl = lane >> 5, ll = lane & 31;
    for (int t = 0; t < nchunks; ++t) {
        const int cur = t & 1;
        const bool more = t + 1 < nchunks;
        if (more) gload(kr_begin + (t + 1) * KRC);
#pragma unroll
        for (int kk = 0; kk < KRC; kk += 2) {
            float av[BI], bv[BJ];
#pragma unroll
            for (int bi = 0; bi < BI; ++bi) av[bi] = As[cur][kk + hl][wk * WTK + bi * 32 + ll];
#pragma unroll
            for (int bj = 0; bj < BJ; ++bj) bv[bj] = Bs[cur][kk + hl][wp * WTP + bj * 32 + ll];
#pragma unroll
            for (int bi = 0; bi < BI; ++bi)
#pragma unroll
                for (int bj = 0; bj < BJ; ++bj)
                    acc[bi][bj] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[bi], bv[bj], acc[bi][bj],
                                                                      0, 0, 0);
        }
        if (more) sstore(cur ^ 1);
        __syncthreads();
    }

    // Epilogue: bias + activation and the NCHW store, or (split reduction)
    // this split's raw fp32 partials, summed later by splitk_reduce_kernel.
#pragma unroll
    for (int bj = 0; bj < BJ; ++bj) {
        const int m = m0 + wp * WTP + bj * 32 + ll;
        if (m >= a.M) continue;
        const int n = m / a.PQ;
        const int pq = m - n * a.PQ;
        const long ybase = (long)n * a.ysn + pq;
#pragma unroll
        for (int bi = 0; bi < BI; ++bi) {
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int k = k0 + wk * WTK + bi * 32 + 8 * (v >> 2) + 4 * hl + (v & 3);
                if (k >= a.Kg) continue;
                const int kg = g * a.Kg + k;
                if (a.splits > 1) {
                    a.ws[((long)split * a.K + kg) * a.M + m] = acc[bi][bj][v];
                } else {
                    float val = acc[bi][bj][v] + (a.bias ? a.bias[kg] : 0.f);
                    if (a.res) val += a.res[ybase + (long)kg * a.PQ];
                    if (a.relu) val = fmaxf(val, 0.f);
                    a.y[ybase + (long)kg * a.PQ] = val;
                }
            }
        }
    }
}

// Sum the split partials in split order (deterministic), add bias and the
// residual, apply the activation and store NCHW.  Lanes walk the partials' [K][M] order, so reads
// are contiguous.  A thread requests its bias value and the partials of up to
// eight splits before it adds any of them: the launch costs one memory round
// trip, not one per split.  Partials are read through a buffer resource, so
// the slots past the last split read as zeros (adding them changes nothing).
// Channel-last bf16 output: the split partials are [splits][M][K] fp32; a
// thread sums 8 consecutive channels of one pixel over the splits in split
// order, adds bias and the bf16 residual (the layout of y), applies the
// activation, rounds to bf16 and stores 16 bytes.
__global__ __launch_bounds__(256) void splitk_reduce_cl_kernel(ConvArgs a)
{
    constexpr int kGroup = 4;                   // splits whose loads are in flight together
    constexpr unsigned kOut = 0x80000000u;      // past the partials: reads as zeros
    const unsigned K8 = (unsigned)a.K / 8;
    const unsigned units = (unsigned)a.M * K8;  // below 2^31, as every offset here (the launcher checks)
    const unsigned plane = (unsigned)a.M * a.K;
    const __amdgpu_buffer_rsrc_t wsr = __builtin_amdgcn_make_buffer_rsrc(
        a.ws, (short)0, (int)(a.splits * plane * 4u), 0x00020000);
    const uint16_t *res = reinterpret_cast<const uint16_t *>(a.res);
    uint16_t *y = reinterpret_cast<uint16_t *>(a.y);
    for (unsigned i = blockIdx.x * blockDim.x + threadIdx.x; i < units; i += gridDim.x * blockDim.x) {
        const unsigned m = fdiv(i, a.dv_kt);    // division by K/8
        const unsigned o = i - m * K8;
        const unsigned off = m * a.K + 8 * o;
        float bv[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) bv[e] = a.bias ? a.bias[8 * o + e] : 0.f;
        uint32_t rr[4] = {0, 0, 0, 0};
        if (res) {
            const uint4 r = *reinterpret_cast<const uint4 *>(res + off);
            rr[0] = r.x;
            rr[1] = r.y;
            rr[2] = r.z;
            rr[3] = r.w;
        }
        // split order from zero, kGroup splits' loads requested before any add
        float s[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) s[e] = 0.f;
        for (int sp = 0; sp < a.splits; sp += kGroup) {
            float4 lo[kGroup], hi[kGroup];
#pragma unroll
            for (int u = 0; u < kGroup; ++u) {
                const unsigned b = sp + u < a.splits ? ((sp + u) * plane + off) * 4u : kOut;
                lo[u] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(wsr, b, 0, 0));
                hi[u] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(wsr, b + 16u, 0, 0));
            }
#pragma unroll
            for (int u = 0; u < kGroup; ++u) {
                s[0] += lo[u].x;
                s[1] += lo[u].y;
                s[2] += lo[u].z;
                s[3] += lo[u].w;
                s[4] += hi[u].x;
                s[5] += hi[u].y;
                s[6] += hi[u].z;
                s[7] += hi[u].w;
            }
        }
        uint32_t d[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            float v0 = s[2 * e] + bv[2 * e];
            float v1 = s[2 * e + 1] + bv[2 * e + 1];
            if (res) {
                v0 += bf16_to_f32((uint16_t)(rr[e] & 0xFFFFu));
                v1 += bf16_to_f32((uint16_t)(rr[e] >> 16));
            }
            if (a.relu) {
                v0 = fmaxf(v0, 0.f);
                v1 = fmaxf(v1, 0.f);
            }
            d[e] = pack_bf16x2(v0, v1);
        }
        *reinterpret_cast<uint4 *>(y + off) = make_uint4(d[0], d[1], d[2], d[3]);
    }
}

__global__ __launch_bounds__(256) void splitk_reduce_kernel(ConvArgs a)
{
    constexpr int kGroup = 8;
    const unsigned total = (unsigned)a.K * a.M;
    const unsigned stride = gridDim.x * blockDim.x;
    const __amdgpu_buffer_rsrc_t wsr = __builtin_amdgcn_make_buffer_rsrc(
        a.ws, (short)0, (int)(a.splits * total * 4u), 0x00020000);
    if (a.vec4) {
        // One image with M % 4 == 0: the partials' order is y's own order and
        // four consecutive elements share one filter.
        const unsigned n4 = total / 4;
        for (unsigned i = blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += stride) {
            const unsigned k = fdiv(4 * i, a.dv_m);
            const float bv = a.bias ? a.bias[k] : 0.f;
            float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
            for (int sp = 0; sp < a.splits; sp += kGroup) {
                float4 v[kGroup];
#pragma unroll
                for (int u = 0; u < kGroup; ++u)
                    v[u] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(
                                                          wsr, ((sp + u) * n4 + i) * 16u, 0, 0));
#pragma unroll
                for (int u = 0; u < kGroup; ++u) {
                    s.x += v[u].x;
                    s.y += v[u].y;
                    s.z += v[u].z;
                    s.w += v[u].w;
                }
            }
            float o[4] = {s.x + bv, s.y + bv, s.z + bv, s.w + bv};
            if (a.res) {
                const float4 r = reinterpret_cast<const float4 *>(a.res)[i];
                o[0] += r.x;
                o[1] += r.y;
                o[2] += r.z;
                o[3] += r.w;
            }
            if (a.relu)
#pragma unroll
                for (int e = 0; e < 4; ++e) o[e] = fmaxf(o[e], 0.f);
            reinterpret_cast<float4 *>(a.y)[i] = make_float4(o[0], o[1], o[2], o[3]);
        }
        return;
    }
    for (unsigned i = blockIdx.x * blockDim.x + threadIdx.x; i < total; i += stride) {
        const unsigned k = fdiv(i, a.dv_m);
        const unsigned m = i - k * a.M;
        const float bv = a.bias ? a.bias[k] : 0.f;
        float s = 0.f;
        for (int sp = 0; sp < a.splits; sp += kGroup) {
            float v[kGroup];
#pragma unroll
            for (int u = 0; u < kGroup; ++u)
                v[u] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(wsr, ((sp + u) * total + i) * 4u, 0, 0));
#pragma unroll
            for (int u = 0; u < kGroup; ++u) s += v[u];
        }
        s += bv;
        const unsigned n = fdiv(m, a.dv_pq);
        const size_t yo = (size_t)n * a.ysn + (size_t)k * a.PQ + (m - n * a.PQ);
        if (a.res) s += a.res[yo];
        if (a.relu) s = fmaxf(s, 0.f);
        a.y[yo] = s;
    }
}

struct TileInfo {
    int bkc, bpx, wk, wp, krc;
};
// Tile table: 0 = 128x128 (large layers), 1 = 64x64, 2 = 32 channels x 64 pixels.
// Bigger reduction chunks for the smaller tiles: small layers are bound by
// the latency of a global-load round trip per chunk, so fewer, larger chunks
// (more loads in flight per round trip) matter more there than occupancy.
const TileInfo kTiles[] = {{128, 128, 2, 2, 16}, {64, 64, 2, 2, 32}, {32, 64, 1, 2, 64}};
constexpr int kNumTiles = 3;

int rs_template(int v) { return (v == 1 || v == 3 || v == 7) ? v : 0; }

template <int R_, int S_>
hipError_t launch_rs(const ConvArgs &a, int tile, dim3 grid, hipStream_t st)
{
    switch (tile) {
    case 0:
        launch_kernel((igemm_f32_kernel<R_, S_, 128, 128, 2, 2, 16>), grid, dim3(256), 0, st, a);
        break;
    case 1:
        launch_kernel((igemm_f32_kernel<R_, S_, 64, 64, 2, 2, 32>), grid, dim3(256), 0, st, a);
        break;
    default:
        launch_kernel((igemm_f32_kernel<R_, S_, 32, 64, 1, 2, 64>), grid, dim3(128), 0, st, a);
        break;
    }
    return hipGetLastError();
}

}  // namespace

// Pick the tile and the reduction split: the biggest tile that still gives
// about 1.5 work-groups per CU (filters of at most 64 channels skip the
// 128-channel tile, which would leave half of its MFMAs idle); otherwise the
// smallest tile, with the reduction split until there are about two
// work-groups per CU (each split keeps at least one whole chunk).  Measured
// on VGG-16 at batch 8: 64x64 runs the 64-filter conv1_2 at 68 TFLOP/s
// against 41 for 128x128.
IgemmPlan plan_igemm_f32(const ConvProblem &p, int num_cus, int max_splits)
{
    IgemmPlan plan{kNumTiles - 1, 1, p.Kred, 0};
    const long target = 3L * num_cus / 2;
    for (int t = p.Kg <= 64 ? 1 : 0; t < kNumTiles; ++t) {
        const long tiles = (long)ceil_div(p.M, kTiles[t].bpx) * ceil_div(p.Kg, kTiles[t].bkc) * p.groups;
        if (tiles < target && t < kNumTiles - 1) continue;
        plan.tile = t;
        const int krc = kTiles[t].krc;
        const int chunks = ceil_div(p.Kred, krc);
        int splits = tiles < target ? (int)((2L * num_cus + tiles - 1) / tiles) : 1;
        if (splits > chunks) splits = chunks;
        if (splits > max_splits) splits = max_splits;
        const int chunks_per = ceil_div(chunks, splits);
        splits = ceil_div(chunks, chunks_per);   // no empty splits
        plan.splits = splits;
        plan.kr_per_split = chunks_per * krc;
        plan.ws_bytes = splits > 1 ? (size_t)splits * p.K * p.M * sizeof(float) : 0;
        break;
    }
    return plan;
}

void describe_igemm_f32(const ConvProblem &p, const IgemmPlan &plan, char *buf, int len,
                        int *launches)
{
    const TileInfo &t = kTiles[plan.tile];
    int R = rs_template(p.R), S = rs_template(p.S);
    if (R == 0 || S == 0 || R != S) R = S = 0;
    snprintf(buf, len, "igemm_f32_kernel<%d, %d, %d, %d, %d, %d, %d>%s", R, S, t.bkc, t.bpx, t.wk,
             t.wp, t.krc, plan.splits > 1 ? " + splitk_reduce_kernel" : "");
    *launches = plan.splits > 1 ? 2 : 1;
}

hipError_t launch_igemm_f32(const ConvProblem &p, const IgemmPlan &plan, const float *x,
                            const float *w, const float *bias, float *y, float *ws,
                            hipStream_t st, const LaunchHook *hook)
{
    ConvArgs a = make_args(p);
    a.x = x;
    a.w = w;
    a.bias = bias;
    a.y = y;
    a.ws = plan.splits > 1 ? ws : nullptr;
    a.splits = plan.splits;
    a.kr_per_split = plan.kr_per_split;
    const TileInfo &ti = kTiles[plan.tile];
    dim3 grid(ceil_div(p.M, ti.bpx), ceil_div(p.Kg, ti.bkc), p.groups * plan.splits);
    hipError_t e = hook ? hook->before_launch(hook->ctx, st) : hipSuccess;
    if (e != hipSuccess) return e;
    if (p.R == 1 && p.S == 1)
        e = launch_rs<1, 1>(a, plan.tile, grid, st);
    else if (p.R == 3 && p.S == 3)
        e = launch_rs<3, 3>(a, plan.tile, grid, st);
    else if (p.R == 7 && p.S == 7)
        e = launch_rs<7, 7>(a, plan.tile, grid, st);
    else
        e = launch_rs<0, 0>(a, plan.tile, grid, st);
    if (e != hipSuccess || plan.splits == 1) return e;
    if (hook && (e = hook->before_launch(hook->ctx, st)) != hipSuccess) return e;
    return launch_splitk_reduce(a, st);
}

hipError_t launch_splitk_reduce(ConvArgs a, hipStream_t st)
{
    if (a.ycl) {
        // channel-last bf16 output: partials [splits][M][K], 8 channels per thread
        const long units = (long)a.M * (a.K / 8);
        if ((long)a.splits * a.M * a.K * 4 >= (1L << 31) || a.K % 8) return hipErrorInvalidValue;
        a.dv_kt = make_fastdiv(a.K / 8);
        long blocks = (units + 255) / 256;
        if (blocks > 8192) blocks = 8192;
        launch_kernel(splitk_reduce_cl_kernel, dim3((unsigned)blocks), dim3(256), 0, st, a);
        return hipGetLastError();
    }
    const long total = (long)a.K * a.M;
    // 32-bit offsets, also for the zero-reading slots of the last group of 8
    if ((long)(a.splits + 7) * total * 4 >= (1L << 31)) return hipErrorInvalidValue;
    a.vec4 = a.N == 1 && a.M % 4 == 0 && (uintptr_t)a.y % 16 == 0 && (uintptr_t)a.ws % 16 == 0 &&
             (uintptr_t)a.res % 16 == 0;
    a.dv_m = make_fastdiv(a.M);
    long blocks = (a.vec4 ? total / 4 : total + 255) / 256 + 1;
    if (blocks > 8192) blocks = 8192;
    launch_kernel(splitk_reduce_kernel, dim3((unsigned)blocks), dim3(256), 0, st, a);
    return hipGetLastError();
}

}  // namespace miconv
