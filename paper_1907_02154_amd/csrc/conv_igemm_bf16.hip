// Dense conv2d with bf16 x and w, fp32 accumulation and fp32 output, as an
// implicit GEMM on gfx950's v_mfma_f32_32x32x16_bf16.
//
// GEMM view as in the fp32 path: D[k][m] = sum_kr W[k][kr] X[kr][m], k =
// output channel, m = (n, p, q), kr = (c, r, s).  The bf16 MFMA wants, in
// every lane, 8 consecutive reduction elements of one row (A) and of one
// column (B).  Both LDS tiles are therefore stored reduction-contiguous:
//   As[k][kr], Bs[m][kr]   (rows padded by 16 bytes: conflict-free 16-byte reads)
// so each operand is a single 16-byte LDS read.  Filter rows are
// reduction-contiguous in KCRS already (16-byte global loads).  The input is
// pixel-contiguous in NCHW, so the B tile is transposed on its way into LDS:
//  * 1x1, stride 1, no padding, H*W % 8 == 0: a lane loads 4 channels x 8
//    consecutive pixels (four 16-byte loads) and transposes the 4x8 block of
//    16-bit values in registers (v_perm) into 8 pixel rows of 4 channels;
//  * any other shape: a lane gathers 8 consecutive taps of one pixel (2-byte
//    loads, zero in the padding) and writes them as one 16-byte row piece.
// Double-buffered LDS, one barrier per chunk, the next chunk's global loads
// in flight during the current chunk's MFMAs.
//
// MFMA 32x32x16 bf16, lane l, half h = l / 32: A = W[i = l%32][8h .. 8h+7],
// B = X[8h .. 8h+7][j = l%32]; D reg v = (i = 8*(v/4) + 4h + v%4, j = l%32).
// A and B put the same reduction index in the same (h, element) slot, which
// is all the product needs.
#include "internal.h"

#include <cstdio>

namespace miconv {
namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

__device__ inline uint32_t pack_lo(uint32_t x, uint32_t y)   // (x.lo, y.lo)
{
    return __builtin_amdgcn_perm(y, x, 0x05040100u);
}
__device__ inline uint32_t pack_hi(uint32_t x, uint32_t y)   // (x.hi, y.hi)
{
    return __builtin_amdgcn_perm(y, x, 0x07060302u);
}

// FAST1X1: the vectorised 1x1 loader; VA: 16-byte filter loads; KRSC:
// filters pre-packed [K][R][S][C/groups] with C/groups % 8 == 0, so a group
// of 8 reduction indices is 8 channels at one filter position (one padding
// check and one address per group).
template <int R_, int S_, int BKC, int BPX, int KRC, bool FAST1X1, bool VA, bool KRSC>
__global__ __launch_bounds__(256) void igemm_bf16_kernel(ConvArgs a)
{
    constexpr int NT = 256;
    constexpr int WTK = BKC / 2, WTP = BPX / 2;      // 2 x 2 wavefronts
    constexpr int BI = WTK / 32, BJ = WTP / 32;
    constexpr int LDR = KRC + 8;                     // row stride in bf16 (16 B pad)
    constexpr int A_GROUPS = BKC * KRC / 8 / NT;     // 8-element groups per lane
    constexpr int B_GROUPS = BPX * KRC / 8 / NT;
    static_assert(BI >= 1 && BJ >= 1, "wave tile");
    static_assert(A_GROUPS >= 1 && B_GROUPS >= 1 && (BKC * KRC / 8) % NT == 0 &&
                  (BPX * KRC / 8) % NT == 0 && NT % BPX == 0, "loader shape");
    constexpr int FAST_LANES = (BPX / 8) * (KRC / 4);  // lanes of the vectorised 1x1 loader
    static_assert(FAST_LANES <= NT, "1x1 loader shape");

    __shared__ __attribute__((aligned(16))) uint16_t As[2][BKC][LDR];
    __shared__ __attribute__((aligned(16))) uint16_t Bs[2][BPX][LDR];

    const uint16_t *__restrict__ x = static_cast<const uint16_t *>(a.x);
    const uint16_t *__restrict__ w = static_cast<const uint16_t *>(a.w);
    const int R = R_ ? R_ : a.R;
    const int S = S_ ? S_ : a.S;
    const int RS = R * S;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wid = tid >> 6;
    const int wk = wid >> 1, wp = wid & 1;
    const int h = lane >> 5, ll = lane & 31;
    const int g = blockIdx.z % a.groups;
    const int split = blockIdx.z / a.groups;
    const int m0 = blockIdx.x * BPX;
    const int k0 = blockIdx.y * BKC;
    const int kr_begin = split * a.kr_per_split;
    const int kr_end = min(a.Kred, kr_begin + a.kr_per_split);
    const uint16_t *wg = w + (long)g * a.Kg * a.Kred;
    const uint16_t *xg = x + (long)g * a.Cg * a.HW;

    // ---- A loader: group gi -> (row k, 8 taps kr8) ----
    uint4 areg[A_GROUPS];
    auto load_a = [&](int kr0) {
#pragma unroll
        for (int i = 0; i < A_GROUPS; ++i) {
            const int gi = tid + i * NT;
            const int k = gi / (KRC / 8);
            const int kr = kr0 + (gi % (KRC / 8)) * 8;
            const bool kv = k0 + k < a.Kg;
            const uint16_t *src = wg + (long)(k0 + k) * a.Kred + kr;
            if (VA && kv && kr + 8 <= kr_end) {
                areg[i] = *reinterpret_cast<const uint4 *>(src);
            } else {
                uint32_t d[4];
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    const uint32_t lo = (kv && kr + 2 * t < kr_end) ? src[2 * t] : 0u;
                    const uint32_t hi = (kv && kr + 2 * t + 1 < kr_end) ? src[2 * t + 1] : 0u;
                    d[t] = lo | (hi << 16);
                }
                areg[i] = make_uint4(d[0], d[1], d[2], d[3]);
            }
        }
    };
    auto store_a = [&](int buf) {
#pragma unroll
        for (int i = 0; i < A_GROUPS; ++i) {
            const int gi = tid + i * NT;
            *reinterpret_cast<uint4 *>(&As[buf][gi / (KRC / 8)][(gi % (KRC / 8)) * 8]) = areg[i];
        }
    };

    // ---- B loader ----
    // Generic: group gi -> pixel (gi % BPX), taps kr8 = gi / BPX; the lane's
    // pixel is the same for all its groups because NT % BPX == 0.
    // Fast 1x1: lane -> 4 channels (tid % (KRC/4)) x 8 pixels (tid / (KRC/4)):
    // channel quads vary fastest across lanes so that the transposed 8-byte
    // LDS writes of one instruction spread over the banks (pixel octets are
    // 8 rows = a multiple of 32 banks apart).
    constexpr int B_REGS = FAST1X1 ? 4 : B_GROUPS;
    uint4 breg[B_REGS];
    const int bpix = FAST1X1 ? (tid / (KRC / 4)) * 8 : tid % BPX;
    const int mB = m0 + bpix;
    const bool fast_lane = !FAST1X1 || tid < FAST_LANES;
    const bool mvalid = mB < a.M && fast_lane;
    int ih0 = 0, iw0 = 0;
    long xoff = 0;
    {
        const int mm = mvalid ? mB : 0;
        const int n = mm / a.PQ;
        const int pq = mm - n * a.PQ;
        const int p = pq / a.Q;
        const int q = pq - p * a.Q;
        ih0 = p * a.stride - a.pad;
        iw0 = q * a.stride - a.pad;
        xoff = (long)n * a.C * a.HW + (FAST1X1 ? pq : 0);
    }
    auto load_b = [&](int kr0) {
        if constexpr (FAST1X1) {
            // rows = 4 consecutive channels, 8 pixels each (pixel groups never
            // straddle an image because H*W % 8 == 0)
            const int c0 = kr0 + (tid % (KRC / 4)) * 4;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int c = c0 + r;
                breg[r] = (mvalid && c < kr_end)
                              ? *reinterpret_cast<const uint4 *>(xg + xoff + (long)c * a.HW)
                              : make_uint4(0, 0, 0, 0);
            }
        } else if constexpr (KRSC) {
#pragma unroll
            for (int i = 0; i < B_GROUPS; ++i) {
                const int kr8 = kr0 + (tid / BPX + i * (NT / BPX)) * 8;
                const int rs = kr8 / a.Cg;
                const int c0 = kr8 - rs * a.Cg;
                const int r = rs / S;
                const int s = rs - r * S;
                const int ih = ih0 + r, iw = iw0 + s;
                const bool okp = mvalid && (unsigned)ih < (unsigned)a.H && (unsigned)iw < (unsigned)a.W;
                const uint16_t *src = xg + xoff + (long)c0 * a.HW + ih * a.W + iw;
                uint32_t d[4];
#pragma unroll
                for (int t = 0; t < 8; t += 2) {
                    const uint32_t lo = (okp && kr8 + t < kr_end) ? src[(long)t * a.HW] : 0u;
                    const uint32_t hi = (okp && kr8 + t + 1 < kr_end) ? src[(long)(t + 1) * a.HW] : 0u;
                    d[t >> 1] = lo | (hi << 16);
                }
                breg[i] = make_uint4(d[0], d[1], d[2], d[3]);
            }
        } else {
#pragma unroll
            for (int i = 0; i < B_GROUPS; ++i) {
                const int kr8 = kr0 + (tid / BPX + i * (NT / BPX)) * 8;
                uint32_t d[4];
#pragma unroll
                for (int t = 0; t < 8; ++t) {
                    const int kr = kr8 + t;
                    const int c = kr / RS;
                    const int rs = kr - c * RS;
                    const int r = rs / S;
                    const int s = rs - r * S;
                    const int ih = ih0 + r, iw = iw0 + s;
                    const bool ok = mvalid && kr < kr_end && (unsigned)ih < (unsigned)a.H &&
                                    (unsigned)iw < (unsigned)a.W;
                    const uint32_t v = ok ? xg[xoff + (long)c * a.HW + ih * a.W + iw] : 0u;
                    if (t & 1)
                        d[t >> 1] |= v << 16;
                    else
                        d[t >> 1] = v;
                }
                breg[i] = make_uint4(d[0], d[1], d[2], d[3]);
            }
        }
    };
    auto store_b = [&](int buf) {
        if constexpr (FAST1X1) {
            if (!fast_lane) return;
            // transpose 4 channel rows x 8 pixels -> 8 pixel rows x 4 channels
            const int kc = (tid % (KRC / 4)) * 4;
            const uint32_t *r0 = reinterpret_cast<const uint32_t *>(&breg[0]);
            const uint32_t *r1 = reinterpret_cast<const uint32_t *>(&breg[1]);
            const uint32_t *r2 = reinterpret_cast<const uint32_t *>(&breg[2]);
            const uint32_t *r3 = reinterpret_cast<const uint32_t *>(&breg[3]);
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                uint2 ev = make_uint2(pack_lo(r0[t], r1[t]), pack_lo(r2[t], r3[t]));
                uint2 od = make_uint2(pack_hi(r0[t], r1[t]), pack_hi(r2[t], r3[t]));
                *reinterpret_cast<uint2 *>(&Bs[buf][bpix + 2 * t][kc]) = ev;
                *reinterpret_cast<uint2 *>(&Bs[buf][bpix + 2 * t + 1][kc]) = od;
            }
        } else {
#pragma unroll
            for (int i = 0; i < B_GROUPS; ++i)
                *reinterpret_cast<uint4 *>(&Bs[buf][bpix][(tid / BPX + i * (NT / BPX)) * 8]) = breg[i];
        }
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
        load_a(kr_begin);
        load_b(kr_begin);
        store_a(0);
        store_b(0);
    }
    __syncthreads();
    for (int t = 0; t < nchunks; ++t) {
        const int cur = t & 1;
        const bool more = t + 1 < nchunks;
        if (more) {
            load_a(kr_begin + (t + 1) * KRC);
            load_b(kr_begin + (t + 1) * KRC);
        }
#pragma unroll
        for (int ks = 0; ks < KRC; ks += 16) {
            bf16x8 av[BI], bv[BJ];
#pragma unroll
            for (int bi = 0; bi < BI; ++bi)
                av[bi] = *reinterpret_cast<const bf16x8 *>(&As[cur][wk * WTK + bi * 32 + ll][ks + 8 * h]);
#pragma unroll
            for (int bj = 0; bj < BJ; ++bj)
                bv[bj] = *reinterpret_cast<const bf16x8 *>(&Bs[cur][wp * WTP + bj * 32 + ll][ks + 8 * h]);
#pragma unroll
            for (int bi = 0; bi < BI; ++bi)
#pragma unroll
                for (int bj = 0; bj < BJ; ++bj)
                    acc[bi][bj] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[bi], bv[bj], acc[bi][bj],
                                                                         0, 0, 0);
        }
        if (more) {
            store_a(cur ^ 1);
            store_b(cur ^ 1);
        }
        __syncthreads();
    }

    // Epilogue: bias + activation and NCHW fp32 store, or split partials.
    // Channel quantities (bias, plane offset) are formed once per register
    // and reused across the pixel blocks.
    long ybase[BJ];
    bool mok[BJ];
#pragma unroll
    for (int bj = 0; bj < BJ; ++bj) {
        const int m = m0 + wp * WTP + bj * 32 + ll;
        mok[bj] = m < a.M;
        const int mm = mok[bj] ? m : 0;
        const int n = mm / a.PQ;
        ybase[bj] = a.splits > 1 ? (long)mm : (long)n * a.ysn + (mm - n * a.PQ);
    }
    const long cstride = a.splits > 1 ? (long)a.M : (long)a.PQ;
    float *out = a.splits > 1 ? a.ws + (long)split * a.K * a.M : a.y;
#pragma unroll
    for (int bi = 0; bi < BI; ++bi) {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const int k = k0 + wk * WTK + bi * 32 + 8 * (v >> 2) + 4 * h + (v & 3);
            if (k >= a.Kg) continue;
            const int kg = g * a.Kg + k;
            const float bv = (a.splits == 1 && a.bias) ? a.bias[kg] : 0.f;
            const long coff = (long)kg * cstride;
#pragma unroll
            for (int bj = 0; bj < BJ; ++bj) {
                if (!mok[bj]) continue;
                float val = acc[bi][bj][v];
                if (a.splits == 1) {
                    val += bv;
                    if (a.res) val += a.res[ybase[bj] + coff];
                    if (a.relu) val = fmaxf(val, 0.f);
                }
                out[ybase[bj] + coff] = val;
            }
        }
    }
}

struct TileB {
    int bkc, bpx;
};
// 0: 128 x 128 (4 wavefronts of 64 x 64); 1: 64 x 64 (4 wavefronts of 32 x 32).
const TileB kTilesB[] = {{128, 128}, {64, 64}};
constexpr int kKrcB = 64;

template <int R_, int S_, bool F, bool VA, bool KRSC>
void launch_tile(const ConvArgs &a, int tile, dim3 grid, hipStream_t st)
{
    if (tile == 0)
        launch_kernel((igemm_bf16_kernel<R_, S_, 128, 128, kKrcB, F, VA, KRSC>), grid, dim3(256), 0, st, a);
    else
        launch_kernel((igemm_bf16_kernel<R_, S_, 64, 64, kKrcB, F, VA, KRSC>), grid, dim3(256), 0, st, a);
}

template <int R_, int S_, bool KRSC>
void launch_rs(const ConvArgs &a, int tile, bool fast, bool va, dim3 grid, hipStream_t st)
{
    if (fast) {
        if (va) launch_tile<1, 1, true, true, false>(a, tile, grid, st);
        else launch_tile<1, 1, true, false, false>(a, tile, grid, st);
    } else {
        if (va) launch_tile<R_, S_, false, true, KRSC>(a, tile, grid, st);
        else launch_tile<R_, S_, false, false, KRSC>(a, tile, grid, st);
    }
}

int rs_template(int v) { return (v == 1 || v == 3 || v == 7) ? v : 0; }

}  // namespace

// The biggest tile that gives about two work-groups per CU, else the small
// tile with a reduction split (at least 2 chunks of 64 taps per split).
IgemmPlan plan_igemm_bf16(const ConvProblem &p, int num_cus, int max_splits)
{
    IgemmPlan plan{1, 1, p.Kred, 0};
    const long target = 2L * num_cus;
    for (int t = 0; t < 2; ++t) {
        const long tiles = (long)ceil_div(p.M, kTilesB[t].bpx) * ceil_div(p.Kg, kTilesB[t].bkc) * p.groups;
        if (tiles < target && t == 0) continue;
        plan.tile = t;
        const int chunks = ceil_div(p.Kred, kKrcB);
        int splits = tiles < target ? (int)((target + tiles - 1) / tiles) : 1;
        if (splits > chunks / 2) splits = chunks / 2;
        if (splits > max_splits) splits = max_splits;
        if (splits < 1) splits = 1;
        const int per = ceil_div(chunks, splits);
        splits = ceil_div(chunks, per);
        plan.splits = splits;
        plan.kr_per_split = per * kKrcB;
        plan.ws_bytes = splits > 1 ? (size_t)splits * p.K * p.M * sizeof(float) : 0;
        break;
    }
    return plan;
}

static bool fast_1x1(const ConvProblem &p, const void *x)
{
    return p.R == 1 && p.S == 1 && p.stride == 1 && p.pad == 0 && (p.H * p.W) % 8 == 0 &&
           ((uintptr_t)x % 16) == 0;
}

void describe_igemm_bf16(const ConvProblem &p, const IgemmPlan &plan, bool fast, bool va,
                         char *buf, int len, int *launches)
{
    const TileB &t = kTilesB[plan.tile];
    int R = rs_template(p.R), S = rs_template(p.S);
    if (R == 0 || S == 0 || R != S) R = S = 0;
    if (fast) R = S = 1;
    const bool krsc = plan.krsc && !(p.R == 1 && p.S == 1);
    if (krsc && R != 3) R = S = 0;
    snprintf(buf, len, "igemm_bf16_kernel<%d, %d, %d, %d, %d, %s, %s, %s>%s", R, S, t.bkc, t.bpx,
             kKrcB, fast ? "true" : "false", va ? "true" : "false", krsc ? "true" : "false",
             plan.splits > 1 ? " + splitk_reduce_kernel" : "");
    *launches = plan.splits > 1 ? 2 : 1;
}

bool bf16_fast_1x1(const ConvProblem &p, const void *x) { return fast_1x1(p, x); }

hipError_t launch_igemm_bf16(const ConvProblem &p, const IgemmPlan &plan, bool fast, bool va,
                             const uint16_t *x, const uint16_t *w, const float *bias, float *y,
                             float *ws, hipStream_t st, const LaunchHook *hook)
{
    ConvArgs a = make_args(p);
    a.x = x;
    a.w = w;
    a.bias = bias;
    a.y = y;
    a.ws = plan.splits > 1 ? ws : nullptr;
    a.splits = plan.splits;
    a.kr_per_split = plan.kr_per_split;
    const TileB &t = kTilesB[plan.tile];
    dim3 grid(ceil_div(p.M, t.bpx), ceil_div(p.Kg, t.bkc), p.groups * plan.splits);
    hipError_t e = hook ? hook->before_launch(hook->ctx, st) : hipSuccess;
    if (e != hipSuccess) return e;
    if (plan.krsc && !(p.R == 1 && p.S == 1)) {   // filters packed KRSC
        if (p.R == 3 && p.S == 3)
            launch_rs<3, 3, true>(a, plan.tile, false, va, grid, st);
        else
            launch_rs<0, 0, true>(a, plan.tile, false, va, grid, st);
    } else if (p.R == 1 && p.S == 1) {
        launch_rs<1, 1, false>(a, plan.tile, fast, va, grid, st);
    } else if (p.R == 3 && p.S == 3) {
        launch_rs<3, 3, false>(a, plan.tile, false, va, grid, st);
    } else if (p.R == 7 && p.S == 7) {
        launch_rs<7, 7, false>(a, plan.tile, false, va, grid, st);
    } else {
        launch_rs<0, 0, false>(a, plan.tile, false, va, grid, st);
    }
    e = hipGetLastError();
    if (e != hipSuccess || plan.splits == 1) return e;
    if (hook && (e = hook->before_launch(hook->ctx, st)) != hipSuccess) return e;
    return launch_splitk_reduce(a, st);
}

}  // namespace miconv
