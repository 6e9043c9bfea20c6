// Dense conv2d in fp32 for small GEMM extents (batch-1 layers): an implicit
// GEMM in which every wavefront feeds the matrix cores straight from global
// memory, with no LDS staging and no barriers in the main loop.
//
// Why: at batch 1 the layers of ResNet-50 / MobileNet have N*P*Q = 49..12544
// output pixels, so an LDS-staged tile kernel runs few chunks per
// work-group and spends its time waiting for one global round trip per chunk
// behind a barrier.  Here each wavefront streams its own share of the
// reduction with several blocks of loads in flight, and the parallelism the
// output tiles lack is recovered by splitting the reduction across the
// wavefronts of a work-group (combined through LDS in a fixed order) and, for
// the smallest layers, across work-groups (splitk_reduce_kernel).
//
// MFMA v_mfma_f32_32x32x2_f32, lane l of 64, half h = l / 32:
//   A operand = W[k0 + l%32][kr],  B operand = X[kr][m0 + l%32]
// The reduction is walked in blocks of 8 taps; in block b, step e (0..3),
// half h supplies tap kr = 8b + 4h + e.  The MFMA sums over both halves, so
// the 4 steps cover the block's 8 taps once, and a lane's A values for the 4
// steps are 4 consecutive floats of a KCRS filter row: one 16-byte load.  Its
// B values are 4 gathered taps of the im2col matrix for one output pixel;
// the 32 lanes of a half read 32 consecutive pixels of the same tap.
// Output: D reg v is channel 8*(v/4) + 4*h + v%4 and pixel l%32, so every
// store writes 32 consecutive pixels (128 bytes) of one NCHW channel plane.
#include "internal.h"

#include <cstdio>

namespace miconv {
namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));


// BJ = 32-pixel blocks per wavefront tile; VA = the filter row length allows
// 16-byte loads (Kred % 4 == 0); KRSC = filters pre-packed [K][R][S][C/groups]
// (reduction ordered r, s, c with C/groups % 8 == 0), so the 4 taps of a
// half-block are 4 channels at one filter position: one padding check and
// one address per half-block.
template <int R_, int S_, int WAVES, int BJ, bool VA, bool KRSC, bool PK>
__global__ __launch_bounds__(64 * WAVES) void igemm_wave_f32_kernel(ConvArgs a)
{
    constexpr int kDepth = BJ == 2 ? 2 : 4;   // blocks of loads in flight per wavefront
    const float *__restrict__ x = static_cast<const float *>(a.x);
    const float *__restrict__ w = static_cast<const float *>(a.w);
    const int R = R_ ? R_ : a.R;
    const int S = S_ ? S_ : a.S;
    const int RS = R * S;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int h = lane >> 5, ll = lane & 31;
    // XCD-aware tile order: the hardware deals work-groups to the 8 XCDs
    // round-robin (work-group b runs on XCD b % 8), so logical tiles are
    // renumbered to give each XCD one contiguous range, pixel tiles fastest:
    // the work-groups that read the same filter rows share an L2.
    const int mtiles = ceil_div(a.M, 32 * BJ), ktiles = ceil_div(a.Kg, 32);
    const int T = gridDim.x;
    const int xcd = blockIdx.x % 8, jx = blockIdx.x / 8;
    const int L = xcd * (T / 8) + min(xcd, T % 8) + jx;
    const int mx = L % mtiles;
    const int ky = (L / mtiles) % ktiles;
    const int z = L / (mtiles * ktiles);
    const int g = z % a.groups;
    const int split = z / a.groups;
    const int m0 = mx * (32 * BJ);
    const int k0 = ky * 32;
    const int kr_begin = split * a.kr_per_split;
    const int kr_end = min(a.Kred, kr_begin + a.kr_per_split);
    const int nblk = kr_end > kr_begin ? ceil_div(kr_end - kr_begin, 8) : 0;

    // A: this lane's filter row, or (PK) its 16-byte slot of the packed
    // filters: w_pk[g][k/32][kr/8][lane][4] holds W[k0 + l%32][8*blk + 4*h + e],
    // zero past K and Kred, so a wavefront's A load is 1 KB contiguous.
    const int kA = k0 + ll;
    const bool kvalid = kA < a.Kg;
    const float *wrow = w + ((long)g * a.Kg + (kvalid ? kA : 0)) * a.Kred;
    const float *wpk = w + (((long)(g * ktiles + ky) * ceil_div(a.Kred, 8) + kr_begin / 8) * 64 + lane) * 4;

    // B: this lane's output pixels, one per 32-pixel block.
    int ih0[BJ], iw0[BJ];
    bool mvalid[BJ];
    const float *xb[BJ];
#pragma unroll
    for (int j = 0; j < BJ; ++j) {
        const int m = m0 + j * 32 + ll;
        mvalid[j] = m < a.M;
        const int mm = mvalid[j] ? m : 0;
        const int n = mm / a.PQ;
        const int pq = mm - n * a.PQ;
        const int p = pq / a.Q;
        const int q = pq - p * a.Q;
        ih0[j] = p * a.stride - a.pad;
        iw0[j] = q * a.stride - a.pad;
        xb[j] = x + ((long)n * a.C + (long)g * a.Cg) * a.HW;
    }

    struct Frag {
        float av[4];
        float bv[BJ][4];
    };

    // Block blk of this split: taps kr_begin + 8*blk + 4h + e, e = 0..3.
    auto load = [&](Frag &f, int blk) {
        const int kr0 = kr_begin + 8 * blk + 4 * h;
        const bool live = blk < nblk;
        if (PK) {
            const float4 v = live ? *reinterpret_cast<const float4 *>(wpk + (long)blk * 256)
                                  : make_float4(0.f, 0.f, 0.f, 0.f);
            f.av[0] = v.x;
            f.av[1] = v.y;
            f.av[2] = v.z;
            f.av[3] = v.w;
        } else if (VA && live && kvalid && kr0 + 4 <= kr_end) {
            const float4 v = *reinterpret_cast<const float4 *>(wrow + kr0);
            f.av[0] = v.x;
            f.av[1] = v.y;
            f.av[2] = v.z;
            f.av[3] = v.w;
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
                f.av[e] = (live && kvalid && kr0 + e < kr_end) ? wrow[kr0 + e] : 0.f;
        }
        if constexpr (KRSC) {
            const int krb = kr_begin + 8 * blk;        // block base: one filter position
            const int rs = krb / a.Cg;
            const int c0 = krb - rs * a.Cg + 4 * h;
            const int r = rs / S;
            const int s = rs - r * S;
#pragma unroll
            for (int j = 0; j < BJ; ++j) {
                const int ih = ih0[j] + r, iw = iw0[j] + s;
                const bool okp = live && mvalid[j] && (unsigned)ih < (unsigned)a.H &&
                                 (unsigned)iw < (unsigned)a.W;
                const float *src = xb[j] + (long)c0 * a.HW + ih * a.W + iw;
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    f.bv[j][e] = (okp && kr0 + e < kr_end) ? src[(long)e * a.HW] : 0.f;
            }
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int kr = kr0 + e;
                const int c = kr / RS;
                const int rs = kr - c * RS;
                const int r = rs / S;
                const int s = rs - r * S;
#pragma unroll
                for (int j = 0; j < BJ; ++j) {
                    const int ih = ih0[j] + r, iw = iw0[j] + s;
                    const bool ok = live && kr < kr_end && mvalid[j] && (unsigned)ih < (unsigned)a.H &&
                                    (unsigned)iw < (unsigned)a.W;
                    f.bv[j][e] = ok ? xb[j][(long)c * a.HW + ih * a.W + iw] : 0.f;
                }
            }
        }
    };

    floatx16 acc[BJ];
#pragma unroll
    for (int j = 0; j < BJ; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[j][v] = 0.f;

    // This wavefront takes blocks wave, wave + WAVES, ...; kDepth in flight.
    const int my_blocks = nblk > wave ? ceil_div(nblk - wave, WAVES) : 0;
    Frag f[kDepth];
#pragma unroll
    for (int d = 0; d < kDepth; ++d) load(f[d], d < my_blocks ? wave + d * WAVES : nblk);
    for (int it = 0; it < my_blocks; it += kDepth) {
#pragma unroll
        for (int d = 0; d < kDepth; ++d) {
            if (it + d < my_blocks) {
#pragma unroll
                for (int e = 0; e < 4; ++e)
#pragma unroll
                    for (int j = 0; j < BJ; ++j)
                        acc[j] = __builtin_amdgcn_mfma_f32_32x32x2f32(f[d].av[e], f[d].bv[j][e],
                                                                      acc[j], 0, 0, 0);
            }
            const int nxt = it + d + kDepth;
            load(f[d], nxt < my_blocks ? wave + nxt * WAVES : nblk);
        }
    }

    // Combine the wavefronts' partial tiles through LDS: every element is
    // summed over the wavefronts in wave order (deterministic), and all lanes
    // of the work-group share the epilogue.  Element (jv, l) of a tile is
    // accumulator register v = jv % 16 of pixel block j = jv / 16 in lane l.
    __shared__ float red[WAVES][BJ * 16][64];
#pragma unroll
    for (int j = 0; j < BJ; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) red[wave][j * 16 + v][lane] = acc[j][v];
    __syncthreads();
    for (int idx = tid; idx < BJ * 16 * 64; idx += 64 * WAVES) {
        const int jv = idx >> 6, l = idx & 63;
        const int j = jv >> 4, v = jv & 15;
        float sum = red[0][jv][l];
#pragma unroll
        for (int ww = 1; ww < WAVES; ++ww) sum += red[ww][jv][l];
        const int m = m0 + j * 32 + (l & 31);
        const int k = k0 + 8 * (v >> 2) + 4 * (l >> 5) + (v & 3);
        if (m >= a.M || k >= a.Kg) continue;
        const int kg = g * a.Kg + k;
        if (a.splits > 1) {
            a.ws[((long)split * a.K + kg) * a.M + m] = sum;
        } else {
            const int n = m / a.PQ;
            const int pq = m - n * a.PQ;
            float val = sum + (a.bias ? a.bias[kg] : 0.f);
            if (a.relu) val = fmaxf(val, 0.f);
            a.y[((long)n * a.K + kg) * a.PQ + pq] = val;
        }
    }
}

template <int R_, int S_, int WAVES, int BJ, bool KRSC>
void launch_va(const ConvArgs &a, bool va, bool pk, dim3 grid, hipStream_t st)
{
    if (pk)
        launch_kernel((igemm_wave_f32_kernel<R_, S_, WAVES, BJ, true, KRSC, true>), grid, dim3(64 * WAVES), 0, st, a);
    else if (va)
        launch_kernel((igemm_wave_f32_kernel<R_, S_, WAVES, BJ, true, KRSC, false>), grid, dim3(64 * WAVES), 0, st, a);
    else
        launch_kernel((igemm_wave_f32_kernel<R_, S_, WAVES, BJ, false, KRSC, false>), grid, dim3(64 * WAVES), 0, st, a);
}

template <int R_, int S_, bool KRSC>
void launch_rs(const ConvArgs &a, int waves, int bj, bool va, bool pk, dim3 grid, hipStream_t st)
{
    if (waves == 8) {
        if (bj == 2) launch_va<R_, S_, 8, 2, KRSC>(a, va, pk, grid, st);
        else launch_va<R_, S_, 8, 1, KRSC>(a, va, pk, grid, st);
    } else {
        if (bj == 2) launch_va<R_, S_, 4, 2, KRSC>(a, va, pk, grid, st);
        else launch_va<R_, S_, 4, 1, KRSC>(a, va, pk, grid, st);
    }
}

int rs_template(int v) { return (v == 1 || v == 3 || v == 7) ? v : 0; }

}  // namespace

// Work-group tile 32 channels x 32*BJ pixels; a work-group runs on one CU,
// so the parallelism across CUs is the number of work-groups, and its
// wavefronts (4 or 8, splitting the tile's reduction) fill that CU's SIMDs.
// The plan minimises a latency model fitted to batch-1 ResNet-50 layers on
// this part: a fixed ~4.5 us per launch (dispatch, first loads, epilogue),
// then per round of work-groups over the CUs, each wavefront's MFMA time
// (blocks * BJ * 4 MFMAs * 64 cycles) plus ~1.2 us per dependent round of
// loads (kDepth blocks in flight), plus ~2.5 us for a split-K reduce launch.
WavePlan plan_wave_f32(const ConvProblem &p, int num_cus, bool w_aligned16)
{
    WavePlan best{};
    best.va = p.Kred % 4 == 0 && w_aligned16;
    const int blocks = ceil_div(p.Kred, 8);
    double best_us = 1e30;
    for (int bj = 1; bj <= 2; ++bj) {
        if (bj == 2 && p.M < 64) continue;
        const long tiles = (long)ceil_div(p.M, 32 * bj) * ceil_div(p.Kg, 32) * p.groups;
        const int depth = bj == 2 ? 2 : 4;
        for (int waves : {8, 4}) {
            for (int sp = 1; sp <= 16; ++sp) {
                const int per = ceil_div(blocks, sp);
                if (sp > 1 && per < 2 * waves) break;           // at least 2 blocks per wavefront
                if (ceil_div(blocks, per) != sp) continue;
                const long wgs = tiles * sp;
                const long rounds = (wgs + num_cus - 1) / num_cus;
                const int bw = ceil_div(per, waves);             // blocks per wavefront
                const double us = 4.5 + rounds * (bw * bj * 4 * 64 / 2400.0 + ceil_div(bw, depth) * 1.2) +
                                  (sp > 1 ? 2.5 : 0.0);
                if (us < best_us - 1e-9) {
                    best_us = us;
                    best.bj = bj;
                    best.waves = waves;
                    best.splits = sp;
                    best.kr_per_split = per * 8;
                }
            }
        }
    }
    best.ws_bytes = best.splits > 1 ? (size_t)best.splits * p.K * p.M * sizeof(float) : 0;
    return best;
}

void describe_wave_f32(const ConvProblem &p, const WavePlan &plan, char *buf, int len,
                       int *launches)
{
    int R = rs_template(p.R), S = rs_template(p.S);
    if (R == 0 || S == 0 || R != S) R = S = 0;
    if (plan.krsc && R != 3) R = S = 0;
    snprintf(buf, len, "igemm_wave_f32_kernel<%d, %d, %d, %d, %s, %s, %s>%s", R, S, plan.waves, plan.bj,
             (plan.va || plan.pk) ? "true" : "false", plan.krsc ? "true" : "false",
             plan.pk ? "true" : "false",
             plan.splits > 1 ? " + splitk_reduce_kernel" : "");
    *launches = plan.splits > 1 ? 2 : 1;
}

hipError_t launch_wave_f32(const ConvProblem &p, const WavePlan &plan, const float *x,
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
    const bool va = plan.va && (uintptr_t)w % 16 == 0;
    const dim3 grid((unsigned)((long)ceil_div(p.M, 32 * plan.bj) * ceil_div(p.Kg, 32) * p.groups *
                               plan.splits));
    hipError_t e = hook ? hook->before_launch(hook->ctx, st) : hipSuccess;
    if (e != hipSuccess) return e;
    if (plan.krsc) {   // filters packed KRSC (R * S > 1)
        if (p.R == 3 && p.S == 3)
            launch_rs<3, 3, true>(a, plan.waves, plan.bj, va, plan.pk, grid, st);
        else
            launch_rs<0, 0, true>(a, plan.waves, plan.bj, va, plan.pk, grid, st);
    } else if (p.R == 1 && p.S == 1) {
        launch_rs<1, 1, false>(a, plan.waves, plan.bj, va, plan.pk, grid, st);
    } else if (p.R == 3 && p.S == 3) {
        launch_rs<3, 3, false>(a, plan.waves, plan.bj, va, plan.pk, grid, st);
    } else if (p.R == 7 && p.S == 7) {
        launch_rs<7, 7, false>(a, plan.waves, plan.bj, va, plan.pk, grid, st);
    } else {
        launch_rs<0, 0, false>(a, plan.waves, plan.bj, va, plan.pk, grid, st);
    }
    e = hipGetLastError();
    if (e != hipSuccess || plan.splits == 1) return e;
    if (hook && (e = hook->before_launch(hook->ctx, st)) != hipSuccess) return e;
    return launch_splitk_reduce(a, st);
}

}  // namespace miconv
