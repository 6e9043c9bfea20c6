// Dense conv2d in fp32 as an implicit GEMM in which every wavefront feeds
// the matrix cores straight from global memory: no LDS staging and no
// barriers in the main loop.  It serves every fp32 dense layer whose tensors
// it can address with 32-bit offsets, from batch-1 ResNet layers to VGG-16
// at batch 32.
//
// Why: at batch 1 the layers of ResNet-50 / MobileNet have N*P*Q = 49..12544
// output pixels, so an LDS-staged tile kernel runs few chunks per
// work-group and spends its time waiting for one global round trip per chunk
// behind a barrier.  Here each wavefront streams its own share of the
// reduction with several blocks of loads in flight, and the parallelism the
// output tiles lack is recovered by splitting the reduction across the
// wavefronts of a work-group (combined through LDS in a fixed order) and, for
// the smallest layers, across work-groups (splitk_reduce_kernel).  At large
// batch the same structure needs no LDS reuse: an fp32 MFMA consumes one
// 4-byte operand per lane per 64 cycles, which the L1 path sustains.
//
// MFMA v_mfma_f32_32x32x2_f32, lane l of 64, half h = l / 32:
//   A operand = W[k0 + l%32][kr],  B operand = X[kr][m0 + l%32]
// The reduction is walked in blocks of 8 taps; in block b, step e (0..3),
// half h supplies tap kr = 8b + 4h + e.  The MFMA sums over both halves, so
// the 4 steps cover the block's 8 taps once, and a lane's A values for the 4
// steps are 4 consecutive floats of a packed filter row: one 16-byte load.
// Its B values are 4 gathered taps of the im2col matrix for one output
// pixel; the 32 lanes of a half read 32 consecutive pixels of the same tap.
// Output: D reg v is channel 8*(v/4) + 4*h + v%4 and pixel l%32, so every
// store writes 32 consecutive pixels (128 bytes) of one NCHW channel plane.
#include "internal.h"

#include <algorithm>
#include <cstdio>

namespace miconv {
namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));

// ok ? off : out, as one v_cndmask.  Written as a plain select, the compiler
// turns each guarded load into two branches with a load on each side.
__device__ __forceinline__ unsigned select_offset(bool ok, unsigned off, unsigned out)
{
    unsigned r;
    asm("v_cndmask_b32_e64 %0, %1, %2, %3" : "=v"(r) : "v"(out), "v"(off), "s"(__builtin_amdgcn_ballot_w64(ok)));
    return r;
}


// BJ = 32-pixel blocks per wavefront tile; ORD = reduction order of the
// packed filters: 1 = (r, s, c) with C/groups % 8 == 0, so the 4 taps of a
// half-block are 4 channels at one filter position (one padding check and
// one address per half-block); 2 = (r, s, c4), C/groups <= 4 padded to 4
// channels (the stems: a half-block is one filter position); 0 = (c, r, s).
// Filters are always read pre-packed (pack_wave_kernel): w_pk[g][k/32][kr/8]
// [lane][4] holds W[k0 + l%32][8*blk + 4*h + e], zero past K and the
// reduction, so a wavefront's A load is 1 KB contiguous.
//
// Both operands are read through buffer resources.  A tap outside the image,
// a pixel past M, a block past the split and a tap past the reduction get the
// offset kOut, which the hardware range check turns into a zero: the loads
// need no branches, which keeps the executed code short.  At batch 1 a
// launch runs a few hundred instructions per wavefront from a cold
// instruction cache, so code size is a first-order cost here.
template <int R_, int S_, int WAVES, int BJ, int ORD, bool IND, bool GEN, int KC>
__device__ __forceinline__ void wave_body(const ConvArgs &a)
{
    constexpr int kDepth = BJ == 2 ? 2 : 4;   // blocks of loads in flight per wavefront
    // Offsets at or past 2^31 bytes are out of range: the x and packed filter
    // buffers are smaller than that (checked by the planner), and adding a
    // channel stride to kOut stays below 2^32.
    constexpr unsigned kOut = 0x80000000u;
    const int R = R_ ? R_ : a.R;
    const int S = S_ ? S_ : a.S;
    const int RS = R * S;
    const __amdgpu_buffer_rsrc_t xres = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<void *>(a.x), (short)0, (int)((long)a.N * a.C * a.HW * 4), 0x00020000);
    const int kblocks = ceil_div(a.Kred, 8);
    const unsigned ktiles = ceil_div(a.Kg, 32);
    // KC: filters read as given, w[K][C/groups][R][S]; the row of filter k
    // holds its C/groups*R*S taps in (c, r, s) order.
    const int KR = a.Cg * RS;
    const __amdgpu_buffer_rsrc_t wres = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<void *>(a.w), (short)0,
        KC ? (int)((long)a.K * KR * 4) : (int)((long)a.groups * ktiles * kblocks * 1024), 0x00020000);

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int h = lane >> 5, ll = lane & 31;
    // XCD-aware tile order: the hardware deals work-groups to the 8 XCDs
    // round-robin (work-group b runs on XCD b % 8), so logical tiles are
    // renumbered to give each XCD one contiguous range, pixel tiles fastest:
    // the work-groups that read the same filter rows share an L2.
    const unsigned mtiles = ceil_div(a.M, 32 * BJ);
    const unsigned T = gridDim.x;
    const unsigned xcd = blockIdx.x % 8, jx = blockIdx.x / 8;
    const unsigned LW = xcd * (T / 8) + min(xcd, T % 8) + jx;
    // IND: every wavefront owns a tile of its own (WAVES consecutive tiles per
    // work-group) and runs its whole reduction: for short reductions over
    // many tiles, where splitting 8-tap blocks across wavefronts would leave
    // most of them idle and add an LDS combine per tile.
    const unsigned L = IND ? LW * WAVES + (threadIdx.x >> 6) : LW;
    if (IND && L >= (unsigned)(ceil_div(a.M, 32 * BJ) * ceil_div(a.Kg, 32) * a.groups)) return;
    const unsigned t1 = fdiv(L, a.dv_mt);
    const unsigned mx = L - t1 * mtiles;
    const unsigned t2 = fdiv(t1, a.dv_kt);
    const unsigned ky = t1 - t2 * ktiles;
    const int split = fdiv(t2, a.dv_g);
    const int g = t2 - split * a.groups;
    const int m0 = mx * (32 * BJ);
    const int k0 = ky * 32;
    const int kr_begin = split * a.kr_per_split;
    const int kr_end = min(a.Kred, kr_begin + a.kr_per_split);
    const int nblk = kr_end > kr_begin ? ceil_div(kr_end - kr_begin, 8) : 0;

    // A: byte offset of this lane's 16-byte slot in block 0 of the split
    // (packed filters), or of its filter row (KC; kOut past K).
    const unsigned aoff = KC ? (k0 + ll < a.Kg ? 4u * (unsigned)((g * a.Kg + k0 + ll) * KR) : kOut)
                             : ((((unsigned)g * ktiles + ky) * kblocks + kr_begin / 8) * 64 + lane) * 16;

    // B: this lane's output pixels, one per 32-pixel block.
    int ih0[BJ], iw0[BJ];
    bool mvalid[BJ];
    unsigned xoff[BJ];   // element offset of (n, channel g*Cg, 0, 0)
#pragma unroll
    for (int j = 0; j < BJ; ++j) {
        const int m = m0 + j * 32 + ll;
        mvalid[j] = m < a.M;
        const int mm = mvalid[j] ? m : 0;
        const int n = fdiv(mm, a.dv_pq);
        const int pq = mm - n * a.PQ;
        const int p = fdiv(pq, a.dv_q);
        const int q = pq - p * a.Q;
        ih0[j] = p * a.stride - a.pad;
        iw0[j] = q * a.stride - a.pad;
        xoff[j] = ((unsigned)n * a.C + (unsigned)g * a.Cg) * a.HW;
    }
    const unsigned hw4 = 4u * a.HW;   // bytes between channel planes

    struct Frag {
        float av[4];
        float bv[BJ][4];
    };

    // KRSC: the filter position of the wavefront's next block, tracked as
    // (block index) = rsq * cb + rsr with cb = C/groups / 8 blocks per filter
    // position; blocks advance by WAVES, so one division at the start.
    const int cb = a.Cg / 8;
    int rsq = 0, rsr = 0, drq = 0, drr = 0;
    if constexpr (ORD == 1 && !(R_ == 1 && S_ == 1)) {
        constexpr int kStep = IND ? 1 : WAVES;   // blocks between a wavefront's blocks
        const int b0 = kr_begin / 8 + (IND ? 0 : wave);
        rsq = fdiv(b0, a.dv_cb);
        rsr = b0 - rsq * cb;
        drq = kStep / cb;
        drr = kStep - drq * cb;
    }

    // Block blk (< nblk) of this split: taps kr_begin + 8*blk + 4h + e,
    // e = 0..3.  Called for the wavefront's blocks in increasing order.
    auto load = [&](Frag &f, int blk) {
        const int kr0 = kr_begin + 8 * blk + 4 * h;
        typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
        if constexpr (KC == 0) {
            const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(wres, aoff + blk * 1024u, 0, 0);
#pragma unroll
            for (int e = 0; e < 4; ++e) f.av[e] = __uint_as_float(v[e]);
        } else if constexpr (ORD == 0 || (ORD == 1 && R_ == 1 && S_ == 1)) {
            // the 4 taps are consecutive in the filter row
            if constexpr (KC == 1) {   // one 16-byte load (C/groups % 8 == 0, w 16-byte aligned)
                const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(wres, aoff + 4u * kr0, 0, 0);
#pragma unroll
                for (int e = 0; e < 4; ++e) f.av[e] = __uint_as_float(v[e]);
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    f.av[e] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(
                        wres, select_offset(kr0 + e < kr_end, aoff + 4u * (kr0 + e), kOut), 0, 0));
            }
        }
        if constexpr (ORD == 1) {
            // The block is one filter position (r, s) and 8 channels; the
            // reduction length is a multiple of 8, so its 4 taps per half are
            // live together and one channel stride apart.
            int c0 = kr0, r = 0, s = 0;
            if constexpr (!(R_ == 1 && S_ == 1)) {
                c0 = 8 * rsr + 4 * h;
                r = rsq / S;
                s = rsq - r * S;
                if constexpr (KC != 0) {
                    // taps (r, s) of channels c0 .. c0+3: R*S floats apart in the filter row
                    const unsigned base = aoff + 4u * (unsigned)(c0 * RS + rsq);
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        f.av[e] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(wres, base, 4 * e * RS, 0));
                }
                rsq += drq;
                rsr += drr;
                if (rsr >= cb) {
                    rsr -= cb;
                    ++rsq;
                }
            }
#pragma unroll
            for (int j = 0; j < BJ; ++j) {
                const int ih = ih0[j] + r, iw = iw0[j] + s;
                const bool ok = mvalid[j] && (unsigned)ih < (unsigned)a.H && (unsigned)iw < (unsigned)a.W;
                const unsigned off = select_offset(ok, 4u * (xoff[j] + (unsigned)c0 * a.HW + ih * a.W + iw), kOut);
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    f.bv[j][e] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(xres, off, e * hw4, 0));
            }
        } else if constexpr (ORD == 2) {
            // Half-block = filter position 2 * (block) + h, channels e < C/groups
            // (the packed filters are zero for the padding channels and past R*S).
            const int pos = 2 * (kr_begin / 8 + blk) + h;
            const int r = pos / S;
            const int s = pos - r * S;
            const bool pok = pos < RS;
            if constexpr (KC != 0) {
                // tap (r, s) of channels e < C/groups, R*S floats apart; zero past them
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    f.av[e] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(
                        wres, select_offset(pok && e < a.Cg, aoff + 4u * (unsigned)(e * RS + pos), kOut), 0, 0));
            }
#pragma unroll
            for (int j = 0; j < BJ; ++j) {
                const int ih = ih0[j] + r, iw = iw0[j] + s;
                const bool ok = pok && mvalid[j] && (unsigned)ih < (unsigned)a.H && (unsigned)iw < (unsigned)a.W;
                const unsigned base = 4u * (xoff[j] + ih * a.W + iw);
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const unsigned off = select_offset(ok && e < a.Cg, base + e * hw4, kOut);
                    f.bv[j][e] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(xres, off, 0, 0));
                }
            }
        } else if constexpr (R_ == 1 && S_ == 1) {
            // 1x1 with C/groups % 8 != 0: tap kr is channel kr at the pixel's
            // own input position; the last block of the reduction is partial.
#pragma unroll
            for (int j = 0; j < BJ; ++j) {
                const int ih = ih0[j], iw = iw0[j];
                const bool ok = mvalid[j] && (unsigned)ih < (unsigned)a.H && (unsigned)iw < (unsigned)a.W;
                const unsigned base = 4u * (xoff[j] + (unsigned)kr0 * a.HW + ih * a.W + iw);
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const unsigned off = select_offset(ok && kr0 + e < kr_end, base + e * hw4, kOut);
                    f.bv[j][e] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(xres, off, 0, 0));
                }
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
                    const bool ok = kr < kr_end && mvalid[j] && (unsigned)ih < (unsigned)a.H &&
                                    (unsigned)iw < (unsigned)a.W;
                    const unsigned off = select_offset(ok, 4u * (xoff[j] + (unsigned)c * a.HW + ih * a.W + iw), kOut);
                    f.bv[j][e] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(xres, off, 0, 0));
                }
            }
        }
    };

    // The epilogue's bias values, loaded now so that their round trip
    // overlaps the main loop (a missing bias is an empty buffer: zeros).
    constexpr int kE = IND ? 16 : BJ * 16 / WAVES;   // bias values per thread
    float bias_v[kE];
    {
        const __amdgpu_buffer_rsrc_t bres = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<float *>(a.bias), (short)0, a.bias ? a.K * 4 : 0, 0x00020000);
#pragma unroll
        for (int i = 0; i < kE; ++i) {
            // IND: the filters of the lane's own accumulator registers v = i
            const int idx = IND ? i * 64 + lane : tid + i * 64 * WAVES;
            const int v = (idx >> 6) & 15, l = idx & 63;
            const int k = k0 + 8 * (v >> 2) + 4 * (l >> 5) + (v & 3);
            bias_v[i] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(
                bres, select_offset(k < a.Kg, 4u * (g * a.Kg + k), kOut), 0, 0));
        }
    }

    floatx16 acc[BJ];
#pragma unroll
    for (int j = 0; j < BJ; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[j][v] = 0.f;

    // This wavefront takes blocks wave, wave + WAVES, ... with kDepth blocks
    // of loads in flight: pass it issues the loads of its blocks it .. it +
    // kDepth - 1 and runs the MFMAs of the previous pass's blocks.  One copy
    // of the loop body serves the whole pipeline (no separate prologue).
    const int my_blocks = IND ? nblk : nblk > wave ? ceil_div(nblk - wave, WAVES) : 0;
    Frag f[kDepth];
#pragma clang loop unroll(disable)
    for (int it = 0; it < my_blocks + kDepth; it += kDepth) {
#pragma unroll
        for (int d = 0; d < kDepth; ++d) {
            if (it >= kDepth && it - kDepth + d < my_blocks) {
#pragma unroll
                for (int e = 0; e < 4; ++e)
#pragma unroll
                    for (int j = 0; j < BJ; ++j)
                        acc[j] = __builtin_amdgcn_mfma_f32_32x32x2f32(f[d].av[e], f[d].bv[j][e], acc[j], 0, 0, 0);
            }
            if (it + d < my_blocks) load(f[d], IND ? it + d : wave + (it + d) * WAVES);
        }
    }

    if constexpr (IND) {
        // Straight from the accumulators: register v of pixel block j holds
        // pixel m0 + 32j + l%32 and filter k0 + 8(v/4) + 4(l/32) + v%4, so each
        // store writes two runs of 32 consecutive pixels.
#pragma unroll
        for (int j = 0; j < BJ; ++j) {
            const int m = m0 + j * 32 + ll;
            if (m >= a.M) continue;
            const int n = fdiv(m, a.dv_pq);
            const long yo = GEN ? (long)n * a.ysn + (long)(g * a.Kg) * a.PQ + (m - n * a.PQ)
                                 : ((long)n * a.K + g * a.Kg) * a.PQ + (m - n * a.PQ);
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int k = k0 + 8 * (v >> 2) + 4 * h + (v & 3);
                if (k >= a.Kg) continue;
                float val = acc[j][v] + bias_v[v];
                if (GEN && a.res) val += a.res[yo + (long)k * a.PQ];
                if (a.relu) val = fmaxf(val, 0.f);
                a.y[yo + (long)k * a.PQ] = val;
            }
        }
    } else {
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
#pragma unroll
        for (int i = 0; i < kE; ++i) {
            const int idx = tid + i * 64 * WAVES;
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
                const int n = fdiv(m, a.dv_pq);
                const int pq = m - n * a.PQ;
                const long yo = GEN ? (long)n * a.ysn + (long)kg * a.PQ + pq : ((long)n * a.K + kg) * a.PQ + pq;
                float val = sum + bias_v[i];
                if (GEN && a.res) val += a.res[yo];
                if (a.relu) val = fmaxf(val, 0.f);
                a.y[yo] = val;
            }
        }
    }
}

template <int R_, int S_, int WAVES, int BJ, int ORD, bool IND = false>
__global__ __launch_bounds__(64 * WAVES) void igemm_wave_f32_kernel(ConvArgs a)
{
    wave_body<R_, S_, WAVES, BJ, ORD, IND, false, 0>(a);
}

// The same kernel with the general epilogue: a residual join and/or an output
// image stride other than K*P*Q.  The plain kernel keeps the dense epilogue,
// whose few instructions matter in batch-1 layers of a few microseconds.
template <int R_, int S_, int WAVES, int BJ, int ORD, bool IND = false>
__global__ __launch_bounds__(64 * WAVES) void igemm_wave_f32_gen_kernel(ConvArgs a)
{
    wave_body<R_, S_, WAVES, BJ, ORD, IND, true, 0>(a);
}

// Filters read as given (KCRS), for calls that have no packed copy: the
// single-layer entry points, which pack nothing.  KC = 1: the 4 taps of a
// half-block are one 16-byte load (1x1, C/groups % 8 == 0, w 16-byte
// aligned); KC = 2: four 4-byte loads.  General epilogue.
template <int R_, int S_, int WAVES, int BJ, int ORD, bool IND, int KC>
__global__ __launch_bounds__(64 * WAVES) void igemm_wave_f32_kcrs_kernel(ConvArgs a)
{
    wave_body<R_, S_, WAVES, BJ, ORD, IND, true, KC>(a);
}

bool general_epilogue(const ConvArgs &a) { return a.res || a.ysn != (long)a.K * a.PQ; }

template <int R_, int S_, int WAVES, int BJ, int ORD, bool IND = false>
void launch_wave(const ConvArgs &a, int kc, dim3 grid, hipStream_t st)
{
    if (kc == 1) {
        if constexpr ((ORD == 0 || (ORD == 1 && R_ == 1 && S_ == 1)) && !IND)
            launch_kernel((igemm_wave_f32_kcrs_kernel<R_, S_, WAVES, BJ, ORD, IND, 1>), grid, dim3(64 * WAVES), 0,
                          st, a);
    } else if (kc == 2) {
        launch_kernel((igemm_wave_f32_kcrs_kernel<R_, S_, WAVES, BJ, ORD, IND, 2>), grid, dim3(64 * WAVES), 0,
                      st, a);
    } else if (general_epilogue(a)) {
        launch_kernel((igemm_wave_f32_gen_kernel<R_, S_, WAVES, BJ, ORD, IND>), grid, dim3(64 * WAVES), 0,
                      st, a);
    } else {
        launch_kernel((igemm_wave_f32_kernel<R_, S_, WAVES, BJ, ORD, IND>), grid, dim3(64 * WAVES), 0, st, a);
    }
}

template <int R_, int S_, int ORD>
void launch_rs(const ConvArgs &a, int waves, int bj, bool ind, int kc, dim3 grid, hipStream_t st)
{
    if constexpr (ORD == 2 && R_ != 7) {
        if (ind) {   // the planner takes IND with 4 wavefronts and 2 pixel blocks only
            launch_wave<R_, S_, 4, 2, ORD, true>(a, kc, grid, st);
            return;
        }
    }
    if (waves == 8) {
        if (bj == 2) launch_wave<R_, S_, 8, 2, ORD>(a, kc, grid, st);
        else launch_wave<R_, S_, 8, 1, ORD>(a, kc, grid, st);
    } else {
        if (bj == 2) launch_wave<R_, S_, 4, 2, ORD>(a, kc, grid, st);
        else launch_wave<R_, S_, 4, 1, ORD>(a, kc, grid, st);
    }
}

int rs_template(int v) { return (v == 1 || v == 3 || v == 7) ? v : 0; }

}  // namespace

// Filters read as given: the 4 taps of a half-block are consecutive in a
// filter row, and 16-byte aligned, in the (c, r, s) order and for 1x1 layers.
bool wave_kc_vector(const ConvProblem &p, const WavePlan &plan, const void *w)
{
    const bool contiguous = plan.order == 0 || (plan.order == 1 && p.R == 1 && p.S == 1);
    return contiguous && !plan.ind && p.Kred % 4 == 0 && (uintptr_t)w % 16 == 0;
}

bool wave_fits(const ConvProblem &p)
{
    return (long)p.N * p.C * p.H * p.W * 4 < (1L << 31) && (long)wave_packed_floats(p) * 4 < (1L << 31);
}

// Work-group tile 32 channels x 32*BJ pixels; a work-group runs on one CU,
// so the parallelism across CUs is the number of work-groups, and its
// wavefronts (4 or 8, splitting the tile's reduction) fill that CU's SIMDs.
// The plan minimises a latency model fitted to batch-1 ResNet-50 layers on
// this part: a fixed ~4.5 us per launch (dispatch, first loads, epilogue),
// then per round of work-groups over the CUs, each wavefront's MFMA time
// (blocks * BJ * 4 MFMAs * 64 cycles) plus ~1.2 us per dependent round of
// loads (kDepth blocks in flight), plus, for a split reduction, ~2.5 us for
// the reduce launch and the partials' HBM round trip.
WavePlan plan_wave_f32(const ConvProblem &p, int num_cus, int max_splits)
{
    WavePlan best{};
    best.order = wave_order(p);
    const int blocks = ceil_div(wave_kred(p), 8);
    double best_us = 1e30;
    for (int bj = 1; bj <= 2; ++bj) {
        if (bj == 2 && p.M < 64) continue;
        const long tiles = (long)ceil_div(p.M, 32 * bj) * ceil_div(p.Kg, 32) * p.groups;
        const int depth = bj == 2 ? 2 : 4;
        for (int waves : {4, 8}) {   // on a tie the smaller work-group: no idle wavefronts
            for (int sp = 1; sp <= std::min(16, max_splits); ++sp) {
                const int per = ceil_div(blocks, sp);
                if (sp > 1 && per < 2 * waves) break;           // at least 2 blocks per wavefront
                if (ceil_div(blocks, per) != sp) continue;
                const long wgs = tiles * sp;
                const long rounds = (wgs + num_cus - 1) / num_cus;
                const int bw = ceil_div(per, waves);             // blocks per wavefront
                // a split also writes and re-reads sp fp32 partial planes (~4 TB/s)
                const double us = 4.5 + rounds * (bw * bj * 4 * 64 / 2400.0 + ceil_div(bw, depth) * 1.2) +
                                  (sp > 1 ? 2.5 + 2.0 * sp * p.K * (double)p.M * 4 / 4.0e6 : 0.0);
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
    // Short reductions (C <= 4 channels, 3x3: at most 8 blocks of 8 taps)
    // over many tiles: one tile per wavefront (VGG-16's first layer at batch 8,
    // 12544 tiles of 64 pixels x 32 filters: the split across wavefronts left
    // 3 of 8 idle and paid an LDS combine per 5 blocks).
    const long tiles2 = (long)ceil_div(p.M, 64) * ceil_div(p.Kg, 32) * p.groups;
    if (best.order == 2 && p.R != 7 && blocks <= 8 && p.M >= 64 && tiles2 >= 16L * num_cus) {
        best.ind = true;
        best.waves = 4;
        best.bj = 2;
        best.splits = 1;
        best.kr_per_split = blocks * 8;
    }
    best.ws_bytes = best.splits > 1 ? (size_t)best.splits * p.K * p.M * sizeof(float) : 0;
    return best;
}

void describe_wave_f32(const ConvProblem &p, const WavePlan &plan, char *buf, int len,
                       int *launches)
{
    int R = rs_template(p.R), S = rs_template(p.S);
    if (R == 0 || S == 0 || R != S) R = S = 0;
    if ((plan.order == 0 || plan.order == 1) && R != 3 && R != 1) R = S = 0;
    if (plan.order == 2 && R != 3 && R != 7) R = S = 0;
    const bool gen = p.res || p.ysn != (long)p.K * p.P * p.Q;
    if (plan.kc) {
        // the 16-byte filter loads need w 16-byte aligned: named as for an aligned w
        alignas(16) static const float stand_in[4] = {};
        const int kc = wave_kc_vector(p, plan, stand_in) ? 1 : 2;
        snprintf(buf, len, "igemm_wave_f32_kcrs_kernel<%d, %d, %d, %d, %d, %s, %d>%s", R, S, plan.waves,
                 plan.bj, plan.order, plan.ind ? "true" : "false", kc,
                 plan.splits > 1 ? " + splitk_reduce_kernel" : "");
    } else {
        snprintf(buf, len, "igemm_wave_f32%s_kernel<%d, %d, %d, %d, %d, %s>%s", gen ? "_gen" : "", R, S,
                 plan.waves, plan.bj, plan.order, plan.ind ? "true" : "false",
                 plan.splits > 1 ? " + splitk_reduce_kernel" : "");
    }
    *launches = plan.splits > 1 ? 2 : 1;
}

hipError_t launch_wave_f32(const ConvProblem &p, const WavePlan &plan, const float *x,
                           const float *w, const float *bias, float *y, float *ws,
                           hipStream_t st, const LaunchHook *hook)
{
    // filters as given: one 16-byte load per half-block where the 4 taps are
    // consecutive and aligned (1x1, C/groups % 8 == 0), else four 4-byte loads
    const int kc = !plan.kc ? 0 : wave_kc_vector(p, plan, w) ? 1 : 2;
    ConvArgs a = make_args(p);
    a.x = x;
    a.w = w;
    a.bias = bias;
    a.y = y;
    a.ws = plan.splits > 1 ? ws : nullptr;
    a.splits = plan.splits;
    a.kr_per_split = plan.kr_per_split;
    a.Kred = wave_kred(p);   // the packed reduction (padded channel quads for order 2)
    a.dv_mt = make_fastdiv(ceil_div(p.M, 32 * plan.bj));
    a.dv_kt = make_fastdiv(ceil_div(p.Kg, 32));
    a.dv_g = make_fastdiv(p.groups);
    a.dv_cb = make_fastdiv(p.Cg / 8 > 0 ? p.Cg / 8 : 1);
    const long tiles = (long)ceil_div(p.M, 32 * plan.bj) * ceil_div(p.Kg, 32) * p.groups * plan.splits;
    if (plan.ind && (plan.order != 2 || p.R == 7 || plan.waves != 4 || plan.bj != 2 || plan.splits != 1))
        return hipErrorInvalidValue;
    const dim3 grid((unsigned)(plan.ind ? (tiles + plan.waves - 1) / plan.waves : tiles));
    hipError_t e = hook ? hook->before_launch(hook->ctx, st) : hipSuccess;
    if (e != hipSuccess) return e;
    if (plan.order == 1) {   // reduction ordered (r, s, c) in the packed filters
        if (p.R == 1 && p.S == 1)
            launch_rs<1, 1, 1>(a, plan.waves, plan.bj, plan.ind, kc, grid, st);
        else if (p.R == 3 && p.S == 3)
            launch_rs<3, 3, 1>(a, plan.waves, plan.bj, plan.ind, kc, grid, st);
        else
            launch_rs<0, 0, 1>(a, plan.waves, plan.bj, plan.ind, kc, grid, st);
    } else if (plan.order == 2) {   // (r, s, c4): C/groups <= 4
        if (p.R == 3 && p.S == 3)
            launch_rs<3, 3, 2>(a, plan.waves, plan.bj, plan.ind, kc, grid, st);
        else if (p.R == 7 && p.S == 7)
            launch_rs<7, 7, 2>(a, plan.waves, plan.bj, plan.ind, kc, grid, st);
        else
            launch_rs<0, 0, 2>(a, plan.waves, plan.bj, plan.ind, kc, grid, st);
    } else if (p.R == 1 && p.S == 1) {
        launch_rs<1, 1, 0>(a, plan.waves, plan.bj, plan.ind, kc, grid, st);
    } else if (p.R == 3 && p.S == 3) {
        launch_rs<3, 3, 0>(a, plan.waves, plan.bj, plan.ind, kc, grid, st);
    } else {
        launch_rs<0, 0, 0>(a, plan.waves, plan.bj, plan.ind, kc, grid, st);
    }
    e = hipGetLastError();
    if (e != hipSuccess || plan.splits == 1) return e;
    if (hook && (e = hook->before_launch(hook->ctx, st)) != hipSuccess) return e;
    return launch_splitk_reduce(a, st);
}

}  // namespace miconv
