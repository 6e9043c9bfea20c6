// Depthwise convolution (groups == C == K): MobileNet's per-channel 3x3 filter.
//
// The operator does 9 FMAs per 8 bytes of HBM traffic, so it is bound by HBM
// bandwidth.  The fast kernel reads every input element from HBM once and
// writes every output once, with wide contiguous accesses:
//
//  * A wavefront is cut into lane groups of G lanes.  A group owns one row
//    segment of one (n, c) plane and a strip of T output rows.  Lane j of a
//    group owns V consecutive outputs of a row (V = 4, 2 or 1), so its loads
//    and stores are V-wide vectors.
//  * Horizontal taps come from the neighbouring lanes through cross-lane
//    shuffles instead of being re-read; only the two lanes at the ends of a
//    group fetch their halo element themselves (zero outside the image).
//  * Vertical taps come from a rolling window of input rows held in
//    registers while the group walks down its strip: stride 1 loads one new
//    input row per output row, stride 2 loads two.
//
// Square planes up to 56x56 use the whole-plane run kernel below instead,
// which streams contiguous runs of planes through LDS; other depthwise shapes
// (filters up to 7x7, any stride and pad) use a plain one-output-per-lane
// kernel.
#include "internal.h"

#include <cstdio>

namespace miconv {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));


template <int V> struct VecT;
template <> struct VecT<1> { typedef float type; };
template <> struct VecT<2> { typedef float2 type; };
template <> struct VecT<4> { typedef float4 type; };
template <> struct VecT<8> { typedef float4 type; };  // two float4 loads

template <int V>
__device__ inline void load_vec(const float *p, float *out)
{
    if constexpr (V == 8) {
        load_vec<4>(p, out);
        load_vec<4>(p + 4, out + 4);
    } else {
        typedef typename VecT<V>::type T;
        T v = *reinterpret_cast<const T *>(p);
        const float *f = reinterpret_cast<const float *>(&v);
#pragma unroll
        for (int i = 0; i < V; ++i) out[i] = f[i];
    }
}

template <int V>
__device__ inline void store_vec(float *p, const float *in)
{
    typedef typename VecT<V>::type T;
    T v;
    float *f = reinterpret_cast<float *>(&v);
#pragma unroll
    for (int i = 0; i < V; ++i) f[i] = in[i];
    *reinterpret_cast<T *>(p) = v;
}

struct DwArgs {
    const float *x, *w, *bias;
    float *y;
    int C, H, W, P, Q;
    int G;          // lanes per group
    int seg_w;      // output columns per row segment (V * G)
    int nseg;       // row segments per plane
    int T;          // output rows per strip
    int nstrip;     // strips per plane
    long items;     // planes * nseg * nstrip
    int relu;
};

// 3x3 depthwise with pad 1, stride ST (1 or 2), V outputs per lane.
template <int ST, int V>
__global__ __launch_bounds__(256) void dw3x3_kernel(DwArgs a)
{
    constexpr int NLD = ST * V;                       // input columns a lane owns per row
    constexpr int NIN = NLD + (ST == 1 ? 2 : 1);      // + halo taps
    const int lane = threadIdx.x & 63;
    const int G = a.G;
    const int gpw = 64 / G;
    const int gi = lane / G;
    const int j = lane - gi * G;
    const long wave = ((long)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
    const long item = wave * gpw + gi;
    const bool live = (gi < gpw) && (item < a.items);
    const long it = live ? item : 0;

    const int strip = (int)(it % a.nstrip);
    const long t1 = it / a.nstrip;
    const int seg = (int)(t1 % a.nseg);
    const long plane = t1 / a.nseg;
    const int ch = (int)(plane % a.C);

    const int q0 = seg * a.seg_w + j * V;             // first output column of this lane
    const bool qlive = live && q0 < a.Q;              // Q % V == 0, so all V outputs exist
    const int col0 = q0 * ST;                         // first owned input column
    const float *xp = a.x + plane * (long)a.H * a.W;
    float *yp = a.y + plane * (long)a.P * a.Q;

    float wt[9];
#pragma unroll
    for (int i = 0; i < 9; ++i) wt[i] = a.w[ch * 9 + i];
    const float b0 = a.bias ? a.bias[ch] : 0.f;

    const int src_l = lane > 0 ? lane - 1 : 0;
    const int src_r = lane < 63 ? lane + 1 : 63;

    // One input row as seen by this lane: [left halo, owned..., (right halo)].
    auto load_row = [&](int h, float *row) {
        const bool hv = (unsigned)h < (unsigned)a.H;
        float own[NLD];
        if (qlive && hv) {
            load_vec<NLD>(xp + (long)h * a.W + col0, own);
        } else {
#pragma unroll
            for (int i = 0; i < NLD; ++i) own[i] = 0.f;
        }
        const float from_l = __shfl(own[NLD - 1], src_l, 64);
        float left;
        if (j == 0) {
            const int cl = col0 - 1;
            left = (qlive && hv && cl >= 0) ? xp[(long)h * a.W + cl] : 0.f;
        } else {
            left = from_l;
        }
        row[0] = left;
#pragma unroll
        for (int i = 0; i < NLD; ++i) row[1 + i] = own[i];
        if constexpr (ST == 1) {
            const float from_r = __shfl(own[0], src_r, 64);
            float right;
            if (j == G - 1) {
                const int cr = col0 + NLD;
                right = (qlive && hv && cr < a.W) ? xp[(long)h * a.W + cr] : 0.f;
            } else {
                right = from_r;
            }
            row[NIN - 1] = right;
        }
    };

    auto emit = [&](int p, const float *r0, const float *r1, const float *r2) {
        float out[V];
#pragma unroll
        for (int v = 0; v < V; ++v) {
            float acc = b0;
#pragma unroll
            for (int s = 0; s < 3; ++s) acc = fmaf(r0[v * ST + s], wt[0 * 3 + s], acc);
#pragma unroll
            for (int s = 0; s < 3; ++s) acc = fmaf(r1[v * ST + s], wt[1 * 3 + s], acc);
#pragma unroll
            for (int s = 0; s < 3; ++s) acc = fmaf(r2[v * ST + s], wt[2 * 3 + s], acc);
            out[v] = a.relu ? fmaxf(acc, 0.f) : acc;
        }
        if (qlive && p < a.P) store_vec<V>(yp + (long)p * a.Q + q0, out);
    };

    const int p0 = strip * a.T;
    float ra[NIN], rb[NIN], rc[NIN];
    if constexpr (ST == 1) {
        load_row(p0 - 1, ra);
        load_row(p0, rb);
        for (int t = 0; t < a.T; ++t) {
            const int p = p0 + t;
            load_row(p + 1, rc);
            emit(p, ra, rb, rc);
#pragma unroll
            for (int i = 0; i < NIN; ++i) { ra[i] = rb[i]; rb[i] = rc[i]; }
        }
    } else {
        load_row(2 * p0 - 1, ra);
        for (int t = 0; t < a.T; ++t) {
            const int p = p0 + t;
            load_row(2 * p, rb);
            load_row(2 * p + 1, rc);
            emit(p, ra, rb, rc);
#pragma unroll
            for (int i = 0; i < NIN; ++i) ra[i] = rc[i];
        }
    }
}

// Planes up to 56x56 (3x3, pad 1): a work-group takes runs of PB whole
// consecutive (n, c) planes -- in NCHW one contiguous stretch of PB*H*W
// inputs -- and reads each run from HBM once with 16-byte loads.  The run is
// laid out in LDS with a zero gap of at least W+1 floats before and after
// every plane, so taps above the first row and below the last row read zeros
// without a test; only the left and right image borders need a mask.  The
// plane extents are compile-time constants, so the lanes' index arithmetic
// is multiplies and shifts.  A lane computes a column of several output rows
// at one position, reading each input row once for all of them; neighbouring
// lanes take neighbouring columns, so LDS reads are conflict-free (stride 1)
// and each output store of a wavefront covers whole row segments.  While the
// lanes compute run i from LDS, the loads of the work-group's next run are
// already in flight into registers.
struct DwRunArgs {
    const float *x, *w, *bias;
    float *y;
    int C;
    long planes;
    int PB;          // planes per run
    long runs;
    int relu;
};

constexpr int kRunLds = 9728;                       // floats of LDS per work-group (38 KB)
constexpr int kTapStride = 12;                      // per plane in LDS: 9 taps, bias, 2 unused

template <int H_, int W_, int ST>
struct DwRunShape {
    static constexpr int P = (H_ - 1) / ST + 1;     // 3x3, pad 1
    static constexpr int Q = (W_ - 1) / ST + 1;
    static constexpr int HW = H_ * W_;
    static constexpr int PQ = P * Q;
    static constexpr int G0 = (W_ + 1 + 3) / 4 * 4;                     // gap before plane 0
    // Stride-1 planes up to 14x14 take whole output columns as work items
    // (item = plane * Q + column), so a wavefront's LDS reads of one input row
    // sit at plane * PP + column: with PP = Q (mod 64 banks) they are 64
    // consecutive banks, conflict-free.  Other shapes pad the pitch to 4.
    static constexpr bool WHOLE = ST == 1 && P <= 14;
    static constexpr int PP_MIN = HW + W_ + 1;
    static constexpr int PP = WHOLE ? PP_MIN + (((Q - PP_MIN) % 64) + 64) % 64 : (PP_MIN + 3) / 4 * 4;
    static constexpr int PUTV = HW % 4 == 0 ? (PP % 4 == 0 ? 4 : (PP % 2 == 0 ? 2 : 1)) : 1;
    static constexpr bool RIGHT_MASK = (Q - 1) * ST + 1 >= W_;         // a right tap can leave the image
    // float4 per lane staged per run (odd planes scatter element-wise and
    // take more registers, so they stage less)
    static constexpr int STAGE4 = HW % 4 == 0 ? 7 : 5;
    static constexpr int STAGE_FLOATS = STAGE4 * 4 * 256;
    // Planes of at most 14 output columns (28 at stride 1) also keep an output
    // region in LDS: items write their columns there and the run's outputs,
    // one contiguous stretch of y, leave with consecutive lanes on
    // consecutive floats.  (Stored straight from the items, a store
    // instruction would write column pieces of many small planes: short,
    // scattered segments.  At 56x56 stride 2 the direct stores measured
    // faster.)
    static constexpr bool OUT_LDS = Q <= 14 || (ST == 1 && Q <= 28);
    static constexpr int MAX_PB_LDS = (kRunLds - G0 - 3) / (PP + kTapStride + (OUT_LDS ? PQ : 0));
    static constexpr int MAX_PB = STAGE_FLOATS / HW < MAX_PB_LDS ? STAGE_FLOATS / HW : MAX_PB_LDS;
    static constexpr int NW = (MAX_PB * kTapStride + 255) / 256;       // tap words staged per lane
    // A lane's work item is a column of RG output rows of one plane: the
    // (RG-1)*ST+3 input rows it reads feed all RG outputs, so each input
    // element is read from LDS about once per item instead of 9 times.
    static constexpr int RG = WHOLE ? P : (P % 7 == 0 ? 7 : P);
    static constexpr int NG = P / RG;                                  // row groups per plane
    static constexpr int IPP = NG * Q;                                 // items per plane
    static_assert(P % RG == 0, "row groups tile the plane");
};

// Planes per run for a shape.  Runs are as large as the register stage and
// LDS allow, then evened out so that the run count is a whole multiple of the
// grid (`grid` work-groups, one run each per round): no round ends with part
// of the chip idle.  0 if one plane does not fit.
template <int H_, int W_, int ST>
int dw_run_planes_for(long planes, long grid)
{
    using S = DwRunShape<H_, W_, ST>;
    const int align = S::HW % 4 == 0 ? 1 : (S::HW % 2 == 0 ? 2 : 4);  // PB*HW % 4 == 0
    long pbmax = S::MAX_PB;
    // A run whose items fill the 256 lanes k times plus a small remainder
    // costs k + 1 passes: trim it to k whole passes.
    const long items = pbmax * S::IPP;
    if (items >= 256 && items % 256 < 128) pbmax = items / 256 * 256 / S::IPP;
    pbmax = pbmax / align * align;
    if (pbmax < align) return 0;
    long rounds = (planes + pbmax * grid - 1) / (pbmax * grid);
    long pb;
    for (;; ++rounds) {
        pb = (planes + rounds * grid - 1) / (rounds * grid);
        pb = (pb + align - 1) / align * align;
        if (pb <= pbmax) break;
    }
    return (int)pb;
}

template <int H_, int W_, int ST>
__global__ __launch_bounds__(256, 4) void dw_run_kernel(DwRunArgs a)
{
    using S = DwRunShape<H_, W_, ST>;
    __shared__ __attribute__((aligned(16))) float lds[kRunLds];
    const int tid = threadIdx.x;
    float *taps = lds + ((S::G0 + a.PB * S::PP + 3) & ~3);      // 16-byte aligned
    float *outs = taps + a.PB * kTapStride;                      // OUT_LDS: [plane][P][Q]

    // The gaps are written here once and never again: runs only write plane slots.
    for (int i = tid; i < kRunLds / 4; i += 256)
        reinterpret_cast<float4 *>(lds)[i] = make_float4(0.f, 0.f, 0.f, 0.f);

    float4 stage[S::STAGE4];
    constexpr int kW = S::NW;
    float wstage[kW];
    float tail = 0.f;
    int c4 = 0, cnt = 0, wcnt = 0;
    long sp0 = 0;          // first plane of the staged run

    auto load = [&](long run) {
        sp0 = run * a.PB;
        const int np = run < a.runs ? (int)min((long)a.PB, a.planes - sp0) : 0;
        cnt = np * S::HW;
        c4 = cnt / 4;
        wcnt = np * kTapStride;
        const float4 *src = reinterpret_cast<const float4 *>(a.x + sp0 * S::HW);
        const int c0 = (int)(sp0 % a.C);            // channel of the run's first plane (uniform)
#pragma unroll
        for (int i = 0; i < S::STAGE4; ++i) {
            const int j = tid + i * 256;
            stage[i] = j < c4 ? src[j] : make_float4(0.f, 0.f, 0.f, 0.f);
        }
        // The last run of an odd-sized tensor ends inside a float4: at most 3 lanes.
        const int tj = 4 * c4 + tid;
        tail = tj < cnt ? a.x[sp0 * S::HW + tj] : 0.f;
#pragma unroll
        for (int i = 0; i < kW; ++i) {
            const int j = tid + i * 256;             // j = plane * kTapStride + tap
            const int pl = j / kTapStride, t = j - pl * kTapStride;
            float v = 0.f;
            if (j < wcnt) {
                const int c = (c0 + pl) % a.C;
                v = t < 9 ? a.w[c * 9 + t] : (t == 9 && a.bias ? a.bias[c] : 0.f);
            }
            wstage[i] = v;
        }
    };
    // Staged inputs -> their plane slots in LDS.
    auto put = [&]() {
#pragma unroll
        for (int i = 0; i < S::STAGE4; ++i) {
            const int j4 = tid + i * 256;
            if (j4 < c4) {
                const int j = 4 * j4;
                if constexpr (S::PUTV == 4) {
                    const int pl = j / S::HW;
                    *reinterpret_cast<float4 *>(lds + S::G0 + pl * S::PP + (j - pl * S::HW)) =
                        stage[i];
                } else if constexpr (S::PUTV == 2) {
                    const int pl = j / S::HW;
                    float2 *d = reinterpret_cast<float2 *>(lds + S::G0 + pl * S::PP + (j - pl * S::HW));
                    d[0] = make_float2(stage[i].x, stage[i].y);
                    d[1] = make_float2(stage[i].z, stage[i].w);
                } else {
                    // a vector may cross into the next plane (at most once: HW >= 4)
                    const float e[4] = {stage[i].x, stage[i].y, stage[i].z, stage[i].w};
                    const int pl = j / S::HW;
                    const int off = j - pl * S::HW;
                    float *d = lds + S::G0 + pl * S::PP + off;
#pragma unroll
                    for (int k = 0; k < 4; ++k) d[k + (off + k >= S::HW ? S::PP - S::HW : 0)] = e[k];
                }
            }
        }
        const int tj = 4 * c4 + tid;
        if (tj < cnt) {
            const int pl = tj / S::HW;
            lds[S::G0 + pl * S::PP + (tj - pl * S::HW)] = tail;
        }
#pragma unroll
        for (int i = 0; i < kW; ++i)
            if (tid + i * 256 < wcnt) taps[tid + i * 256] = wstage[i];
    };

    long run = blockIdx.x;
    __syncthreads();
    load(run);
    put();
    for (; run < a.runs; run += gridDim.x) {
        const long plane0 = sp0;
        load(run + gridDim.x);                      // in flight while this run computes
        __syncthreads();
        const int np = (int)min((long)a.PB, a.planes - plane0);
        const int icnt = np * S::IPP;
        float *dst = a.y + plane0 * S::PQ;
        constexpr int NR = (S::RG - 1) * ST + 3;   // input rows an item reads
        for (int it = tid; it < icnt; it += 256) {
            const int pl = it / S::IPP;
            const int rem = it - pl * S::IPP;
            const int g = rem / S::Q;
            const int q = rem - g * S::Q;
            const int p0 = g * S::RG;
            // input row p0*ST - 1 (a zero gap row for the first group), column q*ST
            const float *xb = lds + S::G0 + pl * S::PP + (p0 * ST - 1) * W_ + q * ST;
            const float4 *tq = reinterpret_cast<const float4 *>(taps + pl * kTapStride);
            const float4 t0 = tq[0], t1 = tq[1], t2 = tq[2];
            const float wt[9] = {t0.x, t0.y, t0.z, t0.w, t1.x, t1.y, t1.z, t1.w, t2.x};
            const bool lok = q != 0;
            const bool rok = !S::RIGHT_MASK || q * ST + 1 < W_;
            float acc[S::RG];
#pragma unroll
            for (int j = 0; j < S::RG; ++j) acc[j] = t2.y;
#pragma unroll
            for (int rr = 0; rr < NR; ++rr) {
                const float *row = xb + rr * W_;
                const float v0 = lok ? row[-1] : 0.f;
                const float v1 = row[0];
                const float v2 = rok ? row[1] : 0.f;
                // input row rr meets output row j through filter row rr - j*ST
#pragma unroll
                for (int j = 0; j < S::RG; ++j) {
                    const int r = rr - j * ST;
                    if (r >= 0 && r < 3) {
                        acc[j] = fmaf(v0, wt[r * 3 + 0], acc[j]);
                        acc[j] = fmaf(v1, wt[r * 3 + 1], acc[j]);
                        acc[j] = fmaf(v2, wt[r * 3 + 2], acc[j]);
                    }
                }
            }
            float *yo = (S::OUT_LDS ? outs : dst) + pl * S::PQ + p0 * S::Q + q;
#pragma unroll
            for (int j = 0; j < S::RG; ++j) yo[j * S::Q] = a.relu ? fmaxf(acc[j], 0.f) : acc[j];
        }
        if constexpr (S::OUT_LDS) {
            __syncthreads();
            const int ocnt = np * S::PQ;
            if (((uintptr_t)dst & 15) == 0) {          // outs is 16-byte aligned
                for (int i = tid; i < ocnt / 4; i += 256)
                    __builtin_nontemporal_store(reinterpret_cast<const f32x4 *>(outs)[i],
                                                reinterpret_cast<f32x4 *>(dst) + i);
                for (int i = ocnt / 4 * 4 + tid; i < ocnt; i += 256) dst[i] = outs[i];
            } else {
                for (int i = tid; i < ocnt; i += 256) dst[i] = outs[i];
            }
        }
        __syncthreads();                            // LDS free for the next run
        put();
    }
}

// Planes too large for one run (112x112): a run is a band of BR output rows
// of one plane.  Its input rows, halo rows included, are one contiguous
// stretch of the plane, staged into LDS as in the whole-plane kernel; halo
// rows outside the image are staged as zeros.  Neighbouring bands share two
// (stride 1) or one (stride 2) input rows, so the input is read 1 + 2/BR
// (1 + 1/(2*BR)) times.
template <int H_, int W_, int ST, int BR>
struct DwBandShape {
    static constexpr int P = (H_ - 1) / ST + 1;
    static constexpr int Q = (W_ - 1) / ST + 1;
    static constexpr int NB = P / BR;                                  // bands per plane
    static constexpr int NRB = (BR - 1) * ST + 3;                      // input rows of a band
    static constexpr int ROW0 = 4;                                     // LDS offset of the band's first row
    static constexpr int STAGE4 = (NRB * W_ / 4 + 255) / 256;
    static constexpr int RG = 7;
    static constexpr int IPB = BR / RG * Q;                            // items per band
    static constexpr bool RIGHT_MASK = (Q - 1) * ST + 1 >= W_;
    static_assert(P % BR == 0 && BR % RG == 0 && W_ % 4 == 0, "band tiling");
    static_assert(ROW0 + NRB * W_ + 4 + kTapStride <= kRunLds, "band fits in LDS");
};

template <int H_, int W_, int ST, int BR>
__global__ __launch_bounds__(256, 4) void dw_band_kernel(DwRunArgs a)
{
    using S = DwBandShape<H_, W_, ST, BR>;
    __shared__ __attribute__((aligned(16))) float lds[kRunLds];
    float *taps = lds + kRunLds - kTapStride;      // 16-byte aligned
    const int tid = threadIdx.x;
    constexpr int NF4 = S::NRB * W_ / 4;           // float4 of a band
    float4 stage[S::STAGE4];
    float wst = 0.f;
    long splane = 0;
    int sband = 0;
    bool slive = false;

    auto load = [&](long run) {
        slive = run < a.runs;
        splane = run / S::NB;
        sband = (int)(run - splane * S::NB);
        const int h0 = sband * BR * ST - 1;        // first input row of the band
        const float *xp = a.x + splane * (H_ * W_);
#pragma unroll
        for (int i = 0; i < S::STAGE4; ++i) {
            const int j = tid + i * 256;
            const int h = h0 + (4 * j) / W_;
            float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
            if (slive && j < NF4 && h >= 0 && h < H_)
                v = *reinterpret_cast<const float4 *>(xp + (long)h0 * W_ + 4 * j);
            stage[i] = v;
        }
        if (slive && tid < kTapStride) {
            const int c = (int)(splane % a.C);
            wst = tid < 9 ? a.w[c * 9 + tid] : (tid == 9 && a.bias ? a.bias[c] : 0.f);
        }
    };
    auto put = [&]() {
#pragma unroll
        for (int i = 0; i < S::STAGE4; ++i) {
            const int j = tid + i * 256;
            if (j < NF4) *reinterpret_cast<float4 *>(lds + S::ROW0 + 4 * j) = stage[i];
        }
        if (tid < kTapStride) taps[tid] = wst;
    };

    long run = blockIdx.x;
    load(run);
    put();
    for (; run < a.runs; run += gridDim.x) {
        const long plane = splane;
        const int band = sband;
        load(run + gridDim.x);                      // in flight while this band computes
        __syncthreads();
        const float4 t0 = reinterpret_cast<const float4 *>(taps)[0];
        const float4 t1 = reinterpret_cast<const float4 *>(taps)[1];
        const float4 t2 = reinterpret_cast<const float4 *>(taps)[2];
        const float wt[9] = {t0.x, t0.y, t0.z, t0.w, t1.x, t1.y, t1.z, t1.w, t2.x};
        float *dst = a.y + plane * (S::P * S::Q) + (long)band * BR * S::Q;
        constexpr int NR = (S::RG - 1) * ST + 3;
        for (int it = tid; it < S::IPB; it += 256) {
            const int g = it / S::Q;
            const int q = it - g * S::Q;
            const int p0 = g * S::RG;                       // output row within the band
            const float *xb = lds + S::ROW0 + p0 * ST * W_ + q * ST;
            const bool lok = q != 0;
            const bool rok = !S::RIGHT_MASK || q * ST + 1 < W_;
            float acc[S::RG];
#pragma unroll
            for (int j = 0; j < S::RG; ++j) acc[j] = t2.y;
#pragma unroll
            for (int rr = 0; rr < NR; ++rr) {
                const float *row = xb + rr * W_;
                const float v0 = lok ? row[-1] : 0.f;
                const float v1 = row[0];
                const float v2 = rok ? row[1] : 0.f;
#pragma unroll
                for (int j = 0; j < S::RG; ++j) {
                    const int r = rr - j * ST;
                    if (r >= 0 && r < 3) {
                        acc[j] = fmaf(v0, wt[r * 3 + 0], acc[j]);
                        acc[j] = fmaf(v1, wt[r * 3 + 1], acc[j]);
                        acc[j] = fmaf(v2, wt[r * 3 + 2], acc[j]);
                    }
                }
            }
            float *yo = dst + p0 * S::Q + q;
#pragma unroll
            for (int j = 0; j < S::RG; ++j) __builtin_nontemporal_store(a.relu ? fmaxf(acc[j], 0.f) : acc[j], &yo[j * S::Q]);
        }
        __syncthreads();
        put();
    }
}

// Any depthwise shape: one output per lane, taps read through the caches.
__global__ __launch_bounds__(256) void dw_generic_kernel(const float *__restrict__ x,
                                                         const float *__restrict__ w,
                                                         const float *__restrict__ bias,
                                                         float *__restrict__ y, int C, int H,
                                                         int W, int R, int S, int stride,
                                                         int pad, int P, int Q, long total,
                                                         int relu)
{
    for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += (long)gridDim.x * blockDim.x) {
        const int q = (int)(i % Q);
        const long t = i / Q;
        const int p = (int)(t % P);
        const long plane = t / P;
        const int ch = (int)(plane % C);
        const float *xp = x + plane * (long)H * W;
        const float *wp = w + (long)ch * R * S;
        float acc = bias ? bias[ch] : 0.f;
        for (int r = 0; r < R; ++r) {
            const int h = p * stride - pad + r;
            if ((unsigned)h >= (unsigned)H) continue;
            for (int s = 0; s < S; ++s) {
                const int ww = q * stride - pad + s;
                if ((unsigned)ww >= (unsigned)W) continue;
                acc = fmaf(xp[(long)h * W + ww], wp[r * S + s], acc);
            }
        }
        y[i] = relu ? fmaxf(acc, 0.f) : acc;
    }
}

template <int ST, int V>
hipError_t launch_fast(DwArgs a, hipStream_t st)
{
    const long gpw = 64 / a.G;
    const long waves = (a.items + gpw - 1) / gpw;
    const long blocks = (waves + 3) / 4;
    launch_kernel((dw3x3_kernel<ST, V>), dim3((unsigned)blocks), dim3(256), 0, st, a);
    return hipGetLastError();
}

bool aligned(const void *p, size_t bytes) { return ((uintptr_t)p % bytes) == 0; }

}  // namespace

// Lanes' output width V for the 3x3 pad-1 fast kernel, or 0 for the generic one.
int dw_vector_width(const ConvProblem &p, const void *x, const void *y)
{
    const bool fast_shape = p.R == 3 && p.S == 3 && p.pad == 1 && (p.stride == 1 || p.stride == 2);
    if (!fast_shape) return 0;
    for (int v : {4, 2, 1}) {
        const int nld = p.stride * v;
        if (p.Q % v == 0 && p.W % nld == 0 && p.W >= nld && aligned(x, 4 * nld) &&
            aligned(y, 4 * v) && (p.stride == 1 ? p.W == p.Q : p.W == 2 * p.Q))
            return v;
    }
    return 0;
}

// Planes per run for the whole-plane kernel (0: not eligible): 3x3 pad 1
// filters, stride 1 or 2, on the square plane sizes it is built for, with a
// 16-byte aligned input.  The grid is four work-groups per compute unit.
int dw_run_planes(const ConvProblem &p, const void *x, int cus)
{
    if (p.R != 3 || p.S != 3 || p.pad != 1 || (p.stride != 1 && p.stride != 2) || p.H != p.W) return 0;
    if (x && !aligned(x, 16)) return 0;
    const long planes = (long)p.N * p.C;
    const long grid = 4L * cus;
    const bool s1 = p.stride == 1;
    switch (p.H) {
    case 7: return s1 ? dw_run_planes_for<7, 7, 1>(planes, grid) : dw_run_planes_for<7, 7, 2>(planes, grid);
    case 14: return s1 ? dw_run_planes_for<14, 14, 1>(planes, grid) : dw_run_planes_for<14, 14, 2>(planes, grid);
    case 28: return s1 ? dw_run_planes_for<28, 28, 1>(planes, grid) : dw_run_planes_for<28, 28, 2>(planes, grid);
    case 56: return s1 ? dw_run_planes_for<56, 56, 1>(planes, grid) : dw_run_planes_for<56, 56, 2>(planes, grid);
    default: return 0;
    }
}

// Bands per launch for the 112x112 band kernel (0: not eligible).  Used
// when there are at least as many bands as the grid has work-groups; fewer
// (small batches) go to the lane-group kernel.
constexpr int kBandRows1 = 56, kBandRows2 = 28;      // output rows per band, stride 1 / 2

long dw_band_runs(const ConvProblem &p, const void *x, int cus)
{
    if (p.R != 3 || p.S != 3 || p.pad != 1 || (p.stride != 1 && p.stride != 2) || p.H != 112 ||
        p.W != 112)
        return 0;
    if (x && !aligned(x, 16)) return 0;
    const long runs = (long)p.N * p.C * (p.P / (p.stride == 1 ? kBandRows1 : kBandRows2));
    return runs >= 4L * cus ? runs : 0;
}

void describe_dwconv(const ConvProblem &p, char *buf, int len, int *launches)
{
    const int V = dw_vector_width(p, nullptr, nullptr);
    if (dw_run_planes(p, nullptr, 256) > 0)
        snprintf(buf, len, "dw_run_kernel<%d, %d, %d>", p.H, p.W, p.stride);
    else if (dw_band_runs(p, nullptr, 256) > 0)
        snprintf(buf, len, "dw_band_kernel<%d, %d, %d, %d>", p.H, p.W, p.stride,
                 p.stride == 1 ? kBandRows1 : kBandRows2);
    else if (V)
        snprintf(buf, len, "dw3x3_kernel<%d, %d>", p.stride, V);
    else
        snprintf(buf, len, "dw_generic_kernel");
    *launches = 1;
}

hipError_t launch_dwconv_f32(const ConvProblem &p, const float *x, const float *w,
                             const float *bias, float *y, hipStream_t st)
{
    const long planes = (long)p.N * p.C;
    const int cus = cu_count();
    const int PB = dw_run_planes(p, x, cus);
    if (PB > 0) {
        DwRunArgs a{};
        a.x = x;
        a.w = w;
        a.bias = bias;
        a.y = y;
        a.C = p.C;
        a.planes = planes;
        a.PB = PB;
        a.runs = (planes + PB - 1) / PB;
        a.relu = p.relu;
        const long grid = a.runs < 4L * cus ? a.runs : 4L * cus;   // four 38 KB work-groups per CU
        const dim3 g((unsigned)grid), b(256);
#define MICONV_DW_RUN(HH, ST)                                                         \
    if (p.H == HH && p.stride == ST) {                                               \
        launch_kernel((dw_run_kernel<HH, HH, ST>), g, b, 0, st, a);             \
        return hipGetLastError();                                                    \
    }
        MICONV_DW_RUN(7, 1) MICONV_DW_RUN(7, 2) MICONV_DW_RUN(14, 1) MICONV_DW_RUN(14, 2)
        MICONV_DW_RUN(28, 1) MICONV_DW_RUN(28, 2) MICONV_DW_RUN(56, 1) MICONV_DW_RUN(56, 2)
#undef MICONV_DW_RUN
        return hipErrorInvalidValue;
    }
    const long band_runs = dw_band_runs(p, x, cus);
    if (band_runs > 0) {
        DwRunArgs a{};
        a.x = x;
        a.w = w;
        a.bias = bias;
        a.y = y;
        a.C = p.C;
        a.planes = planes;
        a.PB = 1;
        a.runs = band_runs;
        a.relu = p.relu;
        const dim3 g((unsigned)(4L * cus)), b(256);
        if (p.stride == 1)
            launch_kernel((dw_band_kernel<112, 112, 1, kBandRows1>), g, b, 0, st, a);
        else
            launch_kernel((dw_band_kernel<112, 112, 2, kBandRows2>), g, b, 0, st, a);
        return hipGetLastError();
    }
    const int V = dw_vector_width(p, x, y);
    if (V) {
        DwArgs a{};
        a.x = x;
        a.w = w;
        a.bias = bias;
        a.y = y;
        a.C = p.C;
        a.H = p.H;
        a.W = p.W;
        a.P = p.P;
        a.Q = p.Q;
        a.G = ceil_div(p.Q, V) < 64 ? ceil_div(p.Q, V) : 64;
        a.seg_w = a.G * V;
        a.nseg = ceil_div(p.Q, a.seg_w);
        a.relu = p.relu;
        const long gpw = 64 / a.G;
        // Longest strip that still leaves enough wavefronts to fill the chip.
        int T = 16;
        while (T > 1) {
            const long items = planes * a.nseg * ceil_div(p.P, T);
            if (items / gpw >= 4096) break;
            T /= 2;
        }
        if (T > p.P) T = p.P;
        a.T = T;
        a.nstrip = ceil_div(p.P, T);
        a.items = planes * a.nseg * a.nstrip;
        if (p.stride == 1) {
            if (V == 4) return launch_fast<1, 4>(a, st);
            if (V == 2) return launch_fast<1, 2>(a, st);
            return launch_fast<1, 1>(a, st);
        }
        if (V == 4) return launch_fast<2, 4>(a, st);
        if (V == 2) return launch_fast<2, 2>(a, st);
        return launch_fast<2, 1>(a, st);
    }
    const long total = planes * p.P * p.Q;
    long blocks = (total + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    launch_kernel(dw_generic_kernel, dim3((unsigned)blocks), dim3(256), 0, st, x, w, bias, y,
                       p.C, p.H, p.W, p.R, p.S, p.stride, p.pad, p.P, p.Q, total, p.relu);
    return hipGetLastError();
}

}  // namespace miconv
