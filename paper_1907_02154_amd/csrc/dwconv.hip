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
// Planes small enough for LDS (every MobileNet depthwise layer) use the
// LDS-run kernel below instead, which reads and writes whole contiguous runs
// of planes; other depthwise shapes (filters up to 7x7, any stride and pad)
// use a plain one-output-per-lane kernel.
#include "internal.h"

#include <cstdio>

namespace miconv {
namespace {

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

// Small planes: a work-group takes runs of PB consecutive (n, c) planes --
// each run one contiguous stretch of PB*H*W inputs in NCHW -- and streams
// them through two LDS buffers: while the lanes compute run i from LDS, the
// 16-byte loads of run i+1 are in flight in registers.  Every lane produces
// 4 consecutive outputs of the run's contiguous output stretch (flattened
// over planes, rows and columns) and writes them with one 16-byte store, so
// HBM sees one contiguous read of x and one contiguous write of y.  The
// filter taps and biases of a run travel with it into LDS.
struct DwLdsArgs {
    const float *x, *w, *bias;
    float *y;
    int C, H, W, P, Q, stride, pad;
    int HW, PQ;
    long planes;
    int PB;          // planes per run (PB*HW <= kRunFloats, PB*HW and PB*PQ multiples of 4)
    long runs;
    int relu;
};

constexpr int kRunFloats = 6144;                   // per LDS buffer (24 KB)
constexpr int kRun4 = kRunFloats / 4 / 256;        // float4 per lane per run

__global__ __launch_bounds__(256) void dw_lds_kernel(DwLdsArgs a)
{
    __shared__ __attribute__((aligned(16))) float xs[2][kRunFloats];
    __shared__ float wb[2][64 * 10];        // per plane of the run: 9 taps, then the bias
    const int tid = threadIdx.x;
    float4 stage[kRun4];
    float tail;          // the last partial run's inputs beyond its last whole float4
    int tail_at;
    float wstage[3];

    auto load = [&](long run) {
        const long plane0 = run * a.PB;
        const int np = run < a.runs ? (int)min((long)a.PB, a.planes - plane0) : 0;
        const int cnt = np * a.HW;
        const int c4 = cnt / 4;
        const float4 *src = reinterpret_cast<const float4 *>(a.x + plane0 * a.HW);
        tail_at = 4 * c4 + tid;
        tail = tail_at < cnt ? a.x[plane0 * a.HW + tail_at] : 0.f;
        if (tail_at >= cnt) tail_at = -1;
#pragma unroll
        for (int i = 0; i < kRun4; ++i) {
            const int j = tid + i * 256;
            stage[i] = j < c4 ? src[j] : make_float4(0.f, 0.f, 0.f, 0.f);
        }
#pragma unroll
        for (int i = 0; i < 3; ++i) {
            const int j = tid + i * 256;          // j = plane * 10 + tap (tap 9 = bias)
            const int pl = j / 10, t = j - pl * 10;
            float v = 0.f;
            if (pl < np) {
                const int c = (int)((plane0 + pl) % a.C);
                v = t < 9 ? a.w[c * 9 + t] : (a.bias ? a.bias[c] : 0.f);
            }
            wstage[i] = v;
        }
    };
    auto store = [&](int buf) {
#pragma unroll
        for (int i = 0; i < kRun4; ++i)
            reinterpret_cast<float4 *>(xs[buf])[tid + i * 256] = stage[i];
        if (tail_at >= 0) xs[buf][tail_at] = tail;
#pragma unroll
        for (int i = 0; i < 3; ++i)
            if (tid + i * 256 < 64 * 10) wb[buf][tid + i * 256] = wstage[i];
    };

    long run = blockIdx.x;
    int buf = 0;
    load(run);
    store(0);
    load(run + gridDim.x);
    __syncthreads();
    for (; run < a.runs; run += gridDim.x) {
        const long plane0 = run * a.PB;
        const int np = (int)min((long)a.PB, a.planes - plane0);
        const float *xr = xs[buf];
        float *dst = a.y + plane0 * a.PQ;
        const int ocnt = np * a.PQ;
        for (int o = tid * 4; o < ocnt; o += 256 * 4) {
            int pl = o / a.PQ;
            int pq = o - pl * a.PQ;
            int p = pq / a.Q;
            int q = pq - p * a.Q;
            float v[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const float *wp = wb[buf] + pl * 10;
                const float *xp = xr + pl * a.HW;
                float acc = wp[9];
                const int h0 = p * a.stride - a.pad, w0 = q * a.stride - a.pad;
#pragma unroll
                for (int r = 0; r < 3; ++r) {
                    const int hh = h0 + r;
                    const bool hv = (unsigned)hh < (unsigned)a.H;
#pragma unroll
                    for (int ss = 0; ss < 3; ++ss) {
                        const int ww = w0 + ss;
                        const bool ok = hv && (unsigned)ww < (unsigned)a.W;
                        acc = fmaf(ok ? xp[hh * a.W + ww] : 0.f, wp[r * 3 + ss], acc);
                    }
                }
                v[e] = a.relu ? fmaxf(acc, 0.f) : acc;
                if (++q == a.Q) {
                    q = 0;
                    if (++p == a.P) {
                        p = 0;
                        ++pl;
                    }
                }
            }
            if (o + 3 < ocnt) {
                *reinterpret_cast<float4 *>(dst + o) = make_float4(v[0], v[1], v[2], v[3]);
            } else {
                for (int e = 0; e < 4; ++e)
                    if (o + e < ocnt) dst[o + e] = v[e];
            }
        }
        // run + gridDim.x is in registers: publish it, start the one after
        buf ^= 1;
        store(buf);
        load(run + 2L * gridDim.x);
        __syncthreads();
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
    hipLaunchKernelGGL((dw3x3_kernel<ST, V>), dim3((unsigned)blocks), dim3(256), 0, st, a);
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

// Planes per LDS run for the small-plane kernel (0: use the lane-group kernel).
// 3x3 filters on planes narrower than 56 columns; runs keep 16-byte alignment.
int dw_lds_planes(const ConvProblem &p, const void *x, const void *y)
{
    if (p.R != 3 || p.S != 3 || p.W >= 56) return 0;
    const long hw = (long)p.H * p.W, pq = (long)p.P * p.Q;
    long pb = kRunFloats / hw;
    if (pb > 64) pb = 64;
    while (pb > 0 && ((pb * hw) % 4 || (pb * pq) % 4)) --pb;
    if (pb <= 0 || !aligned(x, 16) || !aligned(y, 16)) return 0;
    return (int)pb;
}

void describe_dwconv(const ConvProblem &p, char *buf, int len, int *launches)
{
    const int V = dw_vector_width(p, nullptr, nullptr);
    if (dw_lds_planes(p, nullptr, nullptr) > 0)
        snprintf(buf, len, "dw_lds_kernel");
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
    const int PB = dw_lds_planes(p, x, y);
    if (PB > 0) {
        DwLdsArgs a{};
        a.x = x;
        a.w = w;
        a.bias = bias;
        a.y = y;
        a.C = p.C;
        a.H = p.H;
        a.W = p.W;
        a.P = p.P;
        a.Q = p.Q;
        a.stride = p.stride;
        a.pad = p.pad;
        a.HW = p.H * p.W;
        a.PQ = p.P * p.Q;
        a.planes = planes;
        a.PB = PB;
        a.runs = (planes + PB - 1) / PB;
        a.relu = p.relu;
        long grid = a.runs < 2048 ? a.runs : 2048;   // about eight work-groups per CU
        hipLaunchKernelGGL(dw_lds_kernel, dim3((unsigned)grid), dim3(256), 0, st, a);
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
    hipLaunchKernelGGL(dw_generic_kernel, dim3((unsigned)blocks), dim3(256), 0, st, x, w, bias, y,
                       p.C, p.H, p.W, p.R, p.S, p.stride, p.pad, p.P, p.Q, total, p.relu);
    return hipGetLastError();
}

}  // namespace miconv
