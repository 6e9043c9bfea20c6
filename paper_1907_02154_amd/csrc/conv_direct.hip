// Direct convolution (fp32 or bf16 storage): one output element per lane, the plain (c, r, s) FMA
// loop.  It covers every shape and group count the ABI accepts, and serves
// grouped convolutions that are neither dense nor depthwise.  Lanes run along
// the output row (q), so both the x reads of one tap and the y stores are
// contiguous across a wavefront.
#include "internal.h"

#include <cstdio>

namespace miconv {
namespace {

__device__ inline float widen(float v) { return v; }
__device__ inline float widen(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// T = float (fp32 storage) or uint16_t (bf16 bit patterns, widened exactly).
template <typename T>
__global__ __launch_bounds__(256) void conv_direct_kernel(ConvArgs a)
{
    const long total = (long)a.N * a.K * a.PQ;
    const T *__restrict__ x = static_cast<const T *>(a.x);
    const T *__restrict__ w = static_cast<const T *>(a.w);
    for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += (long)gridDim.x * blockDim.x) {
        const int q = (int)(i % a.Q);
        const long t = i / a.Q;
        const int p = (int)(t % a.P);
        const long nk = t / a.P;
        const int k = (int)(nk % a.K);
        const int n = (int)(nk / a.K);
        const int g = k / a.Kg;
        const int h0 = p * a.stride - a.pad, w0 = q * a.stride - a.pad;
        const T *xp = x + ((long)n * a.C + (long)g * a.Cg) * a.HW;
        const T *wp = w + (long)k * a.Kred;
        float acc = 0.f;
        for (int c = 0; c < a.Cg; ++c) {
            for (int r = 0; r < a.R; ++r) {
                const int h = h0 + r;
                if ((unsigned)h >= (unsigned)a.H) continue;
                for (int s = 0; s < a.S; ++s) {
                    const int ww = w0 + s;
                    if ((unsigned)ww >= (unsigned)a.W) continue;
                    acc = fmaf(widen(xp[(long)c * a.HW + h * a.W + ww]),
                               widen(wp[(c * a.R + r) * a.S + s]), acc);
                }
            }
        }
        float v = acc + (a.bias ? a.bias[k] : 0.f);
        const long yi = (long)n * a.ysn + ((long)k * a.P + p) * a.Q + q;
        if (a.res) v += a.res[yi];
        if (a.relu) v = fmaxf(v, 0.f);
        a.y[yi] = v;
    }
}

template <typename T>
hipError_t launch_direct(const ConvProblem &p, const T *x, const T *w, const float *bias, float *y,
                         hipStream_t st)
{
    ConvArgs a = make_args(p);
    a.x = x;
    a.w = w;
    a.bias = bias;
    a.y = y;
    const long total = (long)p.N * p.K * p.P * p.Q;
    long blocks = (total + 255) / 256;
    if (blocks > 65536) blocks = 65536;  // grid-stride loop covers the rest
    launch_kernel(conv_direct_kernel<T>, dim3((unsigned)blocks), dim3(256), 0, st, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_conv_direct_f32(const ConvProblem &p, const float *x, const float *w,
                                  const float *bias, float *y, hipStream_t st)
{
    return launch_direct<float>(p, x, w, bias, y, st);
}

void describe_direct(int bf16, char *buf, int len, int *launches)
{
    snprintf(buf, len, "conv_direct_kernel<%s>", bf16 ? "unsigned short" : "float");
    *launches = 1;
}

hipError_t launch_conv_direct_bf16(const ConvProblem &p, const uint16_t *x, const uint16_t *w,
                                   const float *bias, float *y, hipStream_t st)
{
    return launch_direct<uint16_t>(p, x, w, bias, y, st);
}

}  // namespace miconv
