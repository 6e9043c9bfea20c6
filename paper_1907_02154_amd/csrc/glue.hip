// Glue operators of the evaluated networks, outside the conv operator:
// max-pool (ResNet stem 3x3/2 pad 1, VGG 2x2/2; fp32 NCHW, and bf16
// channel-last between the layers of a channel-last network), the residual join
// act(a + b) of a bottleneck block, and the fp32 -> bf16 rounding that feeds
// a bf16 conv from an fp32 activation.  All are elementwise or near it and
// bound by HBM bandwidth; lanes walk contiguous memory.
#include "internal.h"

namespace miconv {
namespace {

__global__ __launch_bounds__(256) void maxpool_kernel(const float *__restrict__ x,
                                                      float *__restrict__ y, int H, int W, int R,
                                                      int S, int stride, int pad, int P, int Q,
                                                      long total)
{
    for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += (long)gridDim.x * blockDim.x) {
        const int q = (int)(i % Q);
        const long t = i / Q;
        const int p = (int)(t % P);
        const long plane = t / P;
        const float *xp = x + plane * (long)H * W;
        float m = -INFINITY;
        for (int r = 0; r < R; ++r) {
            const int h = p * stride - pad + r;
            if ((unsigned)h >= (unsigned)H) continue;
            for (int s = 0; s < S; ++s) {
                const int ww = q * stride - pad + s;
                if ((unsigned)ww >= (unsigned)W) continue;
                m = fmaxf(m, xp[(long)h * W + ww]);
            }
        }
        y[i] = m;
    }
}

__global__ __launch_bounds__(256) void add_act_vec4_kernel(const float4 *__restrict__ a,
                                                           const float4 *__restrict__ b,
                                                           float4 *__restrict__ y, long n4,
                                                           int relu)
{
    for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < n4;
         i += (long)gridDim.x * blockDim.x) {
        float4 u = a[i], v = b[i];
        float4 o = make_float4(u.x + v.x, u.y + v.y, u.z + v.z, u.w + v.w);
        if (relu) {
            o.x = fmaxf(o.x, 0.f);
            o.y = fmaxf(o.y, 0.f);
            o.z = fmaxf(o.z, 0.f);
            o.w = fmaxf(o.w, 0.f);
        }
        y[i] = o;
    }
}

__global__ __launch_bounds__(256) void add_act_kernel(const float *a, const float *b, float *y,
                                                      long n, int relu)
{
    for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (long)gridDim.x * blockDim.x) {
        float o = a[i] + b[i];
        y[i] = relu ? fmaxf(o, 0.f) : o;
    }
}

// A thread rounds a pair of elements with one conversion instruction.
__global__ __launch_bounds__(256) void cast_bf16_kernel(const float *__restrict__ x,
                                                        uint16_t *__restrict__ y, long n)
{
    for (long i = 2 * ((long)blockIdx.x * blockDim.x + threadIdx.x); i < n;
         i += 2 * (long)gridDim.x * blockDim.x) {
        const bool two = i + 1 < n;
        const uint32_t d = pack_bf16x2(x[i], two ? x[i + 1] : 0.f);
        y[i] = (uint16_t)d;
        if (two) y[i + 1] = (uint16_t)(d >> 16);
    }
}

// Max-pool over bf16 channel-last tensors: a thread takes 8 channels of one
// output pixel (16-byte loads and store); the maximum of bf16 values is one
// of them, so the result is exact.  Padded positions never win.  Every offset
// fits in 32 bits (the host checks both tensors' sizes), and the index
// divisions use launch-time fast dividers; R_ = S_ = 0 takes the window from
// the arguments, otherwise the window's loads are all issued before the
// maxima.
__device__ __forceinline__ void max_bf16x8(float (&m)[8], uint4 v)
{
    const uint32_t d[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        m[2 * e] = fmaxf(m[2 * e], bf16_to_f32((uint16_t)(d[e] & 0xFFFFu)));
        m[2 * e + 1] = fmaxf(m[2 * e + 1], bf16_to_f32((uint16_t)(d[e] >> 16)));
    }
}

template <int R_, int S_>
__global__ __launch_bounds__(256) void maxpool_nhwc_bf16_kernel(const uint16_t *__restrict__ x,
                                                                uint16_t *__restrict__ y, int C, int H,
                                                                int W, int Rr, int Sr, int stride, int pad,
                                                                int P, int Q, unsigned total, FastDiv dv_c8,
                                                                FastDiv dv_q, FastDiv dv_p)
{
    const int R = R_ ? R_ : Rr, S = S_ ? S_ : Sr;
    const unsigned C8 = (unsigned)C / 8;
    for (unsigned i = blockIdx.x * blockDim.x + threadIdx.x; i < total; i += gridDim.x * blockDim.x) {
        const unsigned pix = fdiv(i, dv_c8);
        const unsigned o = i - pix * C8;
        const unsigned t = fdiv(pix, dv_q);
        const int q = (int)(pix - t * (unsigned)Q);
        const unsigned n = fdiv(t, dv_p);
        const int p = (int)(t - n * (unsigned)P);
        const int h0 = p * stride - pad, w0 = q * stride - pad;
        float m[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) m[e] = -INFINITY;
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int h = h0 + r;
            if constexpr (S_ != 0) {
                uint4 v[S_];
                bool ok[S_];
#pragma unroll
                for (int s = 0; s < S_; ++s) {
                    const int w = w0 + s;
                    ok[s] = (unsigned)h < (unsigned)H && (unsigned)w < (unsigned)W;
                    v[s] = ok[s] ? *reinterpret_cast<const uint4 *>(
                                       x + ((n * (unsigned)H + h) * (unsigned)W + w) * (unsigned)C + 8 * o)
                                 : make_uint4(0, 0, 0, 0);
                }
#pragma unroll
                for (int s = 0; s < S_; ++s)
                    if (ok[s]) max_bf16x8(m, v[s]);
            } else {
                if ((unsigned)h >= (unsigned)H) continue;
                for (int s = 0; s < S; ++s) {
                    const int w = w0 + s;
                    if ((unsigned)w < (unsigned)W)
                        max_bf16x8(m, *reinterpret_cast<const uint4 *>(
                                          x + ((n * (unsigned)H + h) * (unsigned)W + w) * (unsigned)C + 8 * o));
                }
            }
        }
        uint32_t d[4];
#pragma unroll
        for (int e = 0; e < 4; ++e)
            d[e] = pack_bf16x2(m[2 * e], m[2 * e + 1]);
        *reinterpret_cast<uint4 *>(y + pix * (unsigned)C + 8 * o) = make_uint4(d[0], d[1], d[2], d[3]);
    }
}

unsigned grid_for(long n)
{
    long b = (n + 255) / 256;
    if (b < 1) b = 1;
    if (b > 65536) b = 65536;
    return (unsigned)b;
}

}  // namespace

hipError_t launch_maxpool_f32(int N, int C, int H, int W, int R, int S, int stride, int pad,
                              int P, int Q, const float *x, float *y, hipStream_t st)
{
    const long total = (long)N * C * P * Q;
    launch_kernel(maxpool_kernel, dim3(grid_for(total)), dim3(256), 0, st, x, y, H, W, R, S,
                       stride, pad, P, Q, total);
    return hipGetLastError();
}

hipError_t launch_add_act_f32(long count, const float *a, const float *b, float *y, int relu,
                              hipStream_t st)
{
    if (count == 0) return hipSuccess;
    const bool vec = (count % 4 == 0) && ((uintptr_t)a % 16 == 0) && ((uintptr_t)b % 16 == 0) &&
                     ((uintptr_t)y % 16 == 0);
    if (vec) {
        launch_kernel(add_act_vec4_kernel, dim3(grid_for(count / 4)), dim3(256), 0, st,
                           (const float4 *)a, (const float4 *)b, (float4 *)y, count / 4, relu);
    } else {
        launch_kernel(add_act_kernel, dim3(grid_for(count)), dim3(256), 0, st, a, b, y, count,
                           relu);
    }
    return hipGetLastError();
}

hipError_t launch_cast_bf16(long count, const float *x, uint16_t *y, hipStream_t st)
{
    if (count == 0) return hipSuccess;
    launch_kernel(cast_bf16_kernel, dim3(grid_for(count)), dim3(256), 0, st, x, y, count);
    return hipGetLastError();
}

}  // namespace miconv

namespace miconv {

hipError_t launch_maxpool_nhwc_bf16(int N, int C, int H, int W, int R, int S, int stride, int pad, int P,
                                    int Q, const uint16_t *x, uint16_t *y, hipStream_t st)
{
    const long total = (long)N * P * Q * (C / 8);
    if ((long)N * H * W * C > INT_MAX || (long)N * P * Q * C > INT_MAX) return hipErrorInvalidValue;
    const FastDiv dc = make_fastdiv(C / 8), dq = make_fastdiv(Q), dp = make_fastdiv(P);
    if (R == 3 && S == 3)
        launch_kernel(maxpool_nhwc_bf16_kernel<3, 3>, dim3(grid_for(total)), dim3(256), 0, st, x, y, C, H, W, R, S,
                      stride, pad, P, Q, (unsigned)total, dc, dq, dp);
    else
        launch_kernel(maxpool_nhwc_bf16_kernel<0, 0>, dim3(grid_for(total)), dim3(256), 0, st, x, y, C, H, W, R, S,
                      stride, pad, P, Q, (unsigned)total, dc, dq, dp);
    return hipGetLastError();
}

}  // namespace miconv
