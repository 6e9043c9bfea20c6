// Weight pre-packing ("pre-computing" at graph level, Sec. 3.2.3): KCRS
// filters -> KRSC, i.e. w_p[k][(r*S + s)*Cg + c] = w[k][c][r][s], or, with a
// channel block B < Cg, KRSC per block of B channels:
// w_p[k][((c/B)*R*S + r*S + s)*B + c%B] = w[k][c][r][s].
//
// With the reduction ordered (r, s, c), c innermost, any 8 consecutive
// reduction indices (Cg % 8 == 0) are 8 channels at one filter tap: a conv
// kernel checks the padding and forms the input address once per 8 taps
// instead of once per tap.  Lanes walk the destination, so stores are
// contiguous; the reads gather within one filter's Cg*R*S block (L2-resident).
#include "internal.h"

namespace miconv {
namespace {

template <typename T>
__global__ __launch_bounds__(256) void pack_krsc_kernel(const T *__restrict__ src, T *__restrict__ dst,
                                                        int K, int Cg, int RS, int cblk, long total)
{
    for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += (long)gridDim.x * blockDim.x) {
        const long k = i / ((long)Cg * RS);
        const int rem = (int)(i - k * Cg * RS);   // (channel block, rs, c) with c fastest
        const int cb = rem / (RS * cblk);
        const int rem2 = rem - cb * RS * cblk;
        const int rs = rem2 / cblk;
        const int c = cb * cblk + (rem2 - rs * cblk);
        dst[i] = src[(k * Cg + c) * RS + rs];
    }
}

// Wave-kernel order: one slot per (group, 32-filter block kb, 8-tap block b,
// lane l, element e) holding W[kb*32 + l%32][8*b + 4*(l/32) + e], where the
// reduction index runs over (c, r, s) (order 0), (r, s, c) (order 1) or
// (r, s, c4) with C/groups <= 4 padded to 4 channels (order 2); zero past
// K/groups and past the reduction.
__global__ __launch_bounds__(256) void pack_wave_kernel(const float *__restrict__ src,
                                                        float *__restrict__ dst, int Kg, int Cg,
                                                        int RS, int KB, int NB, int order, long total)
{
    const int Kred = Cg * RS;                        // source row length
    const int Kpad = order == 2 ? 4 * RS : Kred;     // packed reduction length
    for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += (long)gridDim.x * blockDim.x) {
        const int e = (int)(i & 3);
        const int l = (int)((i >> 2) & 63);
        const long t = i >> 8;                 // (g * KB + kb) * NB + b
        const int b = (int)(t % NB);
        const long gk = t / NB;
        const int kb = (int)(gk % KB);
        const int g = (int)(gk / KB);
        const int k = kb * 32 + (l & 31);
        const int kr = 8 * b + 4 * (l >> 5) + e;
        float v = 0.f;
        if (k < Kg && kr < Kpad) {
            const long row = ((long)g * Kg + k) * Kred;
            if (order == 2) {
                const int rs = kr >> 2, c = kr & 3;
                if (c < Cg) v = src[row + (long)c * RS + rs];
            } else if (order == 1) {
                const int rs = kr / Cg, c = kr - rs * Cg;
                v = src[row + (long)c * RS + rs];
            } else {
                v = src[row + kr];
            }
        }
        dst[i] = v;
    }
}

}  // namespace

int wave_order(const ConvProblem &p)
{
    if (p.Cg % 8 == 0) return 1;
    if (p.Cg <= 4 && p.R * p.S > 1) return 2;
    return 0;
}

int wave_kred(const ConvProblem &p) { return wave_order(p) == 2 ? 4 * p.R * p.S : p.Kred; }

size_t wave_packed_floats(const ConvProblem &p)
{
    return (size_t)p.groups * ceil_div(p.Kg, 32) * ceil_div(wave_kred(p), 8) * 256;
}

hipError_t launch_pack_wave(const ConvProblem &p, const float *w, float *packed, hipStream_t st)
{
    const long total = (long)wave_packed_floats(p);
    long blocks = (total + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    launch_kernel(pack_wave_kernel, dim3((unsigned)blocks), dim3(256), 0, st, w, packed, p.Kg,
                  p.Cg, p.R * p.S, ceil_div(p.Kg, 32), ceil_div(wave_kred(p), 8), wave_order(p), total);
    return hipGetLastError();
}

hipError_t launch_pack_krsc(const ConvProblem &p, const void *w, void *packed, size_t elem,
                            hipStream_t st, int cblk)
{
    const long total = (long)p.K * p.Cg * p.R * p.S;
    if (cblk <= 0) cblk = p.Cg;
    if (p.Cg % cblk != 0) return hipErrorInvalidValue;
    long blocks = (total + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    if (elem == sizeof(float))
        launch_kernel(pack_krsc_kernel<float>, dim3((unsigned)blocks), dim3(256), 0, st,
                           static_cast<const float *>(w), static_cast<float *>(packed), p.K, p.Cg,
                           p.R * p.S, cblk, total);
    else
        launch_kernel(pack_krsc_kernel<uint16_t>, dim3((unsigned)blocks), dim3(256), 0, st,
                           static_cast<const uint16_t *>(w), static_cast<uint16_t *>(packed), p.K,
                           p.Cg, p.R * p.S, cblk, total);
    return hipGetLastError();
}

}  // namespace miconv
