/*
 * CPU oracle for the CNN-inference convolution hot path.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may link, load or
 * call this file; only the tests, the smoke check and the bench's CPU-baseline
 * leg do.  It shares no code, header or table with the HIP library.
 *
 * The paper optimises the Conv2D operator of CNN inference (Sec. 3.2.2) and
 * states that its optimisations keep the model semantics and lose no accuracy
 * (Sec. 4.2, Sec. 5).  It never writes the operator down, so this file is the
 * standard deep-learning definition written out:
 *
 *   P = floor((H + 2*pad - R) / stride) + 1,  Q likewise with W and S
 *   g = k / (K/groups),  Cg = C/groups
 *   y[n][k][p][q] = act( bias[k] + sum_{c<Cg, r<R, s<S}
 *                        x[n][g*Cg+c][p*stride-pad+r][q*stride-pad+s] * w[k][c][r][s] )
 *
 * with zero padding (taps outside the image contribute nothing), no kernel
 * flip (cross-correlation), act = ReLU or identity.  Every product of two
 * fp32 (or bf16) values is exact in fp64; the sum for one output starts at
 * the bias and adds the terms in lexicographic (c, r, s) order in fp64; the
 * result is rounded once to fp32 (round to nearest even).
 *
 * The loop order below is n, k | c, r, s | p, q with one fp64 accumulator
 * per output pixel.  For any single output the terms are still added in
 * (c, r, s) order, so the result is bitwise the same as the textbook
 * n, k, p, q, c, r, s nest.  OpenMP parallelises over (n, k) only.
 *
 * Depthwise convolution (MobileNet, Sec. 4.2) is the same function with
 * groups = C = K.  The glue operators of the evaluated networks (max-pool,
 * residual add + ReLU, fp32 -> bf16 rounding) are written out here too.
 *
 * Build: gcc -O2 -fopenmp -fno-fast-math -ffp-contract=off -shared -fPIC
 */
#include <stddef.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <math.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define REF_OK 0
#define REF_EINVAL -1
#define REF_ENOMEM -2

/* Output extent along one axis: floor((in + 2*pad - k) / stride) + 1; <= 0 if empty. */
static long ref_extent(long in, long k, long stride, long pad)
{
    long span = in + 2 * pad - k;
    if (span < 0) return 0;
    return span / stride + 1;
}

int ref_out_dims(int H, int W, int R, int S, int stride, int pad, int *P, int *Q)
{
    if (H <= 0 || W <= 0 || R <= 0 || S <= 0 || stride <= 0 || pad < 0 || !P || !Q)
        return REF_EINVAL;
    *P = (int)ref_extent(H, R, stride, pad);
    *Q = (int)ref_extent(W, S, stride, pad);
    return REF_OK;
}

/* Threads an OpenMP region of this library uses. */
int ref_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* bf16 bit pattern -> its exact fp32 value (bf16 is the top half of fp32). */
static float ref_bf16_to_f32(uint16_t b)
{
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return f;
}

/*
 * The shared body.  x and w are read through `load`, which widens either
 * fp32 or bf16 storage to an exact fp64 value.
 */
typedef double (*ref_load_fn)(const void *base, size_t i);

static double ref_load_f32(const void *base, size_t i)
{
    return (double)((const float *)base)[i];
}

static double ref_load_bf16(const void *base, size_t i)
{
    return (double)ref_bf16_to_f32(((const uint16_t *)base)[i]);
}

static int ref_conv2d_any(int N, int C, int H, int W, int K, int R, int S,
                          int stride, int pad, int groups,
                          const void *x, const void *w, ref_load_fn load,
                          const float *bias, const float *res, float *y, int relu)
{
    if (N <= 0 || C <= 0 || H <= 0 || W <= 0 || K <= 0 || R <= 0 || S <= 0 ||
        stride <= 0 || pad < 0 || groups <= 0 || !x || !w || !y)
        return REF_EINVAL;
    if (C % groups != 0 || K % groups != 0)
        return REF_EINVAL;
    const long P = ref_extent(H, R, stride, pad);
    const long Q = ref_extent(W, S, stride, pad);
    if (P <= 0 || Q <= 0)
        return REF_EINVAL;
    const long Cg = C / groups, Kg = K / groups;
    const long HW = (long)H * W, PQ = P * Q;
    int status = REF_OK;

#pragma omp parallel
    {
        double *acc = (double *)malloc(sizeof(double) * (size_t)PQ);
        if (!acc) {
#pragma omp atomic write
            status = REF_ENOMEM;
        }
#pragma omp for collapse(2) schedule(dynamic, 1)
        for (long n = 0; n < N; ++n) {
            for (long k = 0; k < K; ++k) {
                if (!acc) continue;
                const long g = k / Kg;
                const double b0 = bias ? (double)bias[k] : 0.0;
                for (long i = 0; i < PQ; ++i) acc[i] = b0;
                for (long c = 0; c < Cg; ++c) {
                    const size_t xplane = (size_t)((n * C + g * Cg + c) * HW);
                    for (long r = 0; r < R; ++r) {
                        for (long s = 0; s < S; ++s) {
                            const double wv = load(w, (size_t)(((k * Cg + c) * R + r) * S + s));
                            for (long p = 0; p < P; ++p) {
                                const long h = p * stride - pad + r;
                                if (h < 0 || h >= H) continue;
                                double *arow = acc + p * Q;
                                for (long q = 0; q < Q; ++q) {
                                    const long ww = q * stride - pad + s;
                                    if (ww < 0 || ww >= W) continue;
                                    arow[q] += load(x, xplane + (size_t)(h * W + ww)) * wv;
                                }
                            }
                        }
                    }
                }
                float *yp = y + (size_t)((n * K + k) * PQ);
                const float *rp = res ? res + (size_t)((n * K + k) * PQ) : NULL;
                for (long i = 0; i < PQ; ++i) {
                    double v = acc[i];
                    if (rp) v += (double)rp[i];   /* residual join, before the activation */
                    if (relu && v < 0.0) v = 0.0;
                    yp[i] = (float)v;
                }
            }
        }
        free(acc);
    }
    return status;
}

/* Dense / grouped conv on fp32 storage.  Layouts: x NCHW, w [K][C/groups][R][S],
 * bias [K] or NULL, y [N][K][P][Q]. */
int ref_conv2d_f32(int N, int C, int H, int W, int K, int R, int S, int stride, int pad,
                   int groups, const float *x, const float *w, const float *bias, float *y,
                   int relu)
{
    return ref_conv2d_any(N, C, H, W, K, R, S, stride, pad, groups, x, w, ref_load_f32,
                          bias, NULL, y, relu);
}

/* Conv2D followed by the residual join of a bottleneck block, fused as the
 * graph-level operator fusion does (Sec. 3.2.3):
 * y = act(conv(x, w) + bias + res), res [N][K][P][Q] fp32, the whole sum in
 * fp64 and rounded once.  x16 != 0: x and w are bf16 bit patterns. */
int ref_conv2d_res(int N, int C, int H, int W, int K, int R, int S, int stride, int pad,
                   int groups, int x16, const void *x, const void *w, const float *bias,
                   const float *res, float *y, int relu)
{
    if (!res) return REF_EINVAL;
    return ref_conv2d_any(N, C, H, W, K, R, S, stride, pad, groups, x, w,
                          x16 ? ref_load_bf16 : ref_load_f32, bias, res, y, relu);
}

/* Same operator with x and w stored as bf16 bit patterns (widened exactly);
 * bias and y stay fp32. */
int ref_conv2d_bf16(int N, int C, int H, int W, int K, int R, int S, int stride, int pad,
                    int groups, const uint16_t *x, const uint16_t *w, const float *bias,
                    float *y, int relu)
{
    return ref_conv2d_any(N, C, H, W, K, R, S, stride, pad, groups, x, w, ref_load_bf16,
                          bias, NULL, y, relu);
}

/* Depthwise conv: one R x S filter per channel, w [C][1][R][S]. */
int ref_dwconv2d_f32(int N, int C, int H, int W, int R, int S, int stride, int pad,
                     const float *x, const float *w, const float *bias, float *y, int relu)
{
    return ref_conv2d_any(N, C, H, W, C, R, S, stride, pad, C, x, w, ref_load_f32, bias, NULL,
                          y, relu);
}

/*
 * Max-pool with window R x S, stride and symmetric pad; padded positions are
 * ignored (they never win).  ResNet's stem pool is 3x3/2 pad 1, VGG's 2x2/2.
 */
int ref_maxpool2d_f32(int N, int C, int H, int W, int R, int S, int stride, int pad,
                      const float *x, float *y)
{
    if (N <= 0 || C <= 0 || H <= 0 || W <= 0 || R <= 0 || S <= 0 || stride <= 0 ||
        pad < 0 || pad >= R || pad >= S || !x || !y)
        return REF_EINVAL;
    const long P = ref_extent(H, R, stride, pad), Q = ref_extent(W, S, stride, pad);
    if (P <= 0 || Q <= 0) return REF_EINVAL;
#pragma omp parallel for collapse(2)
    for (long n = 0; n < N; ++n)
        for (long c = 0; c < C; ++c) {
            const float *xp = x + (size_t)((n * C + c) * H * (long)W);
            float *yp = y + (size_t)((n * C + c) * P * Q);
            for (long p = 0; p < P; ++p)
                for (long q = 0; q < Q; ++q) {
                    float m = -INFINITY;
                    for (long r = 0; r < R; ++r)
                        for (long s = 0; s < S; ++s) {
                            long h = p * stride - pad + r, ww = q * stride - pad + s;
                            if (h < 0 || h >= H || ww < 0 || ww >= W) continue;
                            float v = xp[h * W + ww];
                            if (v > m) m = v;
                        }
                    yp[p * Q + q] = m;
                }
        }
    return REF_OK;
}

/* Residual join of a bottleneck block: y = act(a + b) elementwise in fp32. */
int ref_add_act_f32(long count, const float *a, const float *b, float *y, int relu)
{
    if (count < 0 || (count > 0 && (!a || !b || !y))) return REF_EINVAL;
    for (long i = 0; i < count; ++i) {
        float v = a[i] + b[i];
        if (relu && v < 0.0f) v = 0.0f;
        y[i] = v;
    }
    return REF_OK;
}

/*
 * fp32 -> bf16 with round-to-nearest, ties to even, written from the
 * definition: keep the top 16 bits, look at the 16 discarded bits and round
 * up when they exceed half an ulp, or equal half and the kept part is odd.
 * NaN stays a (quiet) NaN; overflow rounds to infinity as IEEE says.
 */
static uint16_t ref_f32_to_bf16_one(float f)
{
    uint32_t u;
    memcpy(&u, &f, sizeof u);
    if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu) != 0)
        return (uint16_t)((u >> 16) | 0x0040u);
    uint32_t kept = u >> 16;
    uint32_t dropped = u & 0xFFFFu;
    if (dropped > 0x8000u || (dropped == 0x8000u && (kept & 1u)))
        kept += 1u;
    return (uint16_t)kept;
}

int ref_f32_to_bf16(long count, const float *x, uint16_t *y)
{
    if (count < 0 || (count > 0 && (!x || !y))) return REF_EINVAL;
    for (long i = 0; i < count; ++i) y[i] = ref_f32_to_bf16_one(x[i]);
    return REF_OK;
}
