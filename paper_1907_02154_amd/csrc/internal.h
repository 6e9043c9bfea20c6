// Internal declarations shared by the HIP translation units of libmiconv.
// Nothing here is part of the public ABI (include/miconv.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace miconv {

// One conv problem, already validated, with the derived extents filled in.
struct ConvProblem {
    int N, C, H, W, K, R, S, stride, pad, groups;
    int P, Q;
    int Cg, Kg;      // channels per group in / out
    int Kred;        // Cg * R * S: the GEMM reduction length
    int M;           // N * P * Q: the GEMM pixel extent
    int relu;
};

// Kernel argument block for the dense paths (passed by value).
struct ConvArgs {
    const void *x;        // fp32 or bf16 bits, [N][C][H][W]
    const void *w;        // fp32 or bf16 bits, [K][Cg][R][S]
    const float *bias;    // [K] or nullptr
    float *y;             // [N][K][P][Q]
    float *ws;            // split-K partials [splits][K][M] (nullptr when splits == 1)
    int *counters;        // split-K arrival counter per output tile, zero between calls
    int N, C, H, W, K, R, S, stride, pad, groups;
    int P, Q, Cg, Kg, Kred, M, PQ, HW;
    int splits;           // reduction split count (grid.z = groups * splits)
    int kr_per_split;     // reduction length per split, a multiple of the chunk size
    int relu;
};

ConvArgs make_args(const ConvProblem &p);

// Launchers.  Each returns hipSuccess or the launch error.
hipError_t launch_conv_direct_f32(const ConvProblem &p, const float *x, const float *w,
                                  const float *bias, float *y, hipStream_t st);
hipError_t launch_conv_direct_bf16(const ConvProblem &p, const uint16_t *x, const uint16_t *w,
                                   const float *bias, float *y, hipStream_t st);
hipError_t launch_dwconv_f32(const ConvProblem &p, const float *x, const float *w,
                             const float *bias, float *y, hipStream_t st);

// Dense implicit-GEMM paths.  A plan fixes the tile and the reduction split;
// `ws_bytes` is the split-K workspace it needs (0 without a split), which the
// caller passes to the launcher as `ws`.
struct IgemmPlan {
    int tile;           // index into the tile table of the kernel family
    int splits;
    int kr_per_split;
    int counters;       // output tiles needing an arrival counter (0 without a split)
    size_t ws_bytes;    // bytes of fp32 partials (0 without a split)
};
IgemmPlan plan_igemm_f32(const ConvProblem &p, int num_cus);
hipError_t launch_igemm_f32(const ConvProblem &p, const IgemmPlan &plan, const float *x,
                            const float *w, const float *bias, float *y, float *ws, int *counters,
                            hipStream_t st);
// Kernel names (as a profiler prints them, without namespace) and launch counts.
void describe_igemm_f32(const ConvProblem &p, const IgemmPlan &plan, char *buf, int len,
                        int *launches);
void describe_dwconv(const ConvProblem &p, char *buf, int len, int *launches);
void describe_direct(int bf16, char *buf, int len, int *launches);

hipError_t launch_maxpool_f32(int N, int C, int H, int W, int R, int S, int stride, int pad,
                              int P, int Q, const float *x, float *y, hipStream_t st);
hipError_t launch_add_act_f32(long count, const float *a, const float *b, float *y, int relu,
                              hipStream_t st);
hipError_t launch_cast_bf16(long count, const float *x, uint16_t *y, hipStream_t st);

__host__ __device__ inline int ceil_div(int a, int b) { return (a + b - 1) / b; }

}  // namespace miconv
