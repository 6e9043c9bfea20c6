// Internal declarations shared by the HIP translation units of libmiconv.
// Nothing here is part of the public ABI (include/miconv.h).
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace miconv {

// Kernel timing: a caller that wants the execution time of the next kernel
// launch on this thread sets these two events; launch_kernel hands them to
// the runtime, which stamps them with the kernel's start and end, and clears
// them.  Unset (the normal case), launch_kernel is a plain launch.
extern thread_local hipEvent_t t_launch_start, t_launch_stop;

template <typename F, typename... Args>
inline void launch_kernel(F kernel, dim3 grid, dim3 block, uint32_t shm, hipStream_t st, Args... args)
{
    hipEvent_t a = t_launch_start, b = t_launch_stop;
    t_launch_start = t_launch_stop = nullptr;
    if (a)
        hipExtLaunchKernelGGL(kernel, grid, block, shm, st, a, b, 0, args...);
    else
        hipLaunchKernelGGL(kernel, grid, block, shm, st, args...);
}

// One conv problem, already validated, with the derived extents filled in.
struct ConvProblem {
    int N, C, H, W, K, R, S, stride, pad, groups;
    int P, Q;
    int Cg, Kg;      // channels per group in / out
    int Kred;        // Cg * R * S: the GEMM reduction length
    int M;           // N * P * Q: the GEMM pixel extent
    int relu;
    const float *res;  // [N][K][P][Q] added to the conv + bias before the activation, or nullptr
                       // (with ycl: bf16 [N][P][Q][K], the layout of y)
    long ysn;          // elements from one image of y (and res) to the next: K*P*Q when dense
    int xcl;           // x is bf16 channel-last [N][H][W][C] (else NCHW)
    int ycl;           // y (and res) bf16 channel-last [N][P][Q][K] (else fp32 NCHW)
};

// fp32 -> bf16 bits, round to nearest even on the raw bits: add 0x7FFF plus
// the lowest kept bit, keep the upper half.  A NaN keeps its sign and gets the
// quiet bit.
__host__ __device__ inline uint16_t f32_to_bf16_rne(float f)
{
    uint32_t u;
    __builtin_memcpy(&u, &f, 4);
    if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu))
        return (uint16_t)((u >> 16) | 0x0040u);
    return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

// Two floats rounded as f32_to_bf16_rne does, packed lo | hi << 16, in one
// instruction (v_cvt_pk_bf16_f32, round to nearest even; compared with
// f32_to_bf16_rne on the device over all 2^32 bit patterns: identical,
// NaNs included).
typedef __bf16 miconv_bf16x2 __attribute__((ext_vector_type(2)));
typedef float miconv_floatx2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi)
{
    const miconv_floatx2 f = {lo, hi};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, miconv_bf16x2));
}

__host__ __device__ inline float bf16_to_f32(uint16_t b)
{
    const uint32_t u = (uint32_t)b << 16;
    float f;
    __builtin_memcpy(&f, &u, 4);
    return f;
}

// Division by a divisor d >= 1 fixed at launch, for numerators below 2^31:
// n / d = (mulhi(n, mul) + n) >> shift with shift = ceil(log2 d) and
// mul = floor(2^32 (2^shift - d) / d) + 1 (the round-up method of Granlund
// and Montgomery, 1994; the sum stays below 2^32 for n < 2^31).  Three
// instructions in place of a ~20-instruction integer division.
struct FastDiv {
    unsigned mul, shift;
};

inline FastDiv make_fastdiv(unsigned d)
{
    unsigned l = 0;
    while ((1ull << l) < d) ++l;
    return FastDiv{(unsigned)(((1ull << 32) * ((1ull << l) - d)) / d + 1), l};
}

__host__ __device__ __forceinline__ unsigned fdiv(unsigned n, FastDiv f)
{
    return ((unsigned)(((unsigned long long)n * f.mul) >> 32) + n) >> f.shift;   // v_mul_hi_u32 on the GPU
}

// Kernel argument block for the dense paths (passed by value).
struct ConvArgs {
    const void *x;        // fp32 or bf16 bits, [N][C][H][W]
    const void *w;        // fp32 or bf16 bits, [K][Cg][R][S]
    const float *bias;    // [K] or nullptr
    float *y;             // [N][K][P][Q]
    float *ws;            // split-K partials [splits][K][M] (nullptr when splits == 1)
    int N, C, H, W, K, R, S, stride, pad, groups;
    int P, Q, Cg, Kg, Kred, M, PQ, HW;
    int splits;           // reduction split count (grid.z = groups * splits)
    int kr_per_split;     // reduction length per split, a multiple of the chunk size
    int relu;
    int vec4;             // split-K reduce may use 16-byte accesses (one image, aligned)
    FastDiv dv_pq, dv_q;  // division by P*Q and by Q
    FastDiv dv_m;         // division by M (split-K reduce)
    FastDiv dv_mt, dv_kt, dv_g, dv_cb;   // wave kernel: pixel tiles, filter tiles, groups, C/groups/8
                                         // (dv_kt: K/8 in the channel-last split reduce)
    // Last, so that the fields every kernel reads first keep their offsets at
    // the front of the argument block (batch-1 kernels run a few microseconds).
    const float *res;     // [N][K][P][Q] residual added before the activation, or nullptr; it may
                          // be y itself (every element is read and written by one thread)
    long ysn;             // elements from one image of y (and res) to the next (>= K*P*Q)
    int ycl;              // y and res bf16 [N*P*Q][K]; split partials then [splits][M][K]
};

ConvArgs make_args(const ConvProblem &p);

// Compute units of the current device (cached per device).
int cu_count();

// Called before every kernel launch of one conv (the stack executor records
// a timing event there).
struct LaunchHook {
    hipError_t (*before_launch)(void *ctx, hipStream_t st);
    void *ctx;
};

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
    size_t ws_bytes;    // bytes of fp32 partials (0 without a split)
    bool krsc;          // filters pre-packed [K][R][S][C/groups] (reduction order r, s, c)
};
IgemmPlan plan_igemm_f32(const ConvProblem &p, int num_cus, int max_splits);
hipError_t launch_igemm_f32(const ConvProblem &p, const IgemmPlan &plan, const float *x,
                            const float *w, const float *bias, float *y, float *ws,
                            hipStream_t st, const LaunchHook *hook = nullptr);
// Small-extent dense path (batch-1 layers): wavefronts feed the MFMAs from
// global memory and split the reduction among themselves.
struct WavePlan {
    int bj;             // 32-pixel blocks per work-group tile (1 or 2)
    int waves;          // wavefronts per work-group splitting the reduction (4 or 8)
    int splits;         // reduction splits across work-groups
    int kr_per_split;
    size_t ws_bytes;
    int order;          // reduction order of the packed filters (wave_order)
    bool ind;           // each wavefront owns a tile and its whole reduction (short
                        // reductions over many tiles); waves then groups tiles
    bool kc;            // filters read as given (KCRS), not from a packed copy
};
// The wave kernel addresses x and its packed filters with 32-bit offsets.
bool wave_fits(const ConvProblem &p);
WavePlan plan_wave_f32(const ConvProblem &p, int num_cus, int max_splits);
// The kernel reading w as given loads a half-block's 4 taps as one 16-byte load.
bool wave_kc_vector(const ConvProblem &p, const WavePlan &plan, const void *w);
hipError_t launch_wave_f32(const ConvProblem &p, const WavePlan &plan, const float *x,
                           const float *w, const float *bias, float *y, float *ws,
                           hipStream_t st, const LaunchHook *hook = nullptr);
void describe_wave_f32(const ConvProblem &p, const WavePlan &plan, char *buf, int len,
                       int *launches);
// bf16 inputs, fp32 accumulation (v_mfma_f32_32x32x16_bf16).
IgemmPlan plan_igemm_bf16(const ConvProblem &p, int num_cus, int max_splits);
bool bf16_fast_1x1(const ConvProblem &p, const void *x);
hipError_t launch_igemm_bf16(const ConvProblem &p, const IgemmPlan &plan, bool fast, bool va,
                             const uint16_t *x, const uint16_t *w, const float *bias, float *y,
                             float *ws, hipStream_t st, const LaunchHook *hook = nullptr);
void describe_igemm_bf16(const ConvProblem &p, const IgemmPlan &plan, bool fast, bool va,
                         char *buf, int len, int *launches);

// bf16 through an internal channel-last copy of x (C/groups % 32 == 0).
struct NhwcPlan {
    int dma;              // direct-to-LDS kernel (64-channel chunks), else the register-staged one
    int nchwb;            // (dma, 1x1 stride 1) pixel operand read from NCHW x, no channel-last
                          // copy: 1 = 16-byte loads (H*W % 8 == 0), 2 = 4-byte loads (H*W even)
    int tile;             // index into the kernel family's tile table
    int krc;              // reduction chunk (64 or 32 channels at one filter position)
    int splits;
    int kr_per_split;
    size_t partial_bytes; // split-K partials
    size_t xcl_bytes;     // the channel-last copy of x
    int copy_cb;          // channels per work-group of the whole-plane copy
    int halo;             // 3x3 stride-1 layers: patch rows of the halo kernel (0: not used);
                          // its filters are packed in 64-channel blocks
    int x_nhwc;           // x is already channel-last: no copy
};
bool nhwc_bf16_eligible(const ConvProblem &p);
// x_nhwc: x is given channel-last (direct-to-LDS kernels only, C/groups % 64 == 0).
NhwcPlan plan_nhwc_bf16(const ConvProblem &p, int num_cus, const void *x, int max_splits, bool x_nhwc = false);
hipError_t launch_nhwc_bf16(const ConvProblem &p, const NhwcPlan &plan, const uint16_t *x,
                            const uint16_t *w_krsc, const float *bias, float *y, uint16_t *xcl,
                            float *partials, hipStream_t st, const LaunchHook *hook = nullptr);
void describe_nhwc_bf16(const ConvProblem &p, const NhwcPlan &plan, char *buf, int len,
                        int *launches);

// bf16 7x7/2 stem on <= 4 channels with 112 output columns (filters packed by
// launch_pack_stem into [K][28 tap pairs][8]).
bool stem_bf16_eligible(const ConvProblem &p, const void *y);
size_t stem_packed_bytes(const ConvProblem &p);
hipError_t launch_pack_stem(const ConvProblem &p, const uint16_t *w, uint16_t *packed, hipStream_t st);
hipError_t launch_stem_bf16(const ConvProblem &p, const uint16_t *x, const uint16_t *wpacked,
                            const float *bias, float *y, hipStream_t st);
void describe_stem_bf16(char *buf, int len, int *launches);

// Sums split partials [splits][K][M] in split order into y (+ bias, activation).
hipError_t launch_splitk_reduce(ConvArgs a, hipStream_t st);

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
// Max-pool on bf16 channel-last tensors, x [N][H][W][C] -> y [N][P][Q][C].
hipError_t launch_maxpool_nhwc_bf16(int N, int C, int H, int W, int R, int S, int stride, int pad, int P,
                                    int Q, const uint16_t *x, uint16_t *y, hipStream_t st);

// A validated conv call with its kernel fixed (what the ABI entry points and
// the stack executor enqueue).
enum OpKind { OP_DENSE_F32 = 0, OP_DENSE_BF16 = 1, OP_DW_F32 = 2, OP_MAXPOOL_BF16_NHWC = 3, OP_MAXPOOL_F32 = 4 };
// Layout flags of a bf16 dense layer (enum miconv_layout).
enum LayoutFlags { LAYOUT_X_NHWC = 1, LAYOUT_Y_NHWC_BF16 = 2 };
enum Impl {
    IMPL_DIRECT = 0,
    IMPL_IGEMM = 1,
    IMPL_DW = 2,
    IMPL_WAVE = 3,
    IMPL_IGEMM_BF16 = 4,
    IMPL_NHWC_BF16 = 5,
    IMPL_STEM_BF16 = 6,
    IMPL_POOL_NHWC = 7,
    IMPL_POOL_F32 = 8
};
// What a call may use besides its tensors.
enum PlanMode {
    MODE_FREE = 0,      // nothing: no workspace, filters read as given (plain entry points)
    MODE_SCRATCH = 1,   // a caller workspace: split partials, a channel-last copy of x,
                        // filters packed per call
    MODE_PREPACK = 2    // filters packed ahead into a buffer of their own (stack executor,
                        // packed-filter entry point); with MODE_SCRATCH: a stack layer
};
// The filter layout a resolved layer's kernel reads.
enum WeightLayout {
    WL_GIVEN = 0,       // w as the caller holds it, [K][C/groups][R][S]
    WL_STEM = 1,        // bf16 7x7 stem: tap pairs
    WL_WAVE = 2,        // fp32 wave kernel: wavefront load order
    WL_KRSC = 3,        // [K][R][S][C/groups]
    WL_KRSC_BLOCK = 4   // KRSC per block of 64 channels
};
struct Resolved {
    ConvProblem p;
    int kind;
    int impl;
    int mode;           // enum PlanMode the plan was made for
    int wlayout;        // enum WeightLayout the kernel reads
    IgemmPlan plan;     // IMPL_IGEMM only
    WavePlan wplan;     // IMPL_WAVE only
    bool bfast, bva;    // IMPL_IGEMM_BF16: vectorised 1x1 loader, 16-byte filter loads
    NhwcPlan nplan;     // IMPL_NHWC_BF16 only
    bool pack_per_call; // enqueue packs the filters into the workspace first
    const void *wk;     // filters the conv kernel reads when they were packed ahead (else w)
    const void *x, *w;
    const float *bias;
    float *y;
};
int resolve(int kind, int algo, int mode, int N, int C, int H, int W, int K, int R, int S, int stride,
            int pad, int groups, const void *x, const void *w, const float *bias, float *y,
            int relu, Resolved *out, int layout = 0);
// resolve() for tensors at 256-byte boundaries (w may be null: a stand-in).
int resolve_aligned(int N, int C, int H, int W, int K, int R, int S, int stride, int pad, int groups,
                    int dtype, int algo, int mode, const void *w, Resolved *out);
// One dense call with an optional residual and output image stride (dtype 0
// fp32, 1 bf16), planned for `mode`.
int resolve_ex(int mode, int N, int C, int H, int W, int K, int R, int S, int stride, int pad,
               int groups, int dtype, int algo, const void *x, const void *w, const float *bias,
               const float *res, float *y, long y_image_stride, int relu, Resolved *r);
// Enqueue r on a workspace of ws_bytes bytes, 256-byte aligned (ws may be null
// when workspace_bytes(r) is 0); returns a miconv_status.
int run(const Resolved &r, void *ws, size_t ws_bytes, hipStream_t st);
// Adds a residual [N][K][P][Q] (read at y's indices, before the activation) to
// a resolved dense layer; nullptr leaves it unchanged.
int set_residual(Resolved &r, const float *res);
// Sets the distance in elements between images of y (and res); 0 keeps the
// dense K*P*Q.  A larger stride lets y be a channel range of a wider tensor.
int set_output_stride(Resolved &r, long ysn);
// ws: the workspace of workspace_bytes(r) bytes, 256-byte aligned (nullptr when 0).
hipError_t enqueue(const Resolved &r, float *ws, hipStream_t st, const LaunchHook *hook = nullptr);
void describe(const Resolved &r, char *buf, int len, int *launches);
size_t workspace_bytes(const Resolved &r);   // packed filters (per-call packing) + copy + split partials
hipError_t launch_pack(const Resolved &r, void *dst, hipStream_t st);   // the copy its kernel reads
size_t packed_bytes(const Resolved &r);      // bytes of that copy
void set_packed(Resolved &r, const void *packed);  // read filters packed ahead at `packed`
// Filters in the wave kernel's A-operand order, w_pk[g][ceil(Kg/32)][ceil(Kred/8)][64][4]
// (reduction order r, s, c when `krsc`, else c, r, s), zero-padded.
// Reduction order of the wave kernel's packed filters: 0 = (c, r, s),
// 1 = (r, s, c) for C/groups % 8 == 0, 2 = (r, s, c4) with C/groups <= 4
// padded to 4 channels (R*S > 1); wave_kred is the packed reduction length.
int wave_order(const ConvProblem &p);
int wave_kred(const ConvProblem &p);
size_t wave_packed_floats(const ConvProblem &p);
hipError_t launch_pack_wave(const ConvProblem &p, const float *w, float *packed, hipStream_t st);
// cblk: channel block of the (block, r, s, c) order; 0 = C/groups (plain KRSC).
hipError_t launch_pack_krsc(const ConvProblem &p, const void *w, void *packed, size_t elem,
                            hipStream_t st, int cblk = 0);
int set_hip_error(hipError_t e);   // records e for miconv_last_hip_error, returns MICONV_ERR_HIP

__host__ __device__ inline int ceil_div(int a, int b) { return (a + b - 1) / b; }

}  // namespace miconv
