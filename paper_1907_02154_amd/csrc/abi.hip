// The C ABI of libmiconv (include/miconv.h): argument validation, output
// extents and the shape -> kernel choice.  The library owns no device memory
// on this path: a call that needs scratch (split partials, a channel-last
// copy of x, packed filters) takes it from the caller's workspace, and the
// entry points without a workspace pick plans that need none.
//
// The paper's observation that convolutions of different shapes need
// different schedules (Sec. 2.2) is served here by a fixed, hand-written
// dispatch rule instead of a searched tuning log: depthwise shapes go to the
// depthwise kernel, dense shapes to the implicit-GEMM MFMA kernel with a tile
// and reduction split picked from the GEMM extents, and thin grouped
// convolutions to the direct kernel.
#include "../../include/miconv.h"
#include "internal.h"

#include <algorithm>
#include <climits>
#include <map>
#include <mutex>

namespace miconv {

thread_local hipEvent_t t_launch_start = nullptr, t_launch_stop = nullptr;

ConvArgs make_args(const ConvProblem &p)
{
    ConvArgs a{};
    a.N = p.N;
    a.C = p.C;
    a.H = p.H;
    a.W = p.W;
    a.K = p.K;
    a.R = p.R;
    a.S = p.S;
    a.stride = p.stride;
    a.pad = p.pad;
    a.groups = p.groups;
    a.P = p.P;
    a.Q = p.Q;
    a.Cg = p.Cg;
    a.Kg = p.Kg;
    a.Kred = p.Kred;
    a.M = p.M;
    a.PQ = p.P * p.Q;
    a.HW = p.H * p.W;
    a.splits = 1;
    a.kr_per_split = p.Kred;
    a.relu = p.relu;
    a.res = p.res;
    a.ysn = p.ysn;
    a.ycl = p.ycl;
    a.dv_pq = make_fastdiv(p.P * p.Q);
    a.dv_q = make_fastdiv(p.Q);
    return a;
}

namespace {

thread_local int g_last_hip_error = 0;

int hip_fail(hipError_t e)
{
    g_last_hip_error = (int)e;
    return MICONV_ERR_HIP;
}

long extent(long in, long k, long stride, long pad)
{
    const long span = in + 2 * pad - k;
    return span < 0 ? 0 : span / stride + 1;
}

int validate(int N, int C, int H, int W, int K, int R, int S, int stride, int pad, int groups,
             const void *x, const void *w, const void *y, size_t elem, ConvProblem *p)
{
    if (!x || !w || !y) return MICONV_ERR_NULL;
    if (N <= 0 || C <= 0 || H <= 0 || W <= 0 || K <= 0 || R <= 0 || S <= 0 || stride < 1 ||
        pad < 0)
        return MICONV_ERR_SHAPE;
    if (groups < 1 || C % groups != 0 || K % groups != 0) return MICONV_ERR_GROUPS;
    const long P = extent(H, R, stride, pad), Q = extent(W, S, stride, pad);
    if (P < 1 || Q < 1) return MICONV_ERR_SHAPE;
    const long Cg = C / groups, Kg = K / groups;
    const long lim = INT_MAX;
    if ((long)N * C * H * W > lim || K * Cg * R * S > lim || (long)N * K * P * Q > lim ||
        P * Q > lim || (long)H * W > lim || Cg * R * S > lim || (long)N * P * Q > lim)
        return MICONV_ERR_TOO_LARGE;
    if ((uintptr_t)x % elem || (uintptr_t)w % elem || (uintptr_t)y % sizeof(float))
        return MICONV_ERR_ALIGN;
    p->N = N;
    p->C = C;
    p->H = H;
    p->W = W;
    p->K = K;
    p->R = R;
    p->S = S;
    p->stride = stride;
    p->pad = pad;
    p->groups = groups;
    p->P = (int)P;
    p->Q = (int)Q;
    p->Cg = (int)Cg;
    p->Kg = (int)Kg;
    p->Kred = (int)(Cg * R * S);
    p->M = (int)((long)N * P * Q);
    p->relu = 0;
    p->res = nullptr;
    p->ysn = (long)K * P * Q;
    return MICONV_OK;
}

int check_bias(const float *bias)
{
    return (bias && (uintptr_t)bias % sizeof(float)) ? MICONV_ERR_ALIGN : MICONV_OK;
}


int finish(hipError_t e) { return e == hipSuccess ? MICONV_OK : hip_fail(e); }

}  // namespace

int cu_count()
{
    static std::mutex mu;
    static std::map<int, int> cache;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 256;
    std::lock_guard<std::mutex> lk(mu);
    auto it = cache.find(dev);
    if (it != cache.end()) return it->second;
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
        n = 256;
    cache[dev] = n;
    return n;
}

int set_hip_error(hipError_t e) { return hip_fail(e); }

// Validate one conv call and fix the kernel that serves it.  `mode` says what
// the call may use besides its tensors (enum PlanMode): without a workspace
// there is no split reduction, no channel-last copy and no per-call filter
// packing, and filters are read as given unless they were packed ahead.
// Max-pool as a stack layer (K = C, no filters): bf16 channel-last, or fp32 NCHW.
static int resolve_pool(int kind, int N, int C, int H, int W, int K, int R, int S, int stride, int pad,
                        const void *x, float *y, Resolved *out)
{
    if (!x || !y) return MICONV_ERR_NULL;
    if (N <= 0 || C <= 0 || H <= 0 || W <= 0 || R <= 0 || S <= 0 || stride < 1 || pad < 0 || pad >= R ||
        pad >= S)
        return MICONV_ERR_SHAPE;
    if (K != C) return MICONV_ERR_GROUPS;
    const bool cl = kind == OP_MAXPOOL_BF16_NHWC;
    if (cl && C % 8) return MICONV_ERR_UNSUPPORTED;
    const long P = extent(H, R, stride, pad), Q = extent(W, S, stride, pad);
    if (P < 1 || Q < 1) return MICONV_ERR_SHAPE;
    if ((long)N * C * H * W > INT_MAX || (long)N * C * P * Q > INT_MAX) return MICONV_ERR_TOO_LARGE;
    if (cl ? ((uintptr_t)x % 16 || (uintptr_t)y % 16) : ((uintptr_t)x % 4 || (uintptr_t)y % 4))
        return MICONV_ERR_ALIGN;
    Resolved r{};
    r.kind = kind;
    r.impl = cl ? IMPL_POOL_NHWC : IMPL_POOL_F32;
    r.p.N = N;
    r.p.C = C;
    r.p.H = H;
    r.p.W = W;
    r.p.K = K;
    r.p.R = R;
    r.p.S = S;
    r.p.stride = stride;
    r.p.pad = pad;
    r.p.groups = 1;
    r.p.P = (int)P;
    r.p.Q = (int)Q;
    r.p.xcl = r.p.ycl = cl ? 1 : 0;
    r.x = x;
    r.y = y;
    *out = r;
    return MICONV_OK;
}

int resolve(int kind, int algo, int mode, int N, int C, int H, int W, int K, int R, int S, int stride,
            int pad, int groups, const void *x, const void *w, const float *bias, float *y,
            int relu, Resolved *out, int layout)
{
    if (kind == OP_MAXPOOL_BF16_NHWC || kind == OP_MAXPOOL_F32)
        return resolve_pool(kind, N, C, H, W, K, R, S, stride, pad, x, y, out);
    Resolved r{};
    const size_t elem = kind == OP_DENSE_BF16 ? sizeof(uint16_t) : sizeof(float);
    int rc = validate(N, C, H, W, K, R, S, stride, pad, groups, x, w, y, elem, &r.p);
    if (rc != MICONV_OK) return rc;
    if ((rc = check_bias(bias)) != MICONV_OK) return rc;
    if (algo < MICONV_ALGO_AUTO || algo > MICONV_ALGO_WAVE) return MICONV_ERR_UNSUPPORTED;
    if (mode < MODE_FREE || mode > (MODE_SCRATCH | MODE_PREPACK)) return MICONV_ERR_UNSUPPORTED;
    const bool scratch = mode & MODE_SCRATCH;
    const bool can_pack = mode & (MODE_SCRATCH | MODE_PREPACK);   // per call, or ahead
    const int max_splits = scratch ? 64 : 1;
    r.p.relu = relu ? 1 : 0;
    r.kind = kind;
    r.mode = mode;
    r.x = x;
    r.w = w;
    r.bias = bias;
    r.y = y;
    const bool depthwise = groups > 1 && groups == C && K == C;
    if (layout & ~(LAYOUT_X_NHWC | LAYOUT_Y_NHWC_BF16)) return MICONV_ERR_UNSUPPORTED;
    if (layout) {
        // Channel-last bf16 layers of a channel-last network: x [N][H][W][C]
        // read as given by the direct-to-LDS kernels, and/or y (and the
        // residual) bf16 [N][P][Q][K] written by their channel-last epilogue;
        // x in NCHW with a channel-last y is the 7x7 stem's kernel.
        if (kind != OP_DENSE_BF16 || algo != MICONV_ALGO_AUTO) return MICONV_ERR_UNSUPPORTED;
        r.p.xcl = (layout & LAYOUT_X_NHWC) ? 1 : 0;
        r.p.ycl = (layout & LAYOUT_Y_NHWC_BF16) ? 1 : 0;
        if (r.p.ycl && (uintptr_t)y % 16) return MICONV_ERR_ALIGN;
        if (r.p.xcl) {
            const bool fits = (long)N * C * H * W * 2 < (1L << 31) && (long)K * r.p.Kred * 2 < (1L << 31);
            if (r.p.Cg % 64 || !fits || (R * S > 1 && !can_pack)) return MICONV_ERR_UNSUPPORTED;
            if (r.p.ycl && r.p.Kg % 8) return MICONV_ERR_UNSUPPORTED;
            if (R * S == 1 && (uintptr_t)w % 16) return MICONV_ERR_ALIGN;
            if ((uintptr_t)x % 16) return MICONV_ERR_ALIGN;
            r.impl = IMPL_NHWC_BF16;
            r.nplan = plan_nhwc_bf16(r.p, cu_count(), x, max_splits, true);
            r.wlayout = R * S == 1 ? WL_GIVEN : r.nplan.halo ? WL_KRSC_BLOCK : WL_KRSC;
        } else {
            if (!r.p.ycl || !can_pack || !stem_bf16_eligible(r.p, y) || K % 8) return MICONV_ERR_UNSUPPORTED;
            r.impl = IMPL_STEM_BF16;
            r.wlayout = WL_STEM;
        }
        r.pack_per_call = r.wlayout != WL_GIVEN && !(mode & MODE_PREPACK);
        *out = r;
        return MICONV_OK;
    }
    if (kind == OP_DW_F32) {
        if (!depthwise) return MICONV_ERR_GROUPS;
        if (R > 7 || S > 7) return MICONV_ERR_UNSUPPORTED;
        r.impl = IMPL_DW;
    } else if (kind == OP_DENSE_BF16) {
        if (algo == MICONV_ALGO_DIRECT || (groups > 1 && r.p.Cg < 8)) {
            r.impl = IMPL_DIRECT;
        } else if (algo == MICONV_ALGO_AUTO && can_pack && stem_bf16_eligible(r.p, y)) {
            r.impl = IMPL_STEM_BF16;
            r.wlayout = WL_STEM;
        } else {
            r.impl = IMPL_IGEMM_BF16;
            if (algo != MICONV_ALGO_IGEMM && nhwc_bf16_eligible(r.p)) {
                const NhwcPlan np = plan_nhwc_bf16(r.p, cu_count(), x, max_splits);
                const bool one = R * S == 1;
                // a copy of x or split partials need a workspace; filters of
                // more than one tap are read KRSC-packed; 1x1 filters are read
                // as given, with 16-byte loads
                const bool ok = ((np.xcl_bytes == 0 && np.splits == 1) || scratch) &&
                                (one ? (uintptr_t)w % 16 == 0 : can_pack);
                if (ok) {
                    r.impl = IMPL_NHWC_BF16;
                    r.nplan = np;
                    r.wlayout = one ? WL_GIVEN : np.halo ? WL_KRSC_BLOCK : WL_KRSC;
                }
            }
            if (r.impl == IMPL_IGEMM_BF16) {
                r.plan = plan_igemm_bf16(r.p, cu_count(), max_splits);
                r.bfast = bf16_fast_1x1(r.p, x);
                // At the batch sizes the bf16 path serves, packing the filters
                // costs far less than per-tap index decoding in the gather.
                if (can_pack && R * S > 1 && r.p.Cg % 8 == 0) {
                    r.plan.krsc = true;
                    r.wlayout = WL_KRSC;
                }
                // 16-byte filter loads: packed copies are 256-byte aligned
                r.bva = r.p.Kred % 8 == 0 && (r.wlayout != WL_GIVEN || (uintptr_t)w % 16 == 0);
            }
        }
    } else if (kind == OP_DENSE_F32) {
        if (algo == MICONV_ALGO_AUTO) {
            if (depthwise && R <= 7 && S <= 7)
                r.impl = IMPL_DW;
            else
                r.impl = (groups == 1 || r.p.Cg >= 8) ? IMPL_IGEMM : IMPL_DIRECT;
        } else {
            r.impl = algo == MICONV_ALGO_DIRECT ? IMPL_DIRECT
                     : algo == MICONV_ALGO_WAVE ? IMPL_WAVE : IMPL_IGEMM;
        }
        const int cus = cu_count();
        if (r.impl == IMPL_IGEMM) {
            // The wave kernel serves every size it can address (measured faster
            // than the LDS-tiled kernel from batch-1 ResNet layers to VGG-16 at
            // batch 32), unless the caller forced the tiled one.
            if (algo != MICONV_ALGO_IGEMM && wave_fits(r.p))
                r.impl = IMPL_WAVE;
            else
                r.plan = plan_igemm_f32(r.p, cus, max_splits);
        }
        if (r.impl == IMPL_WAVE) {
            if (!wave_fits(r.p)) return MICONV_ERR_UNSUPPORTED;
            r.wplan = plan_wave_f32(r.p, cus, max_splits);
            // filters packed ahead in the wavefront load order, else read as given
            r.wplan.kc = !(mode & MODE_PREPACK);
            r.wlayout = r.wplan.kc ? WL_GIVEN : WL_WAVE;
            // Read as given, a filter row holds its taps in (c, r, s) order:
            // reducing in that order makes a half-block's 4 taps one 16-byte
            // load (the (r, s, c) order would take four 4-byte loads R*S
            // floats apart), for one padding test per tap on the pixel side.
            if (r.wplan.kc && r.wplan.order == 1 && R * S > 1 && r.p.Kred % 4 == 0 && (uintptr_t)w % 16 == 0)
                r.wplan.order = 0;
        }
    } else {
        return MICONV_ERR_UNSUPPORTED;
    }
    r.pack_per_call = r.wlayout != WL_GIVEN && !(mode & MODE_PREPACK);
    *out = r;
    return MICONV_OK;
}

int set_residual(Resolved &r, const float *res)
{
    if (!res) return MICONV_OK;
    if (r.impl == IMPL_POOL_NHWC || r.impl == IMPL_POOL_F32) return MICONV_ERR_UNSUPPORTED;
    if (r.p.ycl) {
        // bf16 [N][P][Q][K] like y, read with 16-byte loads; the stem takes none
        if ((uintptr_t)res % 16) return MICONV_ERR_ALIGN;
        if (r.impl != IMPL_NHWC_BF16) return MICONV_ERR_UNSUPPORTED;
        r.p.res = res;
        return MICONV_OK;
    }
    // Kernels read it with the same (possibly 16-byte) accesses as they write y.
    if ((uintptr_t)res % sizeof(float) || ((uintptr_t)res - (uintptr_t)r.y) % 16)
        return MICONV_ERR_ALIGN;
    if (r.impl == IMPL_DW) return MICONV_ERR_UNSUPPORTED;
    r.p.res = res;
    // the plan of a 1x1 layer reading NCHW x depends on the residual (tile choice)
    if (r.impl == IMPL_NHWC_BF16 && r.nplan.nchwb)
        r.nplan = plan_nhwc_bf16(r.p, cu_count(), r.x, (r.mode & MODE_SCRATCH) ? 64 : 1);
    return MICONV_OK;
}

int set_output_stride(Resolved &r, long ysn)
{
    const long dense = (long)r.p.K * r.p.P * r.p.Q;
    if (ysn == 0 || ysn == dense) return MICONV_OK;
    if (r.p.ycl || r.impl == IMPL_POOL_NHWC || r.impl == IMPL_POOL_F32)
        return MICONV_ERR_UNSUPPORTED;   // channel-last y is dense; pools take no stride
    if (ysn < dense) return MICONV_ERR_SHAPE;                  // images would overlap
    if ((long)(r.p.N - 1) * ysn + dense > INT_MAX) return MICONV_ERR_TOO_LARGE;
    if (r.impl == IMPL_DW) return MICONV_ERR_UNSUPPORTED;
    r.p.ysn = ysn;
    return MICONV_OK;
}

size_t packed_bytes(const Resolved &r)
{
    if (r.wlayout == WL_STEM) return stem_packed_bytes(r.p);
    if (r.wlayout == WL_WAVE) return wave_packed_floats(r.p) * sizeof(float);
    const size_t elem = r.kind == OP_DENSE_BF16 ? sizeof(uint16_t) : sizeof(float);
    return (size_t)r.p.K * r.p.Cg * r.p.R * r.p.S * elem;
}

void set_packed(Resolved &r, const void *packed)
{
    r.wk = packed;
    r.pack_per_call = false;
}

static size_t round256(size_t v) { return (v + 255) / 256 * 256; }

// The layer as the entry point of `mode` resolves it for tensors at 256-byte
// boundaries (w may be null: 256-aligned stand-in).
int resolve_aligned(int N, int C, int H, int W, int K, int R, int S, int stride, int pad, int groups,
                    int dtype, int algo, int mode, const void *w, Resolved *out)
{
    if (dtype != 0 && dtype != 1) return MICONV_ERR_UNSUPPORTED;
    alignas(256) static const float stand_in[64] = {};
    return resolve(dtype == 1 ? OP_DENSE_BF16 : OP_DENSE_F32, algo, mode, N, C, H, W, K, R, S, stride,
                   pad, groups, stand_in, w ? w : stand_in, nullptr, const_cast<float *>(stand_in), 0, out);
}

// The filter copy a layer's kernel reads: tap-pair order for the bf16 stem,
// the wavefront load order for the wave kernel, KRSC (per 64-channel block
// for the halo kernel) otherwise.
hipError_t launch_pack(const Resolved &r, void *dst, hipStream_t st)
{
    if (r.wlayout == WL_STEM)
        return launch_pack_stem(r.p, static_cast<const uint16_t *>(r.w), static_cast<uint16_t *>(dst), st);
    if (r.wlayout == WL_WAVE)
        return launch_pack_wave(r.p, static_cast<const float *>(r.w), static_cast<float *>(dst), st);
    const size_t elem = r.kind == OP_DENSE_BF16 ? sizeof(uint16_t) : sizeof(float);
    const int cblk = r.wlayout == WL_KRSC_BLOCK ? 64 : 0;   // (block, r, s, c) order
    return launch_pack_krsc(r.p, r.w, dst, elem, st, cblk);
}

hipError_t enqueue(const Resolved &r0, float *ws, hipStream_t st, const LaunchHook *hook)
{
    Resolved r = r0;
    // workspace layout: [packed filters (per-call packing)][channel-last x][split partials]
    char *cursor = reinterpret_cast<char *>(ws);
    if (r.pack_per_call) {
        if (hook) {
            hipError_t e = hook->before_launch(hook->ctx, st);
            if (e != hipSuccess) return e;
        }
        hipError_t e = launch_pack(r, cursor, st);
        if (e != hipSuccess) return e;
        r.wk = cursor;
        cursor += round256(packed_bytes(r));
    }
    uint16_t *xcl = nullptr;
    if (r.impl == IMPL_NHWC_BF16) {
        xcl = reinterpret_cast<uint16_t *>(cursor);
        cursor += round256(r.nplan.xcl_bytes);
    }
    ws = reinterpret_cast<float *>(cursor);
    const void *wkern = r.wk ? r.wk : r.w;
    if (r.impl == IMPL_NHWC_BF16)
        return launch_nhwc_bf16(r.p, r.nplan, static_cast<const uint16_t *>(r.x),
                                static_cast<const uint16_t *>(wkern), r.bias, r.y, xcl, ws, st, hook);
    const float *xf = static_cast<const float *>(r.x), *wf = static_cast<const float *>(wkern);
    if (r.impl == IMPL_IGEMM) return launch_igemm_f32(r.p, r.plan, xf, wf, r.bias, r.y, ws, st, hook);
    if (r.impl == IMPL_WAVE) return launch_wave_f32(r.p, r.wplan, xf, wf, r.bias, r.y, ws, st, hook);
    if (r.impl == IMPL_STEM_BF16) {
        if (hook) {
            hipError_t e = hook->before_launch(hook->ctx, st);
            if (e != hipSuccess) return e;
        }
        return launch_stem_bf16(r.p, static_cast<const uint16_t *>(r.x),
                                static_cast<const uint16_t *>(wkern), r.bias, r.y, st);
    }
    if (r.impl == IMPL_IGEMM_BF16)
        return launch_igemm_bf16(r.p, r.plan, r.bfast, r.bva, static_cast<const uint16_t *>(r.x),
                                 static_cast<const uint16_t *>(wkern), r.bias, r.y, ws, st, hook);
    if (hook) {
        hipError_t e = hook->before_launch(hook->ctx, st);
        if (e != hipSuccess) return e;
    }
    switch (r.impl) {
    case IMPL_DW: return launch_dwconv_f32(r.p, xf, wf, r.bias, r.y, st);
    case IMPL_POOL_F32:
        return launch_maxpool_f32(r.p.N, r.p.C, r.p.H, r.p.W, r.p.R, r.p.S, r.p.stride, r.p.pad, r.p.P, r.p.Q,
                                  static_cast<const float *>(r.x), r.y, st);
    case IMPL_POOL_NHWC:
        return launch_maxpool_nhwc_bf16(r.p.N, r.p.C, r.p.H, r.p.W, r.p.R, r.p.S, r.p.stride, r.p.pad, r.p.P,
                                        r.p.Q, static_cast<const uint16_t *>(r.x), reinterpret_cast<uint16_t *>(r.y),
                                        st);
    default:
        if (r.kind == OP_DENSE_BF16)
            return launch_conv_direct_bf16(r.p, static_cast<const uint16_t *>(r.x),
                                           static_cast<const uint16_t *>(r.w), r.bias, r.y, st);
        return launch_conv_direct_f32(r.p, xf, wf, r.bias, r.y, st);
    }
}

void describe_kernel(const Resolved &r, char *buf, int len, int *launches);

size_t workspace_bytes(const Resolved &r)
{
    size_t b = 0;
    if (r.impl == IMPL_IGEMM || r.impl == IMPL_IGEMM_BF16) b = r.plan.ws_bytes;
    if (r.impl == IMPL_WAVE) b = r.wplan.ws_bytes;
    if (r.impl == IMPL_NHWC_BF16) b = round256(r.nplan.xcl_bytes) + r.nplan.partial_bytes;
    if (r.pack_per_call) b = round256(b) + round256(packed_bytes(r));
    return b;
}

void describe(const Resolved &r, char *buf, int len, int *launches)
{
    if (r.pack_per_call) {
        const int n = r.wlayout == WL_STEM ? snprintf(buf, len, "pack_stem_kernel + ")
                      : r.wlayout == WL_WAVE ? snprintf(buf, len, "pack_wave_kernel + ")
                                               : snprintf(buf, len, "pack_krsc_kernel<%s> + ",
                                     r.kind == OP_DENSE_BF16 ? "unsigned short" : "float");
        if (n > 0 && n < len) {
            describe_kernel(r, buf + n, len - n, launches);
            *launches += 1;
            return;
        }
    }
    describe_kernel(r, buf, len, launches);
}

void describe_kernel(const Resolved &r, char *buf, int len, int *launches)
{
    switch (r.impl) {
    case IMPL_DW: describe_dwconv(r.p, buf, len, launches); break;
    case IMPL_IGEMM: describe_igemm_f32(r.p, r.plan, buf, len, launches); break;
    case IMPL_WAVE: describe_wave_f32(r.p, r.wplan, buf, len, launches); break;
    case IMPL_IGEMM_BF16: describe_igemm_bf16(r.p, r.plan, r.bfast, r.bva, buf, len, launches); break;
    case IMPL_NHWC_BF16: describe_nhwc_bf16(r.p, r.nplan, buf, len, launches); break;
    case IMPL_STEM_BF16: describe_stem_bf16(buf, len, launches); break;
    case IMPL_POOL_NHWC:
        snprintf(buf, len, r.p.R == 3 && r.p.S == 3 ? "maxpool_nhwc_bf16_kernel<3, 3>" : "maxpool_nhwc_bf16_kernel<0, 0>");
        *launches = 1;
        break;
    case IMPL_POOL_F32:
        snprintf(buf, len, "maxpool_kernel");
        *launches = 1;
        break;
    default: describe_direct(r.kind == OP_DENSE_BF16, buf, len, launches); break;
    }
}

// Enqueue a resolved call on a workspace of ws_bytes bytes (ws may be null
// when the plan needs none).  Never allocates, frees or synchronises.
int run(const Resolved &r, void *ws, size_t ws_bytes, hipStream_t st)
{
    const size_t need = workspace_bytes(r);
    if (need) {
        if (!ws || ws_bytes < need || (uintptr_t)ws % 256) return MICONV_ERR_WORKSPACE;
    }
    return finish(enqueue(r, need ? static_cast<float *>(ws) : nullptr, st));
}

namespace {

// An entry point without a workspace: the plan takes none by construction.
int run_free(const Resolved &r, hipStream_t st) { return run(r, nullptr, 0, st); }

}  // namespace
}  // namespace miconv

using namespace miconv;

extern "C" {

int miconv_out_dims(int H, int W, int R, int S, int stride, int pad, int *P, int *Q)
{
    if (!P || !Q) return MICONV_ERR_NULL;
    if (H <= 0 || W <= 0 || R <= 0 || S <= 0 || stride < 1 || pad < 0) return MICONV_ERR_SHAPE;
    const long p = extent(H, R, stride, pad), q = extent(W, S, stride, pad);
    *P = (int)p;
    *Q = (int)q;
    return (p < 1 || q < 1) ? MICONV_ERR_SHAPE : MICONV_OK;
}

int conv2d_fwd_algo(int N, int C, int H, int W, int K, int R, int S, int stride, int pad,
                    int groups, const float *x, const float *w, const float *bias, float *y,
                    int relu, int algo, void *stream)
{
    Resolved r;
    int rc = resolve(OP_DENSE_F32, algo, MODE_FREE, N, C, H, W, K, R, S, stride, pad, groups, x, w, bias,
                     y, relu, &r);
    return rc != MICONV_OK ? rc : run_free(r, static_cast<hipStream_t>(stream));
}

int conv2d_fwd(int N, int C, int H, int W, int K, int R, int S, int stride, int pad, int groups,
               const float *x, const float *w, const float *bias, float *y, int relu, void *stream)
{
    return conv2d_fwd_algo(N, C, H, W, K, R, S, stride, pad, groups, x, w, bias, y, relu,
                           MICONV_ALGO_AUTO, stream);
}

int conv2d_fwd_bf16_algo(int N, int C, int H, int W, int K, int R, int S, int stride, int pad,
                         int groups, const uint16_t *x, const uint16_t *w, const float *bias,
                         float *y, int relu, int algo, void *stream)
{
    Resolved r;
    int rc = resolve(OP_DENSE_BF16, algo, MODE_FREE, N, C, H, W, K, R, S, stride, pad, groups, x, w, bias,
                     y, relu, &r);
    return rc != MICONV_OK ? rc : run_free(r, static_cast<hipStream_t>(stream));
}

int conv2d_fwd_bf16(int N, int C, int H, int W, int K, int R, int S, int stride, int pad,
                    int groups, const uint16_t *x, const uint16_t *w, const float *bias, float *y,
                    int relu, void *stream)
{
    return conv2d_fwd_bf16_algo(N, C, H, W, K, R, S, stride, pad, groups, x, w, bias, y, relu,
                                MICONV_ALGO_AUTO, stream);
}

}  // extern "C"

namespace miconv {

// conv2d_fwd_ex / conv2d_fwd_ws: one dense call with an optional residual and
// output image stride, planned for `mode`.
int resolve_ex(int mode, int N, int C, int H, int W, int K, int R, int S, int stride, int pad,
               int groups, int dtype, int algo, const void *x, const void *w, const float *bias,
               const float *res, float *y, long y_image_stride, int relu, Resolved *r)
{
    if (dtype != 0 && dtype != 1) return MICONV_ERR_UNSUPPORTED;
    int rc = resolve(dtype == 1 ? OP_DENSE_BF16 : OP_DENSE_F32, algo, mode, N, C, H, W, K, R, S, stride,
                     pad, groups, x, w, bias, y, relu, r);
    if (rc == MICONV_OK) rc = set_output_stride(*r, y_image_stride);
    if (rc == MICONV_OK) rc = set_residual(*r, res);
    return rc;
}

}  // namespace miconv

extern "C" {

int conv2d_fwd_ex(int N, int C, int H, int W, int K, int R, int S, int stride, int pad,
                  int groups, int dtype, int algo, const void *x, const void *w, const float *bias,
                  const float *res, float *y, long y_image_stride, int relu, void *stream)
{
    Resolved r;
    const int rc = resolve_ex(MODE_FREE, N, C, H, W, K, R, S, stride, pad, groups, dtype, algo, x, w, bias,
                              res, y, y_image_stride, relu, &r);
    return rc != MICONV_OK ? rc : run_free(r, static_cast<hipStream_t>(stream));
}

int conv2d_fwd_res(int N, int C, int H, int W, int K, int R, int S, int stride, int pad,
                   int groups, int dtype, int algo, const void *x, const void *w,
                   const float *bias, const float *res, float *y, int relu, void *stream)
{
    return conv2d_fwd_ex(N, C, H, W, K, R, S, stride, pad, groups, dtype, algo, x, w, bias, res, y, 0,
                         relu, stream);
}

long conv2d_workspace_bytes(int N, int C, int H, int W, int K, int R, int S, int stride, int pad,
                            int groups, int dtype, int algo)
{
    // The plan depends on pointer alignment (16-byte loads, a stem kernel that
    // needs a 16-byte aligned y): take the largest workspace over aligned and
    // misaligned x, w and y, so the figure holds for any pointers.
    if (dtype != 0 && dtype != 1) return MICONV_ERR_UNSUPPORTED;
    alignas(256) static const float stand_in[256] = {};
    const char *base = reinterpret_cast<const char *>(stand_in);
    const int elem = dtype == 1 ? 2 : 4;
    size_t most = 0;
    for (int v = 0; v < 8; ++v) {
        const void *x = base + ((v & 1) ? elem : 0);
        const void *w = base + ((v & 2) ? elem : 0);
        float *y = const_cast<float *>(reinterpret_cast<const float *>(base + ((v & 4) ? 4 : 0)));
        Resolved r;
        const int rc = resolve(dtype == 1 ? OP_DENSE_BF16 : OP_DENSE_F32, algo, MODE_SCRATCH, N, C, H, W, K,
                               R, S, stride, pad, groups, x, w, nullptr, y, 0, &r);
        if (rc != MICONV_OK) return rc;
        most = std::max(most, workspace_bytes(r));
    }
    return (long)most;
}

int conv2d_fwd_ws(int N, int C, int H, int W, int K, int R, int S, int stride, int pad, int groups,
                  int dtype, int algo, const void *x, const void *w, const float *bias, const float *res,
                  float *y, long y_image_stride, int relu, void *ws, size_t ws_bytes, void *stream)
{
    Resolved r;
    const int rc = resolve_ex(MODE_SCRATCH, N, C, H, W, K, R, S, stride, pad, groups, dtype, algo, x, w,
                              bias, res, y, y_image_stride, relu, &r);
    return rc != MICONV_OK ? rc : run(r, ws, ws_bytes, static_cast<hipStream_t>(stream));
}

long conv2d_cl_workspace_bytes(int N, int C, int H, int W, int K, int R, int S, int stride, int pad,
                               int groups, int layout)
{
    if (layout == 0) return conv2d_workspace_bytes(N, C, H, W, K, R, S, stride, pad, groups, 1, MICONV_ALGO_AUTO);
    alignas(256) static const float stand_in[64] = {};
    Resolved r;
    const int rc = resolve(OP_DENSE_BF16, MICONV_ALGO_AUTO, MODE_SCRATCH, N, C, H, W, K, R, S, stride, pad,
                           groups, stand_in, stand_in, nullptr, const_cast<float *>(stand_in), 0, &r, layout);
    return rc != MICONV_OK ? rc : (long)workspace_bytes(r);
}

int conv2d_fwd_cl(int N, int C, int H, int W, int K, int R, int S, int stride, int pad, int groups,
                  int layout, const uint16_t *x, const uint16_t *w, const float *bias, const void *res,
                  void *y, int relu, void *ws, size_t ws_bytes, void *stream)
{
    Resolved r;
    int rc = resolve(OP_DENSE_BF16, MICONV_ALGO_AUTO, MODE_SCRATCH, N, C, H, W, K, R, S, stride, pad, groups,
                     x, w, bias, static_cast<float *>(y), relu, &r, layout);
    if (rc == MICONV_OK) rc = set_residual(r, static_cast<const float *>(res));
    return rc != MICONV_OK ? rc : run(r, ws, ws_bytes, static_cast<hipStream_t>(stream));
}

int conv2d_cl_describe(int N, int C, int H, int W, int K, int R, int S, int stride, int pad, int groups,
                       int layout, char *buf, int buflen, int *launches)
{
    if (!buf || buflen <= 0 || !launches) return MICONV_ERR_NULL;
    buf[0] = 0;
    alignas(256) static const float stand_in[64] = {};
    Resolved r;
    const int rc = resolve(OP_DENSE_BF16, MICONV_ALGO_AUTO, MODE_SCRATCH, N, C, H, W, K, R, S, stride, pad,
                           groups, stand_in, stand_in, nullptr, const_cast<float *>(stand_in), 0, &r, layout);
    if (rc != MICONV_OK) return rc;
    describe(r, buf, buflen, launches);
    return MICONV_OK;
}

int maxpool2d_nhwc_bf16(int N, int C, int H, int W, int R, int S, int stride, int pad, const uint16_t *x,
                        uint16_t *y, void *stream)
{
    Resolved r;
    const int rc = resolve(OP_MAXPOOL_BF16_NHWC, MICONV_ALGO_AUTO, MODE_FREE, N, C, H, W, C, R, S, stride, pad,
                           1, x, nullptr, nullptr, reinterpret_cast<float *>(y), 0, &r);
    return rc != MICONV_OK ? rc : run_free(r, static_cast<hipStream_t>(stream));
}

long conv2d_packed_weight_bytes(int N, int C, int H, int W, int K, int R, int S, int stride,
                                int pad, int groups, int dtype)
{
    Resolved r;
    const int rc = resolve_aligned(N, C, H, W, K, R, S, stride, pad, groups, dtype, MICONV_ALGO_AUTO,
                                   MODE_PREPACK, nullptr, &r);
    if (rc != MICONV_OK) return rc;
    return r.wlayout != WL_GIVEN ? (long)packed_bytes(r) : 0;
}

int conv2d_pack_weights(int N, int C, int H, int W, int K, int R, int S, int stride, int pad,
                        int groups, int dtype, const void *w, void *packed, void *stream)
{
    if (!w || !packed) return MICONV_ERR_NULL;
    Resolved r;
    const int rc = resolve_aligned(N, C, H, W, K, R, S, stride, pad, groups, dtype, MICONV_ALGO_AUTO,
                                   MODE_PREPACK, w, &r);
    if (rc != MICONV_OK) return rc;
    if (r.wlayout == WL_GIVEN) return MICONV_OK;
    if ((uintptr_t)packed % 16 != 0) return MICONV_ERR_ALIGN;
    return finish(launch_pack(r, packed, static_cast<hipStream_t>(stream)));
}

int conv2d_fwd_packed(int N, int C, int H, int W, int K, int R, int S, int stride, int pad,
                      int groups, int dtype, const void *x, const void *packed, const float *bias,
                      float *y, int relu, void *stream)
{
    if (dtype != 0 && dtype != 1) return MICONV_ERR_UNSUPPORTED;
    Resolved r, ref;
    int rc = resolve(dtype == 1 ? OP_DENSE_BF16 : OP_DENSE_F32, MICONV_ALGO_AUTO, MODE_PREPACK, N, C, H, W,
                     K, R, S, stride, pad, groups, x, packed, bias, y, relu, &r);
    if (rc != MICONV_OK) return rc;
    rc = resolve_aligned(N, C, H, W, K, R, S, stride, pad, groups, dtype, MICONV_ALGO_AUTO, MODE_PREPACK,
                         nullptr, &ref);
    if (rc != MICONV_OK) return rc;
    if (r.wlayout != ref.wlayout) return MICONV_ERR_ALIGN;
    if (r.wlayout != WL_GIVEN) {
        if ((uintptr_t)packed % 16 != 0) return MICONV_ERR_ALIGN;
        set_packed(r, packed);
    }
    return run_free(r, static_cast<hipStream_t>(stream));
}

int dwconv2d_fwd(int N, int C, int H, int W, int K, int R, int S, int stride, int pad, int groups,
                 const float *x, const float *w, const float *bias, float *y, int relu,
                 void *stream)
{
    Resolved r;
    int rc = resolve(OP_DW_F32, MICONV_ALGO_AUTO, MODE_FREE, N, C, H, W, K, R, S, stride, pad, groups, x, w,
                     bias, y, relu, &r);
    return rc != MICONV_OK ? rc : run_free(r, static_cast<hipStream_t>(stream));
}

int maxpool2d_fwd(int N, int C, int H, int W, int R, int S, int stride, int pad, const float *x,
                  float *y, void *stream)
{
    if (!x || !y) return MICONV_ERR_NULL;
    if (N <= 0 || C <= 0 || H <= 0 || W <= 0 || R <= 0 || S <= 0 || stride < 1 || pad < 0 ||
        pad >= R || pad >= S)
        return MICONV_ERR_SHAPE;
    const long P = extent(H, R, stride, pad), Q = extent(W, S, stride, pad);
    if (P < 1 || Q < 1) return MICONV_ERR_SHAPE;
    if ((long)N * C * H * W > INT_MAX || (long)N * C * P * Q > INT_MAX) return MICONV_ERR_TOO_LARGE;
    if ((uintptr_t)x % 4 || (uintptr_t)y % 4) return MICONV_ERR_ALIGN;
    return finish(launch_maxpool_f32(N, C, H, W, R, S, stride, pad, (int)P, (int)Q, x, y,
                                     static_cast<hipStream_t>(stream)));
}

int add_act_fwd(long count, const float *a, const float *b, float *y, int relu, void *stream)
{
    if (count < 0) return MICONV_ERR_SHAPE;
    if (count > 0 && (!a || !b || !y)) return MICONV_ERR_NULL;
    if ((uintptr_t)a % 4 || (uintptr_t)b % 4 || (uintptr_t)y % 4) return MICONV_ERR_ALIGN;
    return finish(launch_add_act_f32(count, a, b, y, relu ? 1 : 0, static_cast<hipStream_t>(stream)));
}

int cast_f32_to_bf16(long count, const float *x, uint16_t *y, void *stream)
{
    if (count < 0) return MICONV_ERR_SHAPE;
    if (count > 0 && (!x || !y)) return MICONV_ERR_NULL;
    if ((uintptr_t)x % 4 || (uintptr_t)y % 2) return MICONV_ERR_ALIGN;
    return finish(launch_cast_bf16(count, x, y, static_cast<hipStream_t>(stream)));
}

int conv2d_describe(int N, int C, int H, int W, int K, int R, int S, int stride, int pad,
                    int groups, int dtype, int algo, int mode, char *buf, int buflen, int *launches)
{
    if (!buf || buflen <= 0 || !launches) return MICONV_ERR_NULL;
    buf[0] = 0;
    Resolved r;
    int rc = resolve_aligned(N, C, H, W, K, R, S, stride, pad, groups, dtype, algo, mode, nullptr, &r);
    if (rc != MICONV_OK) return rc;
    if (mode & MODE_PREPACK) set_packed(r, r.w);   // filters packed ahead: no packing launch
    describe(r, buf, buflen, launches);
    return MICONV_OK;
}

const char *miconv_strerror(int status)
{
    switch (status) {
    case MICONV_OK: return "ok";
    case MICONV_ERR_NULL: return "null tensor pointer";
    case MICONV_ERR_SHAPE: return "invalid shape, stride or padding (or empty output)";
    case MICONV_ERR_GROUPS: return "channel counts not divisible by groups (or not depthwise)";
    case MICONV_ERR_UNSUPPORTED: return "valid but unsupported configuration";
    case MICONV_ERR_TOO_LARGE: return "tensor exceeds 2^31-1 elements";
    case MICONV_ERR_ALIGN: return "pointer not aligned to its element size";
    case MICONV_ERR_HIP: return "HIP runtime error";
    case MICONV_ERR_WORKSPACE: return "workspace missing, too small or not 256-byte aligned for this plan";
    default: return "unknown status";
    }
}

int miconv_last_hip_error(void) { return g_last_hip_error; }

int miconv_version(void) { return 20000; }

}  // extern "C"
