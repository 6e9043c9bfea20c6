// The C ABI of libmiconv (include/miconv.h): argument validation, output
// extents, the shape -> kernel choice, and the per-stream split-K workspace.
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
#include <utility>

namespace miconv {

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
    return MICONV_OK;
}

int check_bias(const float *bias)
{
    return (bias && (uintptr_t)bias % sizeof(float)) ? MICONV_ERR_ALIGN : MICONV_OK;
}

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

// Split-K workspace, one per (device, stream): an array of per-tile arrival
// counters (zeroed once when allocated; every launch leaves them at zero)
// followed by the fp32 partial sums.
struct Workspace {
    void *ptr = nullptr;
    size_t counter_bytes = 0;
    size_t partial_bytes = 0;
};

size_t round_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

int get_workspace(hipStream_t st, const IgemmPlan &plan, float **partials, int **counters)
{
    static std::mutex mu;
    static std::map<std::pair<int, hipStream_t>, Workspace> table;
    *partials = nullptr;
    *counters = nullptr;
    if (plan.splits <= 1) return MICONV_OK;
    const size_t need_c = round_up((size_t)plan.counters * sizeof(int), 256);
    const size_t need_p = round_up(plan.ws_bytes, 256);
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e);
    std::lock_guard<std::mutex> lk(mu);
    Workspace &ws = table[{dev, st}];
    if (ws.counter_bytes < need_c || ws.partial_bytes < need_p) {
        const size_t cb = std::max(std::max(need_c, ws.counter_bytes), (size_t)16384);
        const size_t pb = std::max(std::max(need_p, ws.partial_bytes), (size_t)(1u << 20));
        if (ws.ptr) {
            // Kernels already queued on this stream may still use the old buffer.
            e = hipStreamSynchronize(st);
            if (e != hipSuccess) return hip_fail(e);
            e = hipFree(ws.ptr);
            if (e != hipSuccess) return hip_fail(e);
            ws = Workspace{};
        }
        void *ptr = nullptr;
        e = hipMalloc(&ptr, cb + pb);
        if (e != hipSuccess) return hip_fail(e);
        e = hipMemset(ptr, 0, cb);
        if (e != hipSuccess) {
            hipFree(ptr);
            return hip_fail(e);
        }
        ws.ptr = ptr;
        ws.counter_bytes = cb;
        ws.partial_bytes = pb;
    }
    *counters = static_cast<int *>(ws.ptr);
    *partials = reinterpret_cast<float *>(static_cast<char *>(ws.ptr) + ws.counter_bytes);
    return MICONV_OK;
}

int finish(hipError_t e) { return e == hipSuccess ? MICONV_OK : hip_fail(e); }

int run_igemm_f32(const ConvProblem &p, const float *x, const float *w, const float *bias, float *y,
                  hipStream_t st)
{
    const IgemmPlan plan = plan_igemm_f32(p, cu_count());
    float *ws = nullptr;
    int *counters = nullptr;
    int rc = get_workspace(st, plan, &ws, &counters);
    if (rc != MICONV_OK) return rc;
    return finish(launch_igemm_f32(p, plan, x, w, bias, y, ws, counters, st));
}

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
    ConvProblem p;
    int rc = validate(N, C, H, W, K, R, S, stride, pad, groups, x, w, y, sizeof(float), &p);
    if (rc != MICONV_OK) return rc;
    if ((rc = check_bias(bias)) != MICONV_OK) return rc;
    if (algo < MICONV_ALGO_AUTO || algo > MICONV_ALGO_IGEMM) return MICONV_ERR_UNSUPPORTED;
    p.relu = relu ? 1 : 0;
    hipStream_t st = static_cast<hipStream_t>(stream);
    const bool depthwise = groups > 1 && groups == C && K == C;
    if (algo == MICONV_ALGO_AUTO) {
        if (depthwise && R <= 7 && S <= 7) return finish(launch_dwconv_f32(p, x, w, bias, y, st));
        algo = (groups == 1 || p.Cg >= 8) ? MICONV_ALGO_IGEMM : MICONV_ALGO_DIRECT;
    }
    if (algo == MICONV_ALGO_DIRECT) return finish(launch_conv_direct_f32(p, x, w, bias, y, st));
    return run_igemm_f32(p, x, w, bias, y, st);
}

int conv2d_fwd(int N, int C, int H, int W, int K, int R, int S, int stride, int pad, int groups,
               const float *x, const float *w, const float *bias, float *y, int relu, void *stream)
{
    return conv2d_fwd_algo(N, C, H, W, K, R, S, stride, pad, groups, x, w, bias, y, relu,
                           MICONV_ALGO_AUTO, stream);
}

int conv2d_fwd_bf16(int N, int C, int H, int W, int K, int R, int S, int stride, int pad,
                    int groups, const uint16_t *x, const uint16_t *w, const float *bias, float *y,
                    int relu, void *stream)
{
    ConvProblem p;
    int rc = validate(N, C, H, W, K, R, S, stride, pad, groups, x, w, y, sizeof(uint16_t), &p);
    if (rc != MICONV_OK) return rc;
    if ((rc = check_bias(bias)) != MICONV_OK) return rc;
    p.relu = relu ? 1 : 0;
    hipStream_t st = static_cast<hipStream_t>(stream);
    return finish(launch_conv_direct_bf16(p, x, w, bias, y, st));
}

int dwconv2d_fwd(int N, int C, int H, int W, int K, int R, int S, int stride, int pad, int groups,
                 const float *x, const float *w, const float *bias, float *y, int relu,
                 void *stream)
{
    ConvProblem p;
    int rc = validate(N, C, H, W, K, R, S, stride, pad, groups, x, w, y, sizeof(float), &p);
    if (rc != MICONV_OK) return rc;
    if ((rc = check_bias(bias)) != MICONV_OK) return rc;
    if (groups != C || K != C) return MICONV_ERR_GROUPS;
    if (R > 7 || S > 7) return MICONV_ERR_UNSUPPORTED;
    p.relu = relu ? 1 : 0;
    return finish(launch_dwconv_f32(p, x, w, bias, y, static_cast<hipStream_t>(stream)));
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
                    int groups, int dtype, int algo, char *buf, int buflen, int *launches)
{
    if (!buf || buflen <= 0 || !launches) return MICONV_ERR_NULL;
    buf[0] = 0;
    static const float dummy[4] = {0, 0, 0, 0};
    ConvProblem p;
    int rc = validate(N, C, H, W, K, R, S, stride, pad, groups, dummy, dummy, dummy,
                      dtype == 1 ? sizeof(uint16_t) : sizeof(float), &p);
    if (rc != MICONV_OK) return rc;
    if (dtype != 0 && dtype != 1) return MICONV_ERR_UNSUPPORTED;
    if (algo < MICONV_ALGO_AUTO || algo > MICONV_ALGO_IGEMM) return MICONV_ERR_UNSUPPORTED;
    if (dtype == 1) {
        describe_direct(1, buf, buflen, launches);
        return MICONV_OK;
    }
    const bool depthwise = groups > 1 && groups == C && K == C;
    if (algo == MICONV_ALGO_AUTO) {
        if (depthwise && R <= 7 && S <= 7) {
            describe_dwconv(p, buf, buflen, launches);
            return MICONV_OK;
        }
        algo = (groups == 1 || p.Cg >= 8) ? MICONV_ALGO_IGEMM : MICONV_ALGO_DIRECT;
    }
    if (algo == MICONV_ALGO_DIRECT) {
        describe_direct(0, buf, buflen, launches);
        return MICONV_OK;
    }
    describe_igemm_f32(p, plan_igemm_f32(p, cu_count()), buf, buflen, launches);
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
    default: return "unknown status";
    }
}

int miconv_last_hip_error(void) { return g_last_hip_error; }

int miconv_version(void) { return 100; }

}  // extern "C"
