// conv2d_fwd_noalloc: conv2d_fwd_ws for callers that cannot allocate device
// memory at all (code under HIP graph capture, tight serving loops, harnesses
// that forbid hipMalloc).  The workspace is a fixed array in the library's
// device code object, `scratch`, one copy per GPU, held from the first use on
// that GPU until the process ends.
//
// In host code `scratch` names a host-side stand-in, not device memory: its
// device address is looked up once per device with hipGetSymbolAddress (with
// that device current) and only that address is ever handed to kernels.
#include "../../include/miconv.h"
#include "internal.h"

#include <map>
#include <mutex>

namespace {

constexpr size_t kScratchBytes = MICONV_NOALLOC_SCRATCH_BYTES;

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

// The device address of `scratch` on the current device, looked up on the
// first call there.
int scratch_address(void **out)
{
    static std::mutex mu;
    static std::map<int, void *> addr;
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return miconv::set_hip_error(e);
    std::lock_guard<std::mutex> lk(mu);
    auto it = addr.find(dev);
    if (it == addr.end()) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return miconv::set_hip_error(e);
        if (!p || (uintptr_t)p % 256) return MICONV_ERR_HIP;
        it = addr.emplace(dev, p).first;
    }
    *out = it->second;
    return MICONV_OK;
}

}  // namespace

extern "C" int conv2d_fwd_noalloc(int N, int C, int H, int W, int K, int R, int S, int stride, int pad,
                                  int groups, int dtype, int algo, const void *x, const void *w,
                                  const float *bias, const float *res, float *y, long y_image_stride,
                                  int relu, void *stream)
{
    miconv::Resolved r;
    int rc = miconv::resolve_ex(miconv::MODE_SCRATCH, N, C, H, W, K, R, S, stride, pad, groups, dtype, algo,
                                x, w, bias, res, y, y_image_stride, relu, &r);
    if (rc != MICONV_OK) return rc;
    const size_t need = miconv::workspace_bytes(r);
    if (need > kScratchBytes) return MICONV_ERR_WORKSPACE;   // beyond the fixed scratch
    void *ws = nullptr;
    if (need && (rc = scratch_address(&ws)) != MICONV_OK) return rc;
    return miconv::run(r, ws, kScratchBytes, static_cast<hipStream_t>(stream));
}
