// Route prediction that allocates nothing: the router's bf16 weight split lives
// in a file-scope device array instead of a caller workspace, for callers that
// cannot allocate device memory (code under HIP graph capture, tight serving
// loops).  Same kernels and results as pr2_route_predict.
#include <map>
#include <mutex>

#include "common.h"

namespace pr2 {
namespace {

// One copy on each GPU the library runs on, held until the process ends.  In
// host code the name is a host-side stand-in, never a device address: the
// address of a device's copy is looked up once, with that device current, and
// only that pointer reaches kernels.
constexpr size_t kNoAllocScratchBytes = (size_t)6 << 20;
__device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

pr2_status noalloc_scratch(void** out) {
    static std::mutex mu;
    static std::map<int, void*> per_dev;       // device -> address of its copy of scratch
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) {
        (void)hipGetLastError();
        return fail(PR2_ERR_DEVICE, "no usable HIP device");
    }
    std::lock_guard<std::mutex> lk(mu);
    auto it = per_dev.find(dev);
    if (it == per_dev.end()) {
        void* p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || p == nullptr) {
            (void)hipGetLastError();
            return fail(PR2_ERR_HIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev,
                        hipGetErrorString(e));
        }
        it = per_dev.emplace(dev, p).first;
    }
    *out = it->second;
    return PR2_OK;
}

}  // namespace
}  // namespace pr2

using namespace pr2;

extern "C" pr2_status pr2_route_predict_noalloc(const pr2_moe_desc* desc, const void* x,
                                                const float* W_r, const float* b_r,
                                                const float* A, const float* B, void* idx_out,
                                                int64_t ldi, float* gate_out, float* logits_out,
                                                pr2_stream_t stream) {
    bool empty = false;
    pr2_status s = check_route_args(desc, x, W_r, b_r, A, B, idx_out, ldi, gate_out, logits_out,
                                    &empty);
    if (s != PR2_OK) return s;
    if (empty) return ok();
    const pr2_moe_desc& d = *desc;
    // the split this call forms: the predictor folded into N columns when no logits
    // are wanted, [W_r | A] otherwise, none on the fp64 vector path.  The fused
    // router kernel reads only the split (no split-K partial sums at any batch size).
    size_t need = 0;
    if (logits_out == nullptr && router_mfma_ok(d, d.N)) need = router_split_weight_bytes(d.N, d);
    else if (router_mfma_ok(d, d.N + d.r)) need = router_split_weight_bytes(d.N + d.r, d);
    if (need > kNoAllocScratchBytes)
        return fail(PR2_ERR_UNSUPPORTED, "the weight split needs %zu bytes, more than the %zu "
                    "bytes of the no-allocation scratch", need, kNoAllocScratchBytes);
    s = device_ready();
    if (s != PR2_OK) return s;
    void* ptr = nullptr;
    if (need) {
        s = noalloc_scratch(&ptr);
        if (s != PR2_OK) return s;
    }
    const hipError_t e = launch_route_predict(d, x, W_r, b_r, A, B, idx_out, ldi, gate_out,
                                              logits_out, ptr, (hipStream_t)stream,
                                              FeatureCache{}, false, false);
    if (e != hipSuccess) return hip_fail(e, "route_predict launch");
    return ok();
}
