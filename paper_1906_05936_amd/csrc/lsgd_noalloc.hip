// lsgd_lars_step_plan_noalloc: the LARS plan step for callers that cannot
// allocate device memory (code under HIP graph capture, serving loops,
// harnesses that forbid hipMalloc). Its scratch (the mean gradient, the
// per-chunk partial norms and the trust ratios of lsgd_lars_step_plan's
// workspace) is a library-owned array, one per device, instead of a
// caller-owned workspace; the kernels are the same.
#include <mutex>

#include "lsgd_host.hpp"

namespace lsgd {
namespace {

constexpr size_t kScratchBytes = LSGD_NOALLOC_SCRATCH_BYTES;
constexpr int kMaxScratchDevices = 64;

// Every device the library runs on holds its own copy of this array until the
// process ends. In host code `scratch` only names the array for
// hipGetSymbolAddress: kernels get the device address it returns.
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxScratchDevices];   // device address of `scratch`, per device (null until looked up)

// The device address of the current device's array, looked up once per device
// (with that device current) and kept.
lsgd_status scratch_for_current_device(void** out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return fail(LSGD_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
    if (dev < 0 || dev >= kMaxScratchDevices)
        return fail(LSGD_ERR_HIP, "device %d outside the %d devices this entry point serves", dev, kMaxScratchDevices);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            return fail(LSGD_ERR_HIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev, hipGetErrorString(e));
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return LSGD_OK;
}

}  // namespace
}  // namespace lsgd

extern "C" {

LSGD_API lsgd_status lsgd_lars_step_plan_noalloc(const lsgd_plan* plan, float lr, float momentum_coef,
                                                 float weight_decay, float trust_coef, float* trust_out,
                                                 const float* lr_device, void* stream) {
    if (!plan) return lsgd::fail(LSGD_ERR_NULL, "plan is NULL");
    size_t need = 0;
    lsgd_status st = lsgd_lars_workspace_size(plan, &need);
    if (st != LSGD_OK) return st;
    if (need > lsgd::kScratchBytes)
        return lsgd::fail(LSGD_ERR_SIZE,
                          "the plan's LARS scratch needs %zu bytes; lsgd_lars_step_plan_noalloc holds at most %zu "
                          "(LSGD_NOALLOC_SCRATCH_BYTES): use lsgd_lars_step_plan with a workspace",
                          need, lsgd::kScratchBytes);
    void* ws = nullptr;
    if ((st = lsgd::scratch_for_current_device(&ws)) != LSGD_OK) return st;
    return lsgd::lars_step(plan, lr, momentum_coef, weight_decay, trust_coef, ws, lsgd::kScratchBytes, true,
                           trust_out, lr_device, stream);
}

}  // extern "C"
