// pgc_step_noalloc: the linear models' step with the gradient kernel's block
// partial sums in a fixed, library-owned device array instead of the bound
// workspace, for callers that cannot allocate device memory.
#include <hip/hip_runtime.h>

#include <mutex>
#include <string>

#include "pgc.h"
#include "pgc_step.h"

// The array every pgc_step_noalloc call on a device shares.  In host code its
// name is only a host-side stand-in; kernels get its device address, looked up
// once per device with hipGetSymbolAddress.
static __device__ __align__(256) float scratch[PGC_NOALLOC_SCRATCH_BYTES / sizeof(float)];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_lock;
void* g_scratch[kMaxDevices] = {};

// Device address of the current device's scratch array (looked up on the
// first call on that device, with the device current).
hipError_t scratch_ptr(float** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> hold(g_lock);
  if (g_scratch[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    g_scratch[dev] = p;
  }
  *out = static_cast<float*>(g_scratch[dev]);
  return hipSuccess;
}

}  // namespace

extern "C" int pgc_step_noalloc(pgc_ctx* ctx, const void* X, const void* y, float* w,
                                const uint8_t* straggler_mask, float lr) {
  if (ctx == nullptr) return PGC_EINVAL;
  if (!pgc::context_is_configured(ctx)) return pgc::set_error(ctx, PGC_ESTATE, "pgc_configure first");
  if (!pgc::context_is_linear(ctx))
    return pgc::set_error(ctx, PGC_EINVAL, "pgc_step_noalloc runs the linear models only (PGC_LOGISTIC, PGC_LSQ)");
  const size_t need = pgc::linear_partials_bytes(ctx);
  if (need > PGC_NOALLOC_SCRATCH_BYTES) {
    const std::string msg = "pgc_step_noalloc: the gradient's block partials need " + std::to_string(need) +
                            " bytes, more than the fixed scratch of " +
                            std::to_string(static_cast<size_t>(PGC_NOALLOC_SCRATCH_BYTES)) + " bytes";
    return pgc::set_error(ctx, PGC_EINVAL, msg.c_str());
  }
  if (!pgc::context_has_workspace(ctx)) return pgc::set_error(ctx, PGC_ESTATE, "pgc_bind_workspace first");
  float* partials = nullptr;
  const hipError_t e = scratch_ptr(&partials);
  if (e != hipSuccess) {
    const std::string msg = std::string("locating the scratch array: ") + hipGetErrorString(e);
    return pgc::set_error(ctx, PGC_EDEVICE, msg.c_str());
  }
  return pgc::step_impl(ctx, X, y, w, straggler_mask, lr, partials);
}
