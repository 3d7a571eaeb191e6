// thin_compress_static: the compress path over a workspace that is a static
// device array instead of a caller's buffer, for callers that cannot
// allocate device memory.
#include <mutex>

#include "../../include/thin.h"
#include "launch.hpp"

namespace {

// The workspace of thin_compress_static.  Each GPU holds its own copy from
// the time the library's code is loaded on it until the process ends; calls
// on one GPU share it.
static __device__ __align__(256) unsigned char scratch[THIN_STATIC_SCRATCH_BYTES];

// Device address of `scratch` on every device, taken once per device with
// that device current (the host-side name `scratch` is not a device address).
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices];

hipError_t scratch_on_current_device(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return hipSuccess;
}

}  // namespace

extern "C" int thin_compress_static(const void* K, const void* V, int32_t dtype, int64_t B,
                                    int64_t H, int64_t n, int64_t d, int64_t n_out, int32_t g,
                                    const float* uniforms, int64_t n_uniforms, int32_t* idx_out,
                                    int32_t* status, void* stream) {
  // sizes first: a call that cannot fit touches no device
  size_t need = 0;
  int rc = thin::compress_fixed(K, V, dtype, B, H, n, d, n_out, g, uniforms, n_uniforms, idx_out,
                                nullptr, THIN_STATIC_SCRATCH_BYTES, &need, stream);
  if (rc != THIN_OK) return rc;
  void* ws = nullptr;
  if (scratch_on_current_device(&ws) != hipSuccess) return THIN_EHIP;
  rc = thin::compress_fixed(K, V, dtype, B, H, n, d, n_out, g, uniforms, n_uniforms, idx_out, ws,
                            THIN_STATIC_SCRATCH_BYTES, &need, stream);
  if (rc != THIN_OK || !status) return rc;
  // the call's status word (first word of the workspace) into the caller's
  // buffer, ordered after the call's kernels
  const hipError_t e = hipMemcpyAsync(status, ws, sizeof(int32_t), hipMemcpyDeviceToDevice,
                                      static_cast<hipStream_t>(stream));
  return e == hipSuccess ? THIN_OK : THIN_EHIP;
}
