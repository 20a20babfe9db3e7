// static_ws.hip -- lora_linear_bwd for callers that cannot allocate device
// memory: the workspace is a file-scope device array of the library (one
// copy per GPU, held until the process ends) instead of a caller buffer.
#include <hip/hip_runtime.h>

#include <mutex>

#include "../../include/lora_mi355x.h"
#include "launch.hpp"

namespace {

constexpr size_t kScratchBytes = size_t(LORA_NOALLOC_SCRATCH_BYTES);
constexpr int kMaxDevices = 64;

}  // namespace

// The backward's workspace for lora_linear_bwd_noalloc.  In host code this
// name is only a stand-in for the symbol: kernels get the device address that
// hipGetSymbolAddress returns for the current device (scratch_ptr).
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

std::mutex g_mu;
void *g_ptr[kMaxDevices] = {};

// Device address of `scratch` on the current device, looked up once per
// device (each GPU holds its own copy of the array at its own address).
hipError_t scratch_ptr(void **out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_ptr[dev]) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_ptr[dev] = p;
  }
  *out = g_ptr[dev];
  return hipSuccess;
}

}  // namespace

extern "C" lora_status_t lora_linear_bwd_noalloc(const void *x, const void *W, const void *A,
                                                 const void *B, const float *u_saved, const void *dy,
                                                 void *dx, float *dA, float *dB, int64_t T,
                                                 int64_t d_in, int64_t d_out, int64_t r, float scale,
                                                 lora_dtype_t dt, void *hip_stream) {
  const size_t need = lora_linear_workspace_bytes(LORA_OP_BWD, T, d_in, d_out, r, dt);
  if (need == (size_t)-1)  // sizes the entry point rejects: let it report why
    return lora_linear_bwd(x, W, A, B, u_saved, dy, dx, dA, dB, T, d_in, d_out, r, scale, dt, nullptr, 0,
                           hip_stream);
  if (need > kScratchBytes) {
    lora::set_last_error("workspace needed exceeds the static scratch (LORA_NOALLOC_SCRATCH_BYTES)");
    return LORA_EWORKSPACE;
  }
  void *ws = nullptr;
  if (need > 0) {
    const hipError_t e = scratch_ptr(&ws);
    if (e != hipSuccess) {
      lora::set_last_error("hipGetSymbolAddress of the static scratch failed");
      return LORA_EHIP;
    }
  }
  return lora_linear_bwd(x, W, A, B, u_saved, dy, dx, dA, dB, T, d_in, d_out, r, scale, dt, ws,
                         need > 0 ? kScratchBytes : 0, hip_stream);
}
