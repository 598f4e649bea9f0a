// The reparameterized backward with the library's own scratch memory, for
// callers that cannot allocate device memory.  The factor gradient's partial
// sums over token splits live in a file-scope device array; every GPU holds
// its own copy, whose address is looked up once per device.
#include <hip/hip_runtime.h>

#include <mutex>

#include "ssn.h"
#include "ssn_checks.h"

namespace {

// The device array.  In host code this name is only a handle for
// hipGetSymbolAddress, never a device address: kernels receive the pointer
// that lookup returns.
static __device__ __align__(256) unsigned char scratch[SSN_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_scratch[kMaxDevices];   // device address of `scratch` on each device, once looked up

// Address of this device's copy of `scratch` (the current device), looked up
// on the first call on that device.
ssn_status_t scratch_of_current_device(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return SSN_ERR_LAUNCH;
  std::lock_guard<std::mutex> lock(g_mu);
  if (g_scratch[dev] == nullptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr)
      return SSN_ERR_LAUNCH;
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return SSN_OK;
}

}  // namespace

extern "C" ssn_status_t ssn_reparam_backward_noalloc(ssn_dtype_t dtype, int64_t N, int64_t din,
                                                     int64_t d, int64_t k, const void* H,
                                                     const void* Zp, const void* U, const void* G,
                                                     float* GT, void* GH, float* GZp,
                                                     void* stream) {
  // every argument is checked before the first HIP call
  const ssn_status_t chk = ssn::reparam_backward_args(dtype, N, din, d, k, H, Zp, U, G, GT, GH, GZp,
                                                      nullptr, 0, false);
  if (chk != SSN_OK) return chk;
  const size_t need = ssn_reparam_workspace_bytes(dtype, N, din, k);
  if (need > (size_t)SSN_NOALLOC_SCRATCH_BYTES) return SSN_ERR_UNSUPPORTED;
  void* ws = nullptr;
  const ssn_status_t sst = scratch_of_current_device(&ws);
  if (sst != SSN_OK) return sst;
  return ssn_reparam_backward(dtype, N, din, d, k, H, Zp, U, G, GT, GH, GZp, ws,
                              (size_t)SSN_NOALLOC_SCRATCH_BYTES, stream);
}
