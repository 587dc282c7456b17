// Device-resident scratch of the allocation-free profile entry point
// (rk_sensitivity_profile_static): a file-scope device array that the code
// object brings along, so that entry point needs no workspace argument and
// calls no allocator.  Every GPU the library runs on holds its own copy for the
// life of the process.
//
// In host code `scratch` names a host-side stand-in, not device memory: kernels
// receive the device address that hipGetSymbolAddress reports for the current
// device, looked up once per device and kept.
#include <mutex>

#include "rk_internal.h"

namespace rk {

static __device__ __align__(256) unsigned char scratch[RK_STATIC_SCRATCH_BYTES];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_addr[kMaxDevices] = {};
}  // namespace

hipError_t static_scratch(hipStream_t stream, void** out) {
  *out = nullptr;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (stream) {   // the stream's device must be the current one: the address differs per device
    int sdev = -1;
    e = hipStreamGetDevice(stream, &sdev);
    if (e != hipSuccess) return e;
    if (sdev != dev) return hipErrorInvalidDevice;
  }
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p || ((uintptr_t)p & 255)) return hipErrorInvalidSymbol;
    g_addr[dev] = p;
  }
  *out = g_addr[dev];
  return hipSuccess;
}

}  // namespace rk
