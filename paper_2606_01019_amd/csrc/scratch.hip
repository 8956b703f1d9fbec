// Static device scratch of the allocation-free verify entry point
// (hvd_verify_noalloc): one file-scope array per GPU, sized kStaticScratchBytes,
// which each GPU the library runs on holds until the process ends.
//
// In host code `scratch` names a host-side stand-in, not device memory, so
// host code never passes it anywhere: static_scratch() takes the array's
// device address with hipGetSymbolAddress once per device (with that device
// current) and every host use goes through that address.
#include <mutex>

#include "kernels.h"

namespace hvd {

static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};
}  // namespace

hipError_t static_scratch(void** out, size_t* bytes) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  *bytes = kStaticScratchBytes;
  return hipSuccess;
}

}  // namespace hvd
