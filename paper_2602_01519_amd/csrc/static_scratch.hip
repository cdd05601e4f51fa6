// Device memory the library owns without allocating: one file-scope array in
// the code object, which every GPU that loads the library holds (at its own
// address) until the process ends. The entry points that must not allocate
// put their tables and workspace here.
#include <hip/hip_runtime.h>

#include <mutex>

#include "pic_internal.hpp"

__device__ __align__(256) unsigned char scratch[pic::kStaticScratchBytes];

namespace pic {
namespace {
std::mutex g_mu;
void *g_addr[kMaxDevices];   // per device: the array's device address
}  // namespace

// The array's name is a host-side stand-in in host code; its device address
// on the current device comes from the runtime, resolved once per device.
hipError_t static_scratch(void **out) {
  *out = nullptr;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> g(g_mu);
  if (!g_addr[dev]) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_addr[dev] = p;
  }
  *out = g_addr[dev];
  return hipSuccess;
}

}  // namespace pic
