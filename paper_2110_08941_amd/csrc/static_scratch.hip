// The device buffer behind hs_workers_grad_static: a file-scope device array
// of HS_STATIC_SCRATCH_BYTES bytes, which every GPU that loads the library
// holds until the process ends.  Host code never passes the array's name to
// a kernel (on the host it is a stand-in, not a device address): the address
// is looked up once per device with hipGetSymbolAddress, with that device
// current, and kept per device.
#include <hip/hip_runtime.h>

#include <mutex>

#include "../../include/hs.h"
#include "model.h"

namespace {

static __device__ __align__(256) char scratch[HS_STATIC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_addr[kMaxDevices] = {};

}  // namespace

namespace hs {

hipError_t static_scratch(void** ptr) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_addr[dev] = p;
  }
  *ptr = g_addr[dev];
  return hipSuccess;
}

}  // namespace hs
