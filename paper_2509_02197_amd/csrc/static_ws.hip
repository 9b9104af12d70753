// The workspace of adst_vjp_static_ws: a file-scope device array, one copy
// per GPU, for callers that cannot allocate device memory. Host code never
// passes the array's name to a kernel (in host code it names a host-side
// stand-in, not device memory); it looks up each device's address once, with
// that device current, and uses that address everywhere.

#include <hip/hip_runtime.h>

#include <mutex>
#include <vector>

#include "kernels.h"

namespace adst {
namespace {

__device__ __align__(256) unsigned char scratch[kStaticWsBytes];

std::mutex g_mutex;
std::vector<void*> g_addr;  // per device ordinal; null until looked up

}  // namespace

hipError_t static_workspace(void** ptr) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lock(g_mutex);
  if (dev < 0) return hipErrorInvalidDevice;
  if ((size_t)dev >= g_addr.size()) g_addr.resize(dev + 1, nullptr);
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

}  // namespace adst
