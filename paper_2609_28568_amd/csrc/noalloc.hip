// Scratch memory of the entry points that allocate nothing: a file-scope
// device array, of which every GPU the library runs on holds its own copy
// until the process ends. Its device address is looked up once per device
// (with that device current) and kept; host code uses only that address,
// never the array's name, which on the host is a stand-in and not a device
// pointer.
#include <mutex>

#include "common.h"
#include "kernels.h"

static __device__ __align__(256) float scratch[NOALLOC_SCRATCH_FLOATS];

namespace {
constexpr int MAX_DEVICES = 64;
std::mutex g_mu;
float* g_scratch[MAX_DEVICES] = {};
}  // namespace

hipError_t noalloc_scratch(float** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= MAX_DEVICES) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch[dev] = static_cast<float*>(p);
  }
  *out = g_scratch[dev];
  return hipSuccess;
}
