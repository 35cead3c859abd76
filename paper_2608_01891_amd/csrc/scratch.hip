// Library-owned device scratch for the entry points that allocate nothing.
//
// Callers that cannot allocate device memory (code under HIP graph capture,
// tight serving loops, harnesses that forbid hipMalloc) use the *_noalloc
// entry points, whose kernels take their scratch from this file-scope array
// instead of a caller workspace. Each device holds its own copy of the array
// from the time the library's code object is loaded on it until the process
// ends. In host code the array's name is only a host-side stand-in: its
// device address is looked up once per device with hipGetSymbolAddress (with
// that device current) and cached, and only that address is ever handed to
// a kernel.
#include <hip/hip_runtime.h>

#include <mutex>
#include <vector>

#include "kernels.h"

namespace aflex {

static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

namespace {
std::mutex g_scratch_mu;
std::vector<void*> g_scratch_ptr;  // per device: device address of `scratch`
}  // namespace

hipError_t static_scratch(void** ptr) {
  *ptr = nullptr;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if ((int)g_scratch_ptr.size() <= dev) g_scratch_ptr.resize(dev + 1, nullptr);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace aflex
