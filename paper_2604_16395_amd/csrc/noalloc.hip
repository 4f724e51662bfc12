// Library-held scratch memory for the allocation-free attention call
// (s2l_chunk_prefill_attn_noalloc): the plan and the split partials live in a file-scope
// device array instead of a caller workspace, for callers that cannot allocate.
//
// Every GPU the library runs on holds its own copy of the array, from the moment the code
// object is loaded on that device until the process ends.  In host code the array's name is
// only a host-side stand-in; its device address is taken once per device, with that device
// current, by hipGetSymbolAddress, and only that address is ever handed to kernels.
#include <hip/hip_runtime.h>

#include <mutex>

#include "launch.h"

namespace s2l {

namespace {

static __device__ __align__(256) uint8_t scratch[kNoAllocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];   // device address of `scratch` on each device, once taken

}  // namespace

hipError_t noalloc_scratch(void** ptr) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace s2l
