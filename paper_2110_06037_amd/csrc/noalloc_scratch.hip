// Static device memory for the allocation-free run (sn_run_noalloc): one
// region of kNoallocScratchBytes per GPU, defined in the library's code
// object, so callers that may not allocate (code under HIP graph capture,
// tight serving loops) can still run a plan whose intermediate tensors and
// workspaces fit in it.
//
// In host code the array's name is only a host-side handle of the device
// variable, never an address: the device address comes from
// hipGetSymbolAddress, taken once per device with that device current, and
// only that address is ever passed to kernels.  Each GPU holds its own copy
// at its own address until the process ends.
#include <hip/hip_runtime.h>

#include <map>
#include <mutex>
#include <string>

#include "core.hpp"

namespace sn {

constexpr size_t kNoallocScratchBytes = size_t(64) << 20;

static __device__ __align__(256) char scratch[kNoallocScratchBytes];

size_t noalloc_scratch_bytes() { return kNoallocScratchBytes; }

// Device address of `scratch` on the current device (looked up on the first
// call per device and kept).
void* noalloc_scratch_ptr(int device) {
  static std::mutex mu;
  static std::map<int, void*> ptrs;
  std::lock_guard<std::mutex> lock(mu);
  auto it = ptrs.find(device);
  if (it != ptrs.end()) return it->second;
  int cur = -1;
  hipError_t e = hipGetDevice(&cur);
  if (e != hipSuccess || cur != device) fail(SN_E_DEVICE, "scratch lookup needs the graph's device current");
  void* ptr = nullptr;
  e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
  if (e != hipSuccess || !ptr)
    fail(SN_E_DEVICE, std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e));
  ptrs[device] = ptr;
  return ptr;
}

}  // namespace sn
