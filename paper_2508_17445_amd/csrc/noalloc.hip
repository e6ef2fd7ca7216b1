// Device scratch of the decode entry point that allocates nothing
// (treepo_tree_decode_noalloc): the plan image and the partial slots of a
// decode live in one file-scope device array instead of library-allocated
// memory and a caller workspace.  Each device the library runs on holds its
// own copy of the array, for the life of the process.
#include <hip/hip_runtime.h>

#include <mutex>

#include "kernels.h"

namespace {

static __device__ __align__(256) char scratch[treepo::kNoAllocScratchBytes];

constexpr int kMaxDevices = 64;

struct DeviceScratch {
  void* ptr = nullptr;   // the array's device address on this device
  uint64_t holder = 0;   // id of the plan image it holds (0: none)
};

DeviceScratch g_scratch[kMaxDevices];
std::mutex g_lock;

}  // namespace

namespace treepo {

hipError_t noalloc_scratch(void** ptr, uint64_t** holder) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> g(g_lock);
  DeviceScratch& s = g_scratch[dev];
  if (!s.ptr) {
    // The array's name is a host-side stand-in; its address on this device
    // (current at this call) comes from the runtime, once per device.
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p || reinterpret_cast<uintptr_t>(p) % 256 != 0) return hipErrorInvalidSymbol;
    s.ptr = p;
  }
  *ptr = s.ptr;
  *holder = &s.holder;
  return hipSuccess;
}

}  // namespace treepo
