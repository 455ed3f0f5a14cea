// Library-owned scratch for the entry point that allocates nothing
// (mssa_attention_noalloc): the workspace of mssa_pool_kv / mssa_forward as
// one file-scope device array.  Every GPU the library runs on holds its own
// copy at its own address from the time the code object is loaded until the
// process ends.  Host code never uses the array's name as an address: the
// address of the current device's copy comes from hipGetSymbolAddress, taken
// once per device and kept.
#include <hip/hip_runtime.h>

#include <mutex>

#include "noalloc.hpp"

namespace mssa {
namespace {

__device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mutex;
void* g_scratch_ptr[kMaxDevices] = {};

}  // namespace

hipError_t scratch_address(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mutex);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!ptr) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace mssa
