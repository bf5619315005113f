// Library-owned scratch memory of the allocation-free entry point
// (moe_route_count_noalloc): a file-scope device array, one copy per GPU,
// held until the process ends.  Host code never passes the array's name to
// a kernel (on the host it is only a stand-in for the symbol); it looks the
// device address up once per device with hipGetSymbolAddress and passes that.
#include <hip/hip_runtime.h>

#include <mutex>

#include "internal.hpp"

namespace laep {
namespace {

constexpr int kMaxScratchDevices = 64;

static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxScratchDevices];

}  // namespace

hipError_t noalloc_scratch(void** out) {
  *out = nullptr;
  int dev = 0;
  hipError_t err = hipGetDevice(&dev);
  if (err != hipSuccess) return err;
  if (dev < 0 || dev >= kMaxScratchDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (err != hipSuccess) return err;
    if (p == nullptr) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace laep
