// Device-resident scratch for dmoe_expert_ffn_noalloc: the SwiGLU activations
// between the FFN's two kernels live in a file-scope device array instead of
// a caller workspace, for callers that cannot allocate device memory.
//
// Each GPU the library runs on holds its own copy of the array, at its own
// address, until the process ends.  In host code the array's name is only a
// stand-in for the symbol: its device address is looked up once per device
// (hipGetSymbolAddress, with that device current) and only that address is
// ever passed to kernels.
#include <mutex>

#include "dmoe_common.h"

namespace dmoe {
namespace {

__device__ __align__(256) unsigned char scratch[DMOE_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_ptr[kMaxDevices] = {};

}  // namespace

hipError_t noalloc_scratch(void** ptr) {
  int dev = 0;
  hipError_t err = hipGetDevice(&dev);
  if (err != hipSuccess) return err;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_ptr[dev]) {
    void* p = nullptr;
    err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (err != hipSuccess) return err;
    if (!p) return hipErrorInvalidSymbol;
    g_ptr[dev] = p;
  }
  *ptr = g_ptr[dev];
  return hipSuccess;
}

}  // namespace dmoe
