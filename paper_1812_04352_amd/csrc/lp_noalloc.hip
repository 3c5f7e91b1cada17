// Library-owned scratch memory for the allocation-free entry point
// (lp_residual_norm_noalloc): one fixed-size array in the code object's device
// memory, so each GPU the library runs on holds its own copy from the first
// call on it until the process ends. In host code the array's name is only a
// handle for the runtime, not a device address: its address on the current
// device is looked up once per device with hipGetSymbolAddress and cached, and
// only that address is ever handed to kernels.
#include <mutex>

#include "lp_internal.h"

namespace lp {
namespace {

// 2^21 fp64 residual partials plus one 256-byte-aligned slot for the result.
constexpr size_t kScratchBytes = ((size_t)16 << 20) + 256;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

}  // namespace

size_t noalloc_scratch_bytes() { return kScratchBytes; }

hipError_t noalloc_scratch(void** ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace lp
