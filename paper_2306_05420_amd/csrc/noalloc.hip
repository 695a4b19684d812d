// The layer with a library-owned workspace: spin_sph_conv_forward_noalloc.
//
// For callers that cannot allocate device memory (code under graph capture,
// tight serving loops, harnesses that forbid hipMalloc), the layer's
// workspace is a file-scope device array of fixed size.  Each device that
// loads the library holds its own copy at its own address until the process
// ends; host code reaches it only through the address hipGetSymbolAddress
// returns on that device (the array's name in host code is a host-side
// stand-in, not a device address).  The address is looked up once per device
// when a plan is created there, so the entry point itself makes no runtime
// call besides its kernel launches.
#include <mutex>

#include "swsft_internal.h"

namespace swsft {
namespace {

__device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_scratch[kMaxDevices] = {};

}  // namespace

hipError_t register_scratch(int device) {
  if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mu);
  if (g_scratch[device] != nullptr) return hipSuccess;
  void* ptr = nullptr;
  const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
  if (e != hipSuccess) return e;
  g_scratch[device] = ptr;
  return hipSuccess;
}

void* scratch_of(int device) {
  if (device < 0 || device >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_mu);
  return g_scratch[device];
}

}  // namespace swsft
