// Fixed device scratch for the entry point that allocates nothing.
//
// The array lives in the library's code object: each GPU the library runs
// on holds its own copy, from the moment the code object is loaded there
// until the process ends.  In host code `scratch` names a host-side
// stand-in, not device memory; the device address of each GPU's copy comes
// from hipGetSymbolAddress, called once per device with that device current,
// and only that address is ever handed to kernels or copies.
#include <hip/hip_runtime.h>

#include <mutex>

#include "eb_internal.h"

namespace eb {

static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_mu;
void *g_addr[kMaxDevices] = {};
}  // namespace

hipError_t noalloc_scratch_setup(int device, void **addr) {
  *addr = nullptr;
  if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_addr[device]) {
    void *p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_addr[device] = p;
  }
  *addr = g_addr[device];
  return hipSuccess;
}

}  // namespace eb
