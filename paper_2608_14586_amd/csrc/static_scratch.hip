// Fixed device scratch for the decode step that allocates nothing
// (vla_decode_step_static): one file-scope array per GPU, resolved to a
// device address once per device while that device is current.
//
// The array's name is a host-side stand-in in host code; every host use of
// its memory (kernel arguments, copies) goes through the address that
// hipGetSymbolAddress returned for the device.

#include <mutex>

#include "kernels.h"

namespace {

constexpr size_t kStaticScratchBytes = size_t(4) << 20;
constexpr int kMaxDevices = 64;

__device__ __align__(256) char scratch[kStaticScratchBytes];

std::mutex g_mu;
void* g_addr[kMaxDevices] = {};

}  // namespace

namespace vla {

size_t static_scratch_bytes() { return kStaticScratchBytes; }

hipError_t static_scratch_resolve(int device, void** out) {
  *out = nullptr;
  if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_addr[device]) {
    int cur = -1;
    hipError_t e = hipGetDevice(&cur);
    if (e != hipSuccess) return e;
    if (cur != device) return hipErrorInvalidDevice;  // the caller makes `device` current
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_addr[device] = p;
  }
  *out = g_addr[device];
  return hipSuccess;
}

}  // namespace vla
