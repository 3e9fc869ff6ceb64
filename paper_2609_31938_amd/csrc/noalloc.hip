// Device scratch of the allocation-free entry point
// (c3c_conv3d_causal_cached_noalloc): the fp32 split-K partial sums of a
// call that splits its stages live in this file-scope array instead of a
// caller workspace, so the call needs no device allocation at all.
//
// The array exists once per device the library runs on, at a different
// address on each.  Host code never uses the array's name as an address (on
// the host it is only a stand-in for the symbol): the device address is
// looked up with hipGetSymbolAddress on the entry point's first call on each
// device, with that device current, and kept per device.
#include <mutex>

#include "c3c_internal.h"

namespace c3c {
namespace {

static __device__ __align__(256) unsigned char scratch[kNoallocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_addr[kMaxDevices];  // device address of `scratch` per device (NULL: not looked up)

}  // namespace

hipError_t noalloc_scratch(void** ptr) {
  *ptr = nullptr;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mu);
  if (g_addr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr || (reinterpret_cast<uintptr_t>(p) & 255u) != 0) return hipErrorInvalidSymbol;
    g_addr[dev] = p;
  }
  *ptr = g_addr[dev];
  return hipSuccess;
}

}  // namespace c3c
