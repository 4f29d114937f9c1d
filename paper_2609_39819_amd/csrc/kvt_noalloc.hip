// The static scratch of kvt_extend_attention_noalloc.
//
// A file-scope device array holds the split-key partial results of that
// entry point, so it needs no device allocation.  Each GPU the library runs
// on holds its own copy until the process ends.  Host code never passes the
// array's name to a kernel (on the host the name is only a stand-in for the
// symbol, not a device address): the first call on a device, with that
// device current, looks up the copy's device address with
// hipGetSymbolAddress and keeps it per device; kernels receive that address.
// Every call on one GPU shares its copy, so calls that overlap on one GPU
// race; nothing in it needs to start at zero (every partial a combine reads
// is written first by the same call).
#include <hip/hip_runtime.h>

#include <atomic>

#include "kvt.h"
#include "kvt_internal.h"

namespace {

__device__ __attribute__((aligned(256))) unsigned char scratch[KVT_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch[kMaxDevices];

}  // namespace

namespace kvt {

hipError_t noalloc_scratch(void** ptr) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  void* p = g_scratch[dev].load(std::memory_order_acquire);
  if (p == nullptr) {
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    g_scratch[dev].store(p, std::memory_order_release);   // racing first calls store the same address
  }
  *ptr = p;
  return hipSuccess;
}

}  // namespace kvt
