// Fixed device scratch memory for the entry point that allocates nothing
// (higgs_qmatmul_fused_noalloc): callers under stream capture, in tight
// serving loops or in harnesses that forbid allocation cannot hand the
// product a workspace, so the library brings one of its own.
//
// The array below lives in the library's code object: every device the
// library runs on holds its own copy (kScratchBytes) from the moment the code
// object is loaded there until the process ends. Host code never passes the
// array's name to a kernel (in host code it names a host-side stand-in);
// it resolves the device address once per device with hipGetSymbolAddress,
// with that device current, and passes that address on.

#include <atomic>
#include <mutex>

#include "internal.h"

namespace higgs {

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch_ptr[kMaxDevices];
std::mutex g_scratch_mu;

}  // namespace

hipError_t scratch_buffer(void** ptr) {
  int dev = 0;
  hipError_t err = hipGetDevice(&dev);
  if (err != hipSuccess) return err;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  void* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (p == nullptr) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    p = g_scratch_ptr[dev].load(std::memory_order_relaxed);
    if (p == nullptr) {
      err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
      if (err != hipSuccess) return err;
      if (p == nullptr) return hipErrorInvalidSymbol;
      g_scratch_ptr[dev].store(p, std::memory_order_release);
    }
  }
  *ptr = p;
  return hipSuccess;
}

}  // namespace higgs
