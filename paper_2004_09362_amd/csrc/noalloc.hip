// noalloc.hip -- the device scratch of ar_execute_noalloc.
//
// The step-by-step schedule with shifted starting sets (r > 0) keeps its
// primed sums in two scratch buffers X and Y (Secs. 8-9; the buffer
// assignment is plan.cpp's).  ar_execute allocates them per plan;
// ar_execute_noalloc takes them from the file-scope array below instead, so
// that it never allocates.  Every GPU that runs it holds its own copy of the
// array (kNoAllocScratchBytes) from the first call until the process ends,
// and every call on that GPU shares it.
//
// In host code the name `scratch` is a host-side stand-in, not the device
// array: its address must never reach a kernel or a copy.  The device
// address comes from hipGetSymbolAddress, looked up once per device with
// that device current, and only that address is handed out.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cstdint>
#include <mutex>

#include "ar_internal.hpp"

static __device__ __align__(256) unsigned char scratch[ar::kNoAllocScratchBytes];

namespace ar {

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_lookup;
std::atomic<void*> g_scratch[kMaxDevices];
}  // namespace

int noalloc_scratch(int device, void** ptr) {
  *ptr = nullptr;
  if (device < 0 || device >= kMaxDevices) return int(hipErrorInvalidDevice);
  void* p = g_scratch[device].load(std::memory_order_acquire);
  if (p == nullptr) {
    std::lock_guard<std::mutex> lock(g_lookup);
    p = g_scratch[device].load(std::memory_order_relaxed);
    if (p == nullptr) {
      const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
      if (e != hipSuccess || p == nullptr) {
        (void)hipGetLastError();
        return int(e != hipSuccess ? e : hipErrorInvalidSymbol);
      }
      g_scratch[device].store(p, std::memory_order_release);
    }
  }
  *ptr = p;
  return int(hipSuccess);
}

}  // namespace ar
