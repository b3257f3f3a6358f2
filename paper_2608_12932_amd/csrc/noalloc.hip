// The library-owned scratch memory of w4a8_linear_noalloc: a fixed-size
// device array that stands in for the caller's workspace, for callers that
// cannot allocate (code under HIP graph capture, serving loops, harnesses
// that forbid allocation).
//
// The array lives in the library's code object, one copy per GPU, from the
// first use on that GPU until the process ends.  Host code never passes the
// array's name to a kernel (on the host it is a stand-in, not a device
// address): the device address comes from hipGetSymbolAddress, taken once
// per device with that device current, and is what the launches receive.
// Every call on one GPU shares that GPU's copy, so calls that overlap on a
// GPU (concurrent streams) race; calls on one stream are ordered.
#include <mutex>

#include "kernels.h"

namespace w4a8 {

namespace {

static __device__ __align__(256) uint8_t scratch[kNoAllocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxDevices] = {};

// Sets words [0, n) of p to zero (the split-K arrival counters of a call:
// a kernel, not a memory set, so that a captured graph replays it as such).
__global__ __launch_bounds__(256) void clear_words(unsigned* __restrict__ p, int n) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i < n) p[i] = 0u;
}

}  // namespace

hipError_t noalloc_scratch(void** ptr) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_scratch_mutex);
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

hipError_t launch_clear_words(unsigned* p, int n, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(clear_words, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream, p, n);
  return hipGetLastError();
}

}  // namespace w4a8
