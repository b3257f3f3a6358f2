// Weight packing: int8 [N][K] values in [-8, 7] -> the block layout
// described in device.h (two 4-bit two's-complement values per byte).
// One thread per 16-byte output chunk; one-time cost, off the hot path.
#include <mutex>

#include "device.h"
#include "kernels.h"

namespace w4a8 {

// Range-error word, one per device (each device holds its own copy); host
// code reaches it only through the address hipGetSymbolAddress returns.
__device__ __align__(256) unsigned w4a8_pack_err_word;

namespace {

__global__ void clear_word(unsigned* p) { *p = 0u; }

__global__ __launch_bounds__(256) void pack_blocks(const int8_t* __restrict__ w, int K, int KB,
                                                   size_t total, uint8_t* __restrict__ out,
                                                   unsigned* __restrict__ err) {
  const size_t chunk = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (chunk >= total) return;
  const int j = (int)(chunk % 64);
  const size_t blk = chunk / 64;
  const int b = (int)(blk % KB);
  const size_t t = blk / KB;
  const int g = j / 16, c = j % 16;
  const size_t n = t * 16 + c;
  const int8_t* src = w + n * (size_t)K + (size_t)b * 128 + g * 32;
  int8_t lo[16], hi[16];
  *reinterpret_cast<uint4*>(lo) = *reinterpret_cast<const uint4*>(src);
  *reinterpret_cast<uint4*>(hi) = *reinterpret_cast<const uint4*>(src + 16);
  uint8_t o[16];
  bool bad = false;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    bad |= lo[i] < -8 || lo[i] > 7 || hi[i] < -8 || hi[i] > 7;
    o[i] = (uint8_t)((lo[i] & 0xF) | ((hi[i] & 0xF) << 4));
  }
  *reinterpret_cast<uint4*>(out + chunk * 16) = *reinterpret_cast<const uint4*>(o);
  if (bad) atomicOr(err, 1u);
}

std::mutex g_err_mutex;
unsigned* g_err_ptr[64] = {};

}  // namespace

hipError_t pack_error_word(unsigned** err) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_err_mutex);
  if (!g_err_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(w4a8_pack_err_word));
    if (e != hipSuccess) return e;
    g_err_ptr[dev] = static_cast<unsigned*>(p);
  }
  *err = g_err_ptr[dev];
  return hipSuccess;
}

hipError_t launch_pack(const int8_t* w, int N, int K, uint8_t* out, unsigned* err,
                       hipStream_t stream) {
  const int KB = K / 128;
  const size_t total = (size_t)(N / 16) * KB * 64;
  clear_word<<<1, 1, 0, stream>>>(err);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (total == 0) return hipSuccess;
  const unsigned blocks = (unsigned)((total + 255) / 256);
  pack_blocks<<<blocks, 256, 0, stream>>>(w, K, KB, total, out, err);
  return hipGetLastError();
}

}  // namespace w4a8
