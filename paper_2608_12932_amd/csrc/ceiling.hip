// Measured ceilings of the two units the W4A8 layer is bound by, for the
// benchmark's roofline context (the fractions themselves use the published
// peaks: 8 TB/s HBM, 5.0 POPS dense INT8):
//   - HBM read: a plain 16-byte streaming read over a large buffer, each
//     workgroup over its own contiguous range, kUnroll loads in flight per
//     lane;
//   - INT8 matrix cores: independent v_mfma_i32_32x32x32_i8 chains with
//     operands held in registers (no memory traffic at all).
// Built as its own library (libw4a8_ceiling.so); nothing in the layer uses it.
#include <hip/hip_runtime.h>

#include "device.h"
#include "w4a8_ceiling.h"

namespace w4a8 {
namespace {

constexpr int kReadThreads = 512;
constexpr int kUnroll = 16;

// Workgroup b reads its own contiguous range [b per, (b + 1) per) of the
// buffer (the fastest of the patterns measured: grid-wide strided sweeps
// reached ~5.7 TB/s, contiguous ranges ~7.0 TB/s); each instruction of the
// workgroup covers 8 KiB, kUnroll of them in flight per thread.  Offsets
// past the range read zeros.
__global__ __launch_bounds__(kReadThreads) void stream_read(const uint8_t* p, uint32_t bytes, uint32_t per,
                                                            uint32_t* sink) {
  const uint32_t begin = blockIdx.x * per;
  const uint32_t len = begin >= bytes ? 0u : min(per, bytes - begin);
  const __amdgpu_buffer_rsrc_t r = make_rsrc(p + begin, len);
  uint32_t acc = 0;
  for (uint32_t o = threadIdx.x * 16; o < per; o += kReadThreads * 16 * kUnroll) {
    uint4 v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) v[u] = buf_load16<kCacheStream>(r, o + u * kReadThreads * 16);
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  sink[blockIdx.x * kReadThreads + threadIdx.x] = acc;
}

constexpr int kMfmaThreads = 256;
constexpr int kChains = 4;

__global__ __launch_bounds__(kMfmaThreads) void mfma_chain(int iters, int32_t* sink) {
  const v4i ones = {0x01010101, 0x01010101, 0x01010101, 0x01010101};
  v16i c[kChains];
#pragma unroll
  for (int h = 0; h < kChains; ++h) c[h] = v16i{};
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int h = 0; h < kChains; ++h) c[h] = mfma32(ones, ones, c[h]);
  }
  int32_t s = 0;
#pragma unroll
  for (int h = 0; h < kChains; ++h)
#pragma unroll
    for (int e = 0; e < 16; ++e) s += c[h][e];
  sink[blockIdx.x * kMfmaThreads + threadIdx.x] = s;
}

}  // namespace
}  // namespace w4a8

extern "C" {

int w4a8_ceiling_stream_read(const void* buf, size_t bytes, uint32_t* sink, hipStream_t stream) {
  if (!buf || !sink || bytes == 0 || bytes % 16 || bytes > W4A8_CEILING_MAX_READ_BYTES) return (int)hipErrorInvalidValue;
  const size_t per = 16 * ((bytes + 16 * W4A8_CEILING_READ_BLOCKS - 1) / (16 * W4A8_CEILING_READ_BLOCKS));
  hipLaunchKernelGGL(w4a8::stream_read, dim3(W4A8_CEILING_READ_BLOCKS), dim3(w4a8::kReadThreads), 0, stream,
                     static_cast<const uint8_t*>(buf), (uint32_t)bytes, (uint32_t)per, sink);
  return (int)hipGetLastError();
}

int w4a8_ceiling_mfma_i8(int iters, int32_t* sink, hipStream_t stream) {
  if (!sink || iters < 1) return (int)hipErrorInvalidValue;
  hipLaunchKernelGGL(w4a8::mfma_chain, dim3(W4A8_CEILING_MFMA_BLOCKS), dim3(w4a8::kMfmaThreads), 0, stream, iters,
                     sink);
  return (int)hipGetLastError();
}

}  // extern "C"
