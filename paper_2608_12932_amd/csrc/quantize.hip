// Per-token symmetric int8 activation quantization (the 8-bit activation
// cast of FlashDrive Sec. 3.4), one workgroup per token row:
//   s = max_k |x| / 127,  q = round_half_even(x / s),  s = 0 and q = 0 for a
//   zero row.  Bit-identical to the IEEE fp32 definition (see device.h).
// HBM-bound: reads 2K bytes and writes K + 4 bytes per token.
#include "device.h"
#include "kernels.h"

namespace w4a8 {

namespace {

constexpr int kThreads = 256;
constexpr int kCache = 4;  // 16-byte chunks per thread kept in registers

__global__ __launch_bounds__(kThreads) void quantize_rows(const uint16_t* __restrict__ x, int K,
                                                          int8_t* __restrict__ q,
                                                          float* __restrict__ scale) {
  const int row = blockIdx.x;
  const int tid = threadIdx.x;
  const uint4* xr = reinterpret_cast<const uint4*>(x + (size_t)row * K);
  uint2* qr = reinterpret_cast<uint2*>(q + (size_t)row * K);
  const int nchunk = K / 8;

  // Chunks past the row read as zeros from the buffer resource (no branch).
  const __amdgpu_buffer_rsrc_t xres = make_rsrc(xr, (uint32_t)(K * 2));
  uint4 cache[kCache];
  uint32_t m = 0;
#pragma unroll
  for (int j = 0; j < kCache; ++j) {
    const int c = tid + j * kThreads;
    cache[j] = buf_load16(xres, c < nchunk ? (uint32_t)(c * 16) : kOOB);
  }
#pragma unroll
  for (int j = 0; j < kCache; ++j) m = absmax_chunk(m, cache[j]);
  for (int c = tid + kCache * kThreads; c < nchunk; c += kThreads) m = absmax_chunk(m, xr[c]);

  __shared__ uint32_t red[kThreads / 64];
  __shared__ QScale qs;
  m = wave_max_u32(fold_pair_max(m));
  if ((tid & 63) == 0) red[tid >> 6] = m;
  __syncthreads();
  if (tid == 0) {
    uint32_t a = red[0];
#pragma unroll
    for (int w = 1; w < kThreads / 64; ++w) a = a > red[w] ? a : red[w];
    qs = qscale_from_absmax(bf16_lo(a));
    scale[row] = qs.s;
  }
  __syncthreads();
  const float s = __uint_as_float(__builtin_amdgcn_readfirstlane(__float_as_uint(qs.s)));
  const float inv = __uint_as_float(__builtin_amdgcn_readfirstlane(__float_as_uint(qs.inv)));
  const int mode = __builtin_amdgcn_readfirstlane(qs.mode);

#pragma unroll
  for (int j = 0; j < kCache; ++j) {
    const int c = tid + j * kThreads;
    if (c < nchunk) qr[c] = quant_chunk(cache[j], s, inv, mode);
  }
  for (int c = tid + kCache * kThreads; c < nchunk; c += kThreads)
    qr[c] = quant_chunk(xr[c], s, inv, mode);
}

}  // namespace

hipError_t launch_quantize(const uint16_t* x, int M, int K, int8_t* q, float* scale,
                           hipStream_t stream) {
  if (M == 0) return hipSuccess;
  quantize_rows<<<dim3(M), dim3(kThreads), 0, stream>>>(x, K, q, scale);
  return hipGetLastError();
}

}  // namespace w4a8
