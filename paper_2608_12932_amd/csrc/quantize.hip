// Per-token symmetric int8 activation quantization (the 8-bit activation
// cast of FlashDrive Sec. 3.4):
//   s = max_k |x| / 127,  q = round_half_even(x / s),  s = 0 and q = 0 for a
//   zero row.  Bit-identical to the IEEE fp32 definition (see device.h).
// HBM-bound: reads 2K bytes and writes K + 4 bytes per token.
#include "device.h"
#include "kernels.h"

namespace w4a8 {

namespace {

// One workgroup per token row (short rows spread over 256 threads: the
// lowest latency when there are few rows).
constexpr int kBlockThreads = 256;
constexpr int kBlockCache = 4;  // 16-byte chunks per thread kept in registers

__global__ __launch_bounds__(kBlockThreads) void quantize_rows_block(const uint16_t* __restrict__ x, int K,
                                                          int8_t* __restrict__ q,
                                                          float* __restrict__ scale) {
  const int row = blockIdx.x;
  const int tid = threadIdx.x;
  const uint4* xr = reinterpret_cast<const uint4*>(x + (size_t)row * K);
  uint2* qr = reinterpret_cast<uint2*>(q + (size_t)row * K);
  const int nchunk = K / 8;

  // Chunks past the row read as zeros from the buffer resource (no branch).
  const __amdgpu_buffer_rsrc_t xres = make_rsrc(xr, (uint32_t)(K * 2));
  uint4 cache[kBlockCache];
  uint32_t m = 0;
#pragma unroll
  for (int j = 0; j < kBlockCache; ++j) {
    const int c = tid + j * kBlockThreads;
    cache[j] = buf_load16(xres, c < nchunk ? (uint32_t)(c * 16) : kOOB);
  }
#pragma unroll
  for (int j = 0; j < kBlockCache; ++j) m = absmax_chunk(m, cache[j]);
  for (int c = tid + kBlockCache * kBlockThreads; c < nchunk; c += kBlockThreads) m = absmax_chunk(m, xr[c]);

  __shared__ uint32_t red[kBlockThreads / 64];
  __shared__ QScale qs;
  m = wave_max_u32(fold_pair_max(m));
  if ((tid & 63) == 0) red[tid >> 6] = m;
  __syncthreads();
  if (tid == 0) {
    uint32_t a = red[0];
#pragma unroll
    for (int w = 1; w < kBlockThreads / 64; ++w) a = a > red[w] ? a : red[w];
    qs = qscale_from_absmax(bf16_lo(a));
    scale[row] = qs.s;
  }
  __syncthreads();
  const float s = __uint_as_float(__builtin_amdgcn_readfirstlane(__float_as_uint(qs.s)));
  const float inv = __uint_as_float(__builtin_amdgcn_readfirstlane(__float_as_uint(qs.inv)));
  const int mode = __builtin_amdgcn_readfirstlane(qs.mode);

#pragma unroll
  for (int j = 0; j < kBlockCache; ++j) {
    const int c = tid + j * kBlockThreads;
    if (c < nchunk) qr[c] = quant_chunk(cache[j], s, inv, mode);
  }
  for (int c = tid + kBlockCache * kBlockThreads; c < nchunk; c += kBlockThreads)
    qr[c] = quant_chunk(xr[c], s, inv, mode);
}

// One wave per token row (many rows: no barrier, no LDS round trip).
constexpr int kRowsPerBlock = 4;
constexpr int kWaveThreads = 64 * kRowsPerBlock;
constexpr int kWaveCache = 8;  // 16-byte chunks per lane held in registers (K <= 4096: the whole row)

// Every wave works alone (no barrier): a wave whose row is past M exits.
__global__ __launch_bounds__(kWaveThreads) void quantize_rows_wave(const uint16_t* __restrict__ x, int M, int K,
                                                          int8_t* __restrict__ q,
                                                          float* __restrict__ scale) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * kRowsPerBlock + (int)__builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (row >= M) return;
  const uint4* xr = reinterpret_cast<const uint4*>(x + (size_t)row * K);
  uint2* qr = reinterpret_cast<uint2*>(q + (size_t)row * K);
  const int nchunk = K / 8;

  // Chunks past the row read as zeros from the buffer resource (no branch);
  // lane l holds chunks l + 64 j, so each load is 1 KiB contiguous.
  const __amdgpu_buffer_rsrc_t xres = make_rsrc(xr, (uint32_t)(K * 2));
  uint4 cache[kWaveCache];
#pragma unroll
  for (int j = 0; j < kWaveCache; ++j) {
    const int c = lane + j * 64;
    cache[j] = buf_load16(xres, c < nchunk ? (uint32_t)(c * 16) : kOOB);
  }
  uint32_t m = 0;
#pragma unroll
  for (int j = 0; j < kWaveCache; ++j) m = absmax_chunk(m, cache[j]);
  for (int c = lane + kWaveCache * 64; c < nchunk; c += 64) m = absmax_chunk(m, xr[c]);
  m = wave_max_u32(fold_pair_max(m));
  const QScale qs = qscale_from_absmax(bf16_lo(__builtin_amdgcn_readfirstlane(m)));
  if (lane == 0) scale[row] = qs.s;

#pragma unroll
  for (int j = 0; j < kWaveCache; ++j) {
    const int c = lane + j * 64;
    if (c < nchunk) qr[c] = quant_chunk(cache[j], qs.s, qs.inv, qs.mode);
  }
  for (int c = lane + kWaveCache * 64; c < nchunk; c += 64) qr[c] = quant_chunk(xr[c], qs.s, qs.inv, qs.mode);
}

}  // namespace

hipError_t launch_quantize(const uint16_t* x, int M, int K, int8_t* q, float* scale,
                           hipStream_t stream) {
  if (M == 0) return hipSuccess;
  if (M <= 64)
    quantize_rows_block<<<dim3(M), dim3(kBlockThreads), 0, stream>>>(x, K, q, scale);
  else
    quantize_rows_wave<<<dim3((M + kRowsPerBlock - 1) / kRowsPerBlock), dim3(kWaveThreads), 0, stream>>>(x, M, K, q, scale);
  return hipGetLastError();
}

}  // namespace w4a8
