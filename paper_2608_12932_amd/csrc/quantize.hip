// Per-token symmetric int8 activation quantization (the 8-bit activation
// cast of FlashDrive Sec. 3.4):
//   s = max_k |x| / 127,  q = round_half_even(x / s),  s = 0 and q = 0 for a
//   zero row.  Bit-identical to the IEEE fp32 definition (see device.h).
// HBM-bound: reads 2K bytes and writes K + 4 bytes per token.
#include "device.h"
#include "kernels.h"

namespace w4a8 {

namespace {

// One workgroup of T threads per token row; thread t keeps the row's 16-byte
// chunks t + T j (j < C) in registers between the absmax and the quantize
// pass (chunks past C T, for rows longer than the planner sized C for, are
// read again from memory).
template <int T, int C>
__global__ __launch_bounds__(T) void quantize_rows_block(const uint16_t* __restrict__ x, int K,
                                                         int8_t* __restrict__ q, float* __restrict__ scale) {
  const int row = blockIdx.x;
  const int tid = threadIdx.x;
  const uint4* xr = reinterpret_cast<const uint4*>(x + (size_t)row * K);
  uint2* qr = reinterpret_cast<uint2*>(q + (size_t)row * K);
  const int nchunk = K / 8;

  // Chunks past the row read as zeros from the buffer resource (no branch).
  const __amdgpu_buffer_rsrc_t xres = make_rsrc(xr, (uint32_t)(K * 2));
  uint4 cache[C];
  uint32_t m = 0;
#pragma unroll
  for (int j = 0; j < C; ++j) {
    const int c = tid + j * T;
    cache[j] = buf_load16(xres, c < nchunk ? (uint32_t)(c * 16) : kOOB);
  }
#pragma unroll
  for (int j = 0; j < C; ++j) m = absmax_chunk(m, cache[j]);
  for (int c = tid + C * T; c < nchunk; c += T) m = absmax_chunk(m, xr[c]);

  __shared__ uint32_t red[T / 64];
  __shared__ QScale qs;
  m = wave_max_u32(fold_pair_max(m));
  if ((tid & 63) == 0) red[tid >> 6] = m;
  __syncthreads();
  if (tid == 0) {
    uint32_t a = red[0];
#pragma unroll
    for (int w = 1; w < T / 64; ++w) a = a > red[w] ? a : red[w];
    qs = qscale_from_absmax(bf16_lo(a));
    scale[row] = qs.s;
  }
  __syncthreads();
  const float s = __uint_as_float(__builtin_amdgcn_readfirstlane(__float_as_uint(qs.s)));
  const float inv = __uint_as_float(__builtin_amdgcn_readfirstlane(__float_as_uint(qs.inv)));
  const int mode = __builtin_amdgcn_readfirstlane(qs.mode);

#pragma unroll
  for (int j = 0; j < C; ++j) {
    const int c = tid + j * T;
    if (c < nchunk) qr[c] = quant_chunk(cache[j], s, inv, mode);
  }
  for (int c = tid + C * T; c < nchunk; c += T) qr[c] = quant_chunk(xr[c], s, inv, mode);
}

// One wave per token row, four rows per workgroup (short rows: no barrier,
// no LDS round trip).  Every wave works alone: a wave whose row is past M
// exits.
constexpr int kRowsPerBlock = 4;
constexpr int kWaveThreads = 64 * kRowsPerBlock;

template <int C>
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
  uint4 cache[C];
#pragma unroll
  for (int j = 0; j < C; ++j) {
    const int c = lane + j * 64;
    cache[j] = buf_load16(xres, c < nchunk ? (uint32_t)(c * 16) : kOOB);
  }
  uint32_t m = 0;
#pragma unroll
  for (int j = 0; j < C; ++j) m = absmax_chunk(m, cache[j]);
  for (int c = lane + C * 64; c < nchunk; c += 64) m = absmax_chunk(m, xr[c]);
  m = wave_max_u32(fold_pair_max(m));
  const QScale qs = qscale_from_absmax(bf16_lo(__builtin_amdgcn_readfirstlane(m)));
  if (lane == 0) scale[row] = qs.s;

#pragma unroll
  for (int j = 0; j < C; ++j) {
    const int c = lane + j * 64;
    if (c < nchunk) qr[c] = quant_chunk(cache[j], qs.s, qs.inv, qs.mode);
  }
  for (int c = lane + C * 64; c < nchunk; c += 64) qr[c] = quant_chunk(xr[c], qs.s, qs.inv, qs.mode);
}

typedef void (*QuantBlockFn)(const uint16_t*, int, int8_t*, float*);
typedef void (*QuantWaveFn)(const uint16_t*, int, int, int8_t*, float*);

template <int T>
QuantBlockFn block_kernel(int C) {
  switch (C) {
    case 1: return quantize_rows_block<T, 1>;
    case 2: return quantize_rows_block<T, 2>;
    case 4: return quantize_rows_block<T, 4>;
    default: return quantize_rows_block<T, 8>;
  }
}

QuantWaveFn wave_kernel(int C) {
  switch (C) {
    case 1: return quantize_rows_wave<1>;
    case 2: return quantize_rows_wave<2>;
    case 4: return quantize_rows_wave<4>;
    default: return quantize_rows_wave<8>;
  }
}

}  // namespace

hipError_t launch_quantize(const uint16_t* x, int M, int K, int8_t* q, float* scale,
                           hipStream_t stream) {
  if (M == 0) return hipSuccess;
  // Threads per row: with few rows (the whole call is one round of short
  // workgroups) one chunk per thread, for the lowest latency; with many
  // rows four, so that fewer, fuller workgroups stream the rows.  A power of
  // two from 64 (one wave, four rows per workgroup) to 512.  Measured on
  // K = 4096 and 12288, M = 1 .. 4096: a fixed 256 threads per row took 3x
  // the time of 512 at K = 12288, M = 256, and one wave per row 1.6x.
  const int nchunk = K / 8;
  const int per = M <= 64 ? 1 : 4;
  int T = 64;
  while (T < 512 && T * per < nchunk) T *= 2;
  int C = 1;
  while (C < 8 && C * T < nchunk) C *= 2;
  if (T == 64) {
    wave_kernel(C)<<<dim3((M + kRowsPerBlock - 1) / kRowsPerBlock), dim3(kWaveThreads), 0, stream>>>(x, M, K, q, scale);
  } else {
    const QuantBlockFn k = T == 128 ? block_kernel<128>(C) : T == 256 ? block_kernel<256>(C) : block_kernel<512>(C);
    k<<<dim3(M), dim3(T), 0, stream>>>(x, K, q, scale);
  }
  return hipGetLastError();
}

}  // namespace w4a8
