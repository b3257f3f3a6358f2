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

// RMSNorm in front of the quantize (the normalization prologue of a
// backbone linear; FlashDrive Sec. 3.5, Kernel Fusion, merges such
// reduction and element-wise operations with the GEMMs).  Per row:
//   ss = sum_k x_k^2 in fp64 (every square exact; a fixed reduction tree),
//   v = fl32(ss / K), r = 1 / sqrt(v + eps) (IEEE fp32 operations),
//   h_k = (x_k * r) * gamma_k in fp32,
// then the per-token quantize of the fp32 h with IEEE division.  One
// workgroup of T threads per row, chunks t + T j (j < C) of x and gamma
// held in registers between the passes.
template <int T, int C>
__global__ __launch_bounds__(T) void rmsnorm_quantize_rows(const uint16_t* __restrict__ x,
                                                           const uint16_t* __restrict__ gamma, float eps, int K,
                                                           int8_t* __restrict__ q, float* __restrict__ scale) {
  const int row = blockIdx.x;
  const int tid = threadIdx.x;
  const uint4* xr = reinterpret_cast<const uint4*>(x + (size_t)row * K);
  const uint4* gr = reinterpret_cast<const uint4*>(gamma);
  uint2* qr = reinterpret_cast<uint2*>(q + (size_t)row * K);
  const int nchunk = K / 8;
  const __amdgpu_buffer_rsrc_t xres = make_rsrc(xr, (uint32_t)(K * 2));
  const __amdgpu_buffer_rsrc_t gres = make_rsrc(gr, (uint32_t)(K * 2));
  uint4 xc[C], gc[C];
#pragma unroll
  for (int j = 0; j < C; ++j) {
    const int c = tid + j * T;
    const uint32_t off = c < nchunk ? (uint32_t)(c * 16) : kOOB;
    xc[j] = buf_load16(xres, off);
    gc[j] = buf_load16(gres, off);
  }
  auto words = [](const uint4& v, int e) { return e == 0 ? v.x : e == 1 ? v.y : e == 2 ? v.z : v.w; };
  auto sq_sum = [&](const uint4& v, double acc) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const double lo = (double)bf16_lo(words(v, e)), hi = (double)bf16_hi(words(v, e));
      acc += lo * lo;  // exact product (8-bit significands)
      acc += hi * hi;
    }
    return acc;
  };
  double ss = 0.0;
#pragma unroll
  for (int j = 0; j < C; ++j) ss = sq_sum(xc[j], ss);
  for (int c = tid + C * T; c < nchunk; c += T) ss = sq_sum(xr[c], ss);

  __shared__ double red_d[T / 64];
  __shared__ float red_f[T / 64];
  __shared__ float l_r, l_s;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) ss += __shfl_xor(ss, off, 64);
  if ((tid & 63) == 0) red_d[tid >> 6] = ss;
  __syncthreads();
  if (tid == 0) {
    double t = red_d[0];
#pragma unroll
    for (int w = 1; w < T / 64; ++w) t += red_d[w];
    const float v = (float)(t / (double)K);
    // The correctly rounded fp32 root, through fp64: the hardware fp32 root
    // (what the fp32 intrinsic compiles to) is only faithful.  Rounding an
    // fp64 root within one fp64 ulp to fp32 is exact: the square root of an
    // fp32 value lies at least 2^-51 (relative) from any fp32 midpoint.
    const float root = (float)__dsqrt_rn((double)__fadd_rn(v, eps));
    l_r = __fdiv_rn(1.0f, root);
  }
  __syncthreads();
  const float r = __uint_as_float(__builtin_amdgcn_readfirstlane(__float_as_uint(l_r)));

  // h for one chunk of x and gamma (8 values), and the running max of |h|
  auto h_of = [&](const uint4& xv, const uint4& gv, float (&h)[8]) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      h[2 * e] = __fmul_rn(__fmul_rn(bf16_lo(words(xv, e)), r), bf16_lo(words(gv, e)));
      h[2 * e + 1] = __fmul_rn(__fmul_rn(bf16_hi(words(xv, e)), r), bf16_hi(words(gv, e)));
    }
  };
  float m = 0.0f;
  auto max_of = [&](const uint4& xv, const uint4& gv) {
    float h[8];
    h_of(xv, gv, h);
#pragma unroll
    for (int e = 0; e < 8; ++e) m = fmaxf(m, fabsf(h[e]));
  };
#pragma unroll
  for (int j = 0; j < C; ++j) max_of(xc[j], gc[j]);
  for (int c = tid + C * T; c < nchunk; c += T) max_of(xr[c], gr[c]);
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) m = fmaxf(m, __shfl_xor(m, off, 64));
  if ((tid & 63) == 0) red_f[tid >> 6] = m;
  __syncthreads();
  if (tid == 0) {
    float a = red_f[0];
#pragma unroll
    for (int w = 1; w < T / 64; ++w) a = fmaxf(a, red_f[w]);
    l_s = __fdiv_rn(a, 127.0f);
    scale[row] = l_s;
  }
  __syncthreads();
  const float sc = __uint_as_float(__builtin_amdgcn_readfirstlane(__float_as_uint(l_s)));

  // codes: round_half_even(h / s) by IEEE division; |h / s| <= 127 (1 +
  // 2^-24), so adding 1.5 * 2^23 rounds it and leaves the code in the low byte
  auto codes = [&](const uint4& xv, const uint4& gv) {
    float h[8];
    h_of(xv, gv, h);
    uint32_t b[8];
#pragma unroll
    for (int e = 0; e < 8; ++e)
      b[e] = sc == 0.0f ? 0u : (__float_as_uint(__fadd_rn(__fdiv_rn(h[e], sc), 12582912.0f)) & 0xFFu);
    return make_uint2(b[0] | (b[1] << 8) | (b[2] << 16) | (b[3] << 24), b[4] | (b[5] << 8) | (b[6] << 16) | (b[7] << 24));
  };
#pragma unroll
  for (int j = 0; j < C; ++j) {
    const int c = tid + j * T;
    if (c < nchunk) qr[c] = codes(xc[j], gc[j]);
  }
  for (int c = tid + C * T; c < nchunk; c += T) qr[c] = codes(xr[c], gr[c]);
}

typedef void (*NormQuantFn)(const uint16_t*, const uint16_t*, float, int, int8_t*, float*);

template <int T>
NormQuantFn norm_kernel(int C) {
  switch (C) {
    case 1: return rmsnorm_quantize_rows<T, 1>;
    case 2: return rmsnorm_quantize_rows<T, 2>;
    case 4: return rmsnorm_quantize_rows<T, 4>;
    default: return rmsnorm_quantize_rows<T, 8>;
  }
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

hipError_t launch_rmsnorm_quantize(const uint16_t* x, const uint16_t* gamma, float eps, int M, int K, int8_t* q,
                                   float* scale, hipStream_t stream) {
  if (M == 0) return hipSuccess;
  // the quantize launcher's shapes, one workgroup of at least 128 threads per row
  const int nchunk = K / 8;
  const int per = M <= 64 ? 1 : 4;
  int T = 128;
  while (T < 512 && T * per < nchunk) T *= 2;
  int C = 1;
  while (C < 8 && C * T < nchunk) C *= 2;
  const NormQuantFn k = T == 128 ? norm_kernel<128>(C) : T == 256 ? norm_kernel<256>(C) : norm_kernel<512>(C);
  k<<<dim3(M), dim3(T), 0, stream>>>(x, gamma, eps, K, q, scale);
  return hipGetLastError();
}

}  // namespace w4a8
