// Euler step of the flow-matching action solve with the velocity cache
// (FlashDrive Sec. 3.3, adaptive-step flow matching).
//
// The action head integrates dx/dt = v(x, t) over a fixed number of steps;
// the steps in the middle of the path reuse the velocity cached at the last
// evaluated step instead of calling the network.  A step is elementwise over
// the trajectory state and HBM-bound: fp32 x is read and written, the bf16
// velocity is read, and on an evaluated step the cache is rewritten and
// compared with the new velocity (the four row sums behind the
// consecutive-velocity relative difference and cosine similarity).
//
// A call may apply several consecutive steps with the same velocity: an
// evaluated step and the reused steps after it take one launch and one
// pass over the state, with the roundings of separate steps.
//
// One workgroup of 256 threads per row; with n % 8 == 0 each thread moves 8
// elements per pass as 16-byte loads and stores, otherwise one.  The row
// sums are fp64: the products of two bf16 values are exact there.  v may be
// the cache itself (each element is read before the same thread rewrites it).
#include "device.h"
#include "kernels.h"

namespace w4a8 {

namespace {

constexpr int kFlowThreads = 256;

struct Sums {
  double vc = 0, vv = 0, cc = 0, dd = 0;
  __device__ __forceinline__ void add(float v, float c) {
    const double a = v, b = c, d = a - b;
    vc += a * b;
    vv += a * a;
    cc += b * b;
    dd += d * d;
  }
};

__device__ __forceinline__ double wave_sum(double s) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) s += __shfl_xor(s, o);
  return s;
}

// x' = fl32(x + fl32(dt v)) applied `repeat` times, no contraction into a
// fused multiply-add
__device__ __forceinline__ float euler(float x, float dt, float v, int repeat) {
#pragma clang fp contract(off)
  const float p = dt * v;
  for (int r = 0; r < repeat; ++r) x = x + p;
  return x;
}

template <bool FRESH, bool STATS, bool VEC>
__global__ __launch_bounds__(kFlowThreads) void flow_step_rows(float* __restrict__ x, const uint16_t* v,
                                                               uint16_t* cache, int n, float dt, int repeat,
                                                               double* __restrict__ stats) {
  const int64_t base = int64_t(blockIdx.x) * n;
  float* xr = x + base;
  uint16_t* cr = cache + base;
  const uint16_t* vr = FRESH ? v + base : cr;
  Sums s;
  if constexpr (VEC) {
    for (int i = threadIdx.x * 8; i < n; i += kFlowThreads * 8) {
      const uint4 vw = *reinterpret_cast<const uint4*>(vr + i);
      uint4 cw = vw;
      if constexpr (STATS) cw = *reinterpret_cast<const uint4*>(cr + i);
      float4 x0 = *reinterpret_cast<const float4*>(xr + i);
      float4 x1 = *reinterpret_cast<const float4*>(xr + i + 4);
      const uint32_t vp[4] = {vw.x, vw.y, vw.z, vw.w};
      float f[8];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        f[2 * e] = bf16_lo(vp[e]);
        f[2 * e + 1] = bf16_hi(vp[e]);
      }
      if constexpr (STATS) {
        const uint32_t cp[4] = {cw.x, cw.y, cw.z, cw.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          s.add(f[2 * e], bf16_lo(cp[e]));
          s.add(f[2 * e + 1], bf16_hi(cp[e]));
        }
      }
      x0.x = euler(x0.x, dt, f[0], repeat);
      x0.y = euler(x0.y, dt, f[1], repeat);
      x0.z = euler(x0.z, dt, f[2], repeat);
      x0.w = euler(x0.w, dt, f[3], repeat);
      x1.x = euler(x1.x, dt, f[4], repeat);
      x1.y = euler(x1.y, dt, f[5], repeat);
      x1.z = euler(x1.z, dt, f[6], repeat);
      x1.w = euler(x1.w, dt, f[7], repeat);
      *reinterpret_cast<float4*>(xr + i) = x0;
      *reinterpret_cast<float4*>(xr + i + 4) = x1;
      if constexpr (FRESH) *reinterpret_cast<uint4*>(cr + i) = vw;
    }
  } else {
    for (int i = threadIdx.x; i < n; i += kFlowThreads) {
      const uint16_t vb = vr[i];
      const float f = __uint_as_float(uint32_t(vb) << 16);
      if constexpr (STATS) s.add(f, __uint_as_float(uint32_t(cr[i]) << 16));
      xr[i] = euler(xr[i], dt, f, repeat);
      if constexpr (FRESH) cr[i] = vb;
    }
  }
  if constexpr (STATS) {
    __shared__ double red[kFlowThreads / 64][4];
    const double w0 = wave_sum(s.vc), w1 = wave_sum(s.vv), w2 = wave_sum(s.cc), w3 = wave_sum(s.dd);
    const int wave = threadIdx.x / 64;
    if ((threadIdx.x & 63) == 0) {
      red[wave][0] = w0;
      red[wave][1] = w1;
      red[wave][2] = w2;
      red[wave][3] = w3;
    }
    __syncthreads();
    if (threadIdx.x < 4) {
      double t = 0;
#pragma unroll
      for (int w = 0; w < kFlowThreads / 64; ++w) t += red[w][threadIdx.x];
      stats[int64_t(blockIdx.x) * 4 + threadIdx.x] = t;
    }
  }
}

template <bool FRESH, bool STATS>
hipError_t launch_rows(float* x, const uint16_t* v, uint16_t* cache, int B, int n, float dt, int repeat,
                       double* stats, hipStream_t stream) {
  if (n % 8 == 0)
    hipLaunchKernelGGL((flow_step_rows<FRESH, STATS, true>), dim3(B), dim3(kFlowThreads), 0, stream, x, v, cache, n,
                       dt, repeat, stats);
  else
    hipLaunchKernelGGL((flow_step_rows<FRESH, STATS, false>), dim3(B), dim3(kFlowThreads), 0, stream, x, v, cache, n,
                       dt, repeat, stats);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_flow_step(float* x, const uint16_t* v, uint16_t* cache, int B, int n, float dt, int repeat,
                            double* stats, hipStream_t stream) {
  if (!v) return launch_rows<false, false>(x, v, cache, B, n, dt, repeat, stats, stream);
  if (!stats) return launch_rows<true, false>(x, v, cache, B, n, dt, repeat, stats, stream);
  return launch_rows<true, true>(x, v, cache, B, n, dt, repeat, stats, stream);
}

}  // namespace w4a8
