// Small-M W4A8 GEMM (decode / draft-block verification, M <= 64).
//
// At small M the layer is bound by the packed-weight stream from HBM
// (FlashDrive Sec. 4.2: decode gains from the 4x smaller weights), so the
// kernel is built around that stream:
//   - each workgroup owns NT 16-column tiles and one K split; its 8 waves
//     interleave over the 128-k blocks of the split, each lane loading one
//     16-byte chunk per tile and block straight into registers (one 1 KiB
//     contiguous load per wave), several blocks deep in flight;
//   - the chunk unpacks in registers into the B fragments of two
//     v_mfma_i32_16x16x64_i8 (no LDS round trip for weights);
//   - the partial sums of the 8 waves are reduced through LDS, and K splits
//     across workgroups (S > 1) meet in a workspace, where the last arriving
//     workgroup of a column group sums them in split order and finishes;
//   - with bf16 input and a small enough M*K, the per-token quantize is fused
//     in front: every workgroup reads the whole token rows (from L2) for the
//     absmax, then quantizes only its own K split into LDS, while its first
//     weight loads are already in flight.
// The epilogue applies the per-token and per-channel (or per-group) scales.
#include <cstdio>

#include "device.h"
#include "kernels.h"

namespace w4a8 {

namespace {

constexpr int kWaves = kSmallMWaves;
constexpr int kThreads = kWaves * 64;
constexpr int kXCache = 16;       // fused quantize: x chunks held per thread
constexpr int kOperandVgprs = 112;
constexpr int kLdsHeader = 256;   // per-row absmax / s / inv / mode
constexpr int kMaxTilesPerWave = 12;

template <int MT, int NT, bool FUSED>
constexpr int stage_depth() {
  int per = NT * 4 + (FUSED ? 0 : MT * 8);
  int d = kOperandVgprs / per;
  return d < 1 ? 1 : (d > 16 ? 16 : d);
}

struct Emit {
  const SmallMArgs& a;
  const float* lds_scale;  // fused: per-row s in LDS; else nullptr
  __device__ float sx(int row) const { return lds_scale ? lds_scale[row] : a.x_scale[row]; }
  // per-channel: v = 16 * acc
  __device__ void channel(int row, int n, int v) const {
    const size_t o = (size_t)row * a.N + n;
    const int acc = v >> 4;
    if (a.out_kind == kOutI32) {
      static_cast<int*>(a.y)[o] = acc;
      return;
    }
    const float y32 = __fmul_rn(__fmul_rn((float)acc, sx(row)), static_cast<const float*>(a.w_scale)[n]);
    if (a.out_kind == kOutF32)
      static_cast<float*>(a.y)[o] = y32;
    else
      static_cast<uint16_t*>(a.y)[o] = (uint16_t)f32_to_bf16(y32);
  }
  // group: t = sum_g p_g * s_g
  __device__ void group(int row, int n, float t) const {
    const size_t o = (size_t)row * a.N + n;
    const float y32 = __fmul_rn(t, sx(row));
    if (a.out_kind == kOutF32)
      static_cast<float*>(a.y)[o] = y32;
    else
      static_cast<uint16_t*>(a.y)[o] = (uint16_t)f32_to_bf16(y32);
  }
};

template <int MT, int NT, bool GROUP, bool FUSED>
__global__ __launch_bounds__(kThreads) void smallm(const SmallMArgs a) {
  constexpr int D = stage_depth<MT, NT, FUSED>();
  extern __shared__ __align__(16) uint8_t lds[];
  uint32_t* l_amax = reinterpret_cast<uint32_t*>(lds);
  float* l_s = reinterpret_cast<float*>(lds + 64);
  float* l_inv = reinterpret_cast<float*>(lds + 128);
  int* l_mode = reinterpret_cast<int*>(lds + 192);
  uint8_t* l_body = lds + kLdsHeader;
  __shared__ int l_last;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int gid = blockIdx.x / a.S, split = blockIdx.x % a.S;
  const int M = a.M, N = a.N, K = a.K, KB = a.KB;
  const int ntiles = N / 16;
  const int nt0 = gid * NT;
  const int kb_begin = split * a.kbs;
  const int kb_end = min(KB, kb_begin + a.kbs);
  const int nkb = kb_end - kb_begin;
  const int iters = wave < nkb ? (nkb - wave + kWaves - 1) / kWaves : 0;
  const int r16 = lane & 15, g4 = lane >> 4;
  const int ldq = nkb * 128 + 16;  // fused: LDS row stride of the codes

  // ---- fused quantize: load this thread's x chunks first (so that waiting
  // for them later does not wait for the weight stream issued after them)
  uint4 xc[FUSED ? kXCache : 1];
  int cpr = 1, nx = 0;
  if constexpr (FUSED) {
    cpr = (K / 8) / kThreads;
    nx = M * cpr;
    const uint4* xg = static_cast<const uint4*>(a.x);
#pragma unroll
    for (int j = 0; j < kXCache; ++j)
      if (j < nx) xc[j] = xg[(size_t)j * kThreads + tid];
    if (tid < 16) l_amax[tid] = 0u;
  }

  // ---- weight stream, D blocks deep
  uint4 wb[D][NT];
  uint4 ab[FUSED ? 1 : D][MT][2];
  float sgb[GROUP ? D : 1][NT];
  const uint8_t* wp = a.wp;
  auto load_stage = [&](int slot, int i) {
    const int kb = kb_begin + wave + i * kWaves;
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const int tile = nt0 + t;
      wb[slot][t] = tile < ntiles
                        ? ldg_nt(reinterpret_cast<const uint4*>(wp + ((size_t)tile * KB + kb) * kBlockBytes) + lane)
                        : make_uint4(0, 0, 0, 0);
      if constexpr (GROUP) {
        const uint16_t* sg = static_cast<const uint16_t*>(a.w_scale);
        sgb[slot][t] = tile < ntiles ? f16_to_f32(sg[(size_t)kb * N + tile * 16 + r16]) * 0.0625f : 0.0f;
      }
    }
    if constexpr (!FUSED) {
      const int8_t* xq = static_cast<const int8_t*>(a.x);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const int row = mt * 16 + r16;
        if (row < M) {
          const uint4* p = reinterpret_cast<const uint4*>(xq + (size_t)row * K + kb * 128 + g4 * 32);
          ab[slot][mt][0] = p[0];
          ab[slot][mt][1] = p[1];
        } else {
          ab[slot][mt][0] = make_uint4(0, 0, 0, 0);
          ab[slot][mt][1] = make_uint4(0, 0, 0, 0);
        }
      }
    }
  };
#pragma unroll
  for (int s = 0; s < D; ++s)
    if (s < iters) load_stage(s, s);

  // ---- fused quantize: absmax over the full rows, codes for this split
  if constexpr (FUSED) {
    lds_barrier();  // l_amax initialised
    uint32_t pm = 0;
#pragma unroll
    for (int j = 0; j < kXCache; ++j) {
      if (j < nx) {
        pm = absmax_chunk(pm, xc[j]);
        if ((j + 1) % cpr == 0) {
          const uint32_t v = wave_max_u32(fold_pair_max(pm));
          if (lane == 0) atomicMax(&l_amax[j / cpr], v);
          pm = 0;
        }
      }
    }
    lds_barrier();
    if (tid < M) {
      const QScale q = qscale_from_absmax(bf16_lo(l_amax[tid]));
      l_s[tid] = q.s;
      l_inv[tid] = q.inv;
      l_mode[tid] = q.mode;
    }
    lds_barrier();
    const int k_lo = kb_begin * 128, k_hi = kb_end * 128;
#pragma unroll
    for (int j = 0; j < kXCache; ++j) {
      if (j < nx) {
        const int row = j / cpr;
        const int k = ((j % cpr) * kThreads + tid) * 8;
        if (k >= k_lo && k < k_hi) {
          const int mode = __builtin_amdgcn_readfirstlane(l_mode[row]);
          const uint2 o = quant_chunk(xc[j], l_s[row], l_inv[row], mode);
          *reinterpret_cast<uint2*>(l_body + row * ldq + (k - k_lo)) = o;
        }
      }
    }
    lds_barrier();
  }

  // ---- main loop
  v4i acc[MT][NT];
  float facc[GROUP ? MT : 1][NT][4];
  const v4i zero4 = {0, 0, 0, 0};
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      acc[mt][t] = zero4;
      if constexpr (GROUP)
#pragma unroll
        for (int r = 0; r < 4; ++r) facc[mt][t][r] = 0.0f;
    }

  for (int base = 0; base < iters; base += D) {
#pragma unroll
    for (int s = 0; s < D; ++s) {
      const int i = base + s;
      if (i < iters) {
        v4i alo[MT], ahi[MT];
        if constexpr (FUSED) {
          if (r16 < M) {
            const int kb = kb_begin + wave + i * kWaves;
            const uint8_t* p = l_body + r16 * ldq + (kb - kb_begin) * 128 + g4 * 32;
            alo[0] = *reinterpret_cast<const v4i*>(p);
            ahi[0] = *reinterpret_cast<const v4i*>(p + 16);
          } else {
            alo[0] = zero4;
            ahi[0] = zero4;
          }
        } else {
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) {
            alo[mt] = as_v4i(ab[s][mt][0]);
            ahi[mt] = as_v4i(ab[s][mt][1]);
          }
        }
#pragma unroll
        for (int t = 0; t < NT; ++t) {
          const v4i blo = nib_lo(wb[s][t]);
          const v4i bhi = nib_hi(wb[s][t]);
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) {
            if constexpr (GROUP) {
              v4i p = mfma16(alo[mt], blo, zero4);
              p = mfma16(ahi[mt], bhi, p);
#pragma unroll
              for (int r = 0; r < 4; ++r) facc[mt][t][r] = __fmaf_rn((float)p[r], sgb[s][t], facc[mt][t][r]);
            } else {
              acc[mt][t] = mfma16(alo[mt], blo, acc[mt][t]);
              acc[mt][t] = mfma16(ahi[mt], bhi, acc[mt][t]);
            }
          }
        }
        if (i + D < iters) load_stage(s, i + D);
      }
    }
  }

  // ---- reduce the waves' partial sums through LDS
  lds_barrier();  // every wave is done reading the codes
  uint32_t* red = reinterpret_cast<uint32_t*>(l_body);
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      uint4 v;
      if constexpr (GROUP) {
        v = make_uint4(__float_as_uint(facc[mt][t][0]), __float_as_uint(facc[mt][t][1]),
                       __float_as_uint(facc[mt][t][2]), __float_as_uint(facc[mt][t][3]));
      } else {
        v = make_uint4((uint32_t)acc[mt][t][0], (uint32_t)acc[mt][t][1], (uint32_t)acc[mt][t][2],
                       (uint32_t)acc[mt][t][3]);
      }
      *reinterpret_cast<uint4*>(red + ((wave * MT + mt) * NT + t) * 256 + lane * 4) = v;
    }
  lds_barrier();

  const Emit emit{a, FUSED ? l_s : nullptr};
  constexpr int kOut = MT * 16 * NT * 16;
  const int tiles_here = min(NT, ntiles - nt0);
  for (int o = tid; o < kOut; o += kThreads) {
    const int row = o / (NT * 16), col = o % (NT * 16);
    const int mt = row >> 4, rr = row & 15, t = col >> 4, cc = col & 15;
    if (row >= M || t >= tiles_here) continue;
    const int src = ((rr >> 2) * 16 + cc) * 4 + (rr & 3);
    const int n = (nt0 + t) * 16 + cc;
    if constexpr (GROUP) {
      float v = 0.0f;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) v += __uint_as_float(red[((w * MT + mt) * NT + t) * 256 + src]);
      if (a.S == 1)
        emit.group(row, n, v);
      else
        static_cast<float*>(a.partial)[((size_t)split * M + row) * N + n] = v;
    } else {
      int v = 0;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) v += (int)red[((w * MT + mt) * NT + t) * 256 + src];
      if (a.S == 1)
        emit.channel(row, n, v);
      else
        static_cast<int*>(a.partial)[((size_t)split * M + row) * N + n] = v;
    }
  }
  if (a.S == 1) return;

  // ---- split-K: the last workgroup of this column group finishes
  __threadfence();
  __syncthreads();
  if (tid == 0) {
    const unsigned prev = atomicAdd(&a.counters[gid], 1u);
    l_last = prev == (unsigned)(a.S - 1);
  }
  __syncthreads();
  if (!l_last) return;
  __threadfence();
  for (int o = tid; o < kOut; o += kThreads) {
    const int row = o / (NT * 16), col = o % (NT * 16);
    const int t = col >> 4, cc = col & 15;
    if (row >= M || t >= tiles_here) continue;
    const int n = (nt0 + t) * 16 + cc;
    if constexpr (GROUP) {
      const float* part = static_cast<const float*>(a.partial);
      float v = 0.0f;
      for (int s = 0; s < a.S; ++s) v += __builtin_nontemporal_load(part + ((size_t)s * M + row) * N + n);
      emit.group(row, n, v);
    } else {
      const int* part = static_cast<const int*>(a.partial);
      int v = 0;
      for (int s = 0; s < a.S; ++s) v += __builtin_nontemporal_load(part + ((size_t)s * M + row) * N + n);
      emit.channel(row, n, v);
    }
  }
  if (tid == 0) atomicExch(&a.counters[gid], 0u);
}

typedef void (*SmallMKernel)(const SmallMArgs);

// MT * NT is capped at 12 (kMaxTilesPerWave): beyond it the accumulators
// and in-flight operands no longer fit in 256 registers.
template <int MT, int NT, bool GROUP, bool FUSED>
SmallMKernel instance() {
  if constexpr (MT * NT <= kMaxTilesPerWave)
    return smallm<MT, NT, GROUP, FUSED>;
  else
    return nullptr;
}

template <int MT, bool GROUP, bool FUSED>
SmallMKernel pick_nt(int NT) {
  switch (NT) {
    case 1: return instance<MT, 1, GROUP, FUSED>();
    case 2: return instance<MT, 2, GROUP, FUSED>();
    case 3: return instance<MT, 3, GROUP, FUSED>();
    case 4: return instance<MT, 4, GROUP, FUSED>();
    case 6: return instance<MT, 6, GROUP, FUSED>();
    default: return nullptr;
  }
}

SmallMKernel pick(const SmallMPlan& p) {
  if (p.fused) {
    if (p.MT != 1) return nullptr;
    return p.group ? pick_nt<1, true, true>(p.NT) : pick_nt<1, false, true>(p.NT);
  }
  switch (p.MT) {
    case 1: return p.group ? pick_nt<1, true, false>(p.NT) : pick_nt<1, false, false>(p.NT);
    case 2: return p.group ? pick_nt<2, true, false>(p.NT) : pick_nt<2, false, false>(p.NT);
    case 4: return p.group ? pick_nt<4, true, false>(p.NT) : pick_nt<4, false, false>(p.NT);
    default: return nullptr;
  }
}

}  // namespace

SmallMPlan plan_smallm(int M, int N, int K, bool group, bool bf16_in) {
  SmallMPlan p{};
  p.MT = M <= 16 ? 1 : (M <= 32 ? 2 : 4);
  p.group = group;
  const int ntiles = N / 16, KB = K / 128;
  const double ideal = (double)ntiles * KB / 256.0;  // blocks per CU if perfectly spread
  const int nts[] = {6, 4, 3, 2, 1};
  const int ss[] = {1, 2, 3, 4, 6, 8};
  double best = -1.0;
  for (int nt : nts) {
    if (ntiles % nt || p.MT * nt > kMaxTilesPerWave) continue;
    for (int s : ss) {
      if (s > KB) continue;
      const int kbs = (KB + s - 1) / s;
      const int wgs = ntiles / nt * s;
      const double per_cu = (double)((wgs + 255) / 256) * nt * kbs;
      double score = ideal / per_cu;
      if (s > 1) score /= 1.0 + (double)s * M * N * 8.0 / ((double)N * K / 2.0);
      // prefer fewer workgroups on a tie (less redundant activation traffic)
      if (score > best + 1e-9 || (score > best - 1e-9 && wgs < p.groups * p.S)) {
        best = score;
        p.NT = nt;
        p.S = s;
        p.groups = ntiles / nt;
      }
    }
  }
  const int kbs = (KB + p.S - 1) / p.S;
  p.fused = bf16_in && p.MT == 1 && (K / 8) % kThreads == 0 && M * ((K / 8) / kThreads) <= kXCache &&
            (size_t)M * (kbs * 128 + 16) <= 96 * 1024;
  const size_t red = (size_t)kWaves * p.MT * p.NT * 1024;
  const size_t codes = p.fused ? (size_t)M * (kbs * 128 + 16) : 0;
  p.lds_bytes = kLdsHeader + (red > codes ? red : codes);
  return p;
}

hipError_t launch_smallm(const SmallMPlan& p, const SmallMArgs& a, hipStream_t stream) {
  SmallMKernel k = pick(p);
  if (!k) return hipErrorInvalidValue;
  const unsigned grid = (unsigned)(p.groups * p.S);
  hipLaunchKernelGGL(k, dim3(grid), dim3(kThreads), p.lds_bytes, stream, a);
  return hipGetLastError();
}

const char* smallm_kernel_name(const SmallMPlan& p) {
  static thread_local char buf[96];
  snprintf(buf, sizeof buf, "smallm<MT=%d,NT=%d,%s,%s> S=%d groups=%d", p.MT, p.NT,
           p.group ? "group" : "channel", p.fused ? "fused-quant" : "int8-in", p.S, p.groups);
  return buf;
}

}  // namespace w4a8
