// Streaming prefill attention (FlashDrive Sec. 3.1, streaming design).
//
// Streaming inference encodes only the newest frame: its tokens are the
// queries, the window's KV cache (the cached frames plus the new one, laid
// out view-major) holds the keys and values.  Keys are cached before their
// rotary embedding and rotated here at their current window positions, so
// a slide of the window only changes the positions; the streaming mask
// admits key j to query i iff pos_k[j] <= pos_q[i], the causal order of the
// view-major window.
//
// One workgroup per (64 queries, head); each of its 4 waves owns 16
// queries.  Per 32-key tile:
//   - the workgroup stages the rotated keys (bf16, [key][d]) and the values
//     transposed ([d][key]) in LDS;
//   - a wave forms S^T = K Q^T with v_mfma_f32_16x16x32_bf16 (its rotated
//     queries are the B operand, held in registers), so a lane holds one
//     query's scores for 8 keys;
//   - online softmax in fp32 (base-2 exponentials, the scale folded into
//     log2 e), the weights rounded to bf16 as the B operand of O^T += V^T P^T;
//     the 8 keys a lane holds are the reduction indices of its lane group,
//     and V^T is read from LDS in the same key order.
// Rotations are fp32 IEEE operations rounded to bf16, as a bf16 model holds
// its rotated operands.
#include <climits>

#include "device.h"
#include "kernels.h"

namespace w4a8 {

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr int kD = 128;          // head dimension
constexpr int kHalf = kD / 2;    // rotate-half pairing (d, d + 64)
constexpr int kQPerWave = 16;
constexpr int kAttnWaves = 4;
constexpr int kQPerBlock = kQPerWave * kAttnWaves;
constexpr int kKeys = 32;        // keys per tile
constexpr int kVtPitch = kKeys + 8;  // bf16 elements per row of the transposed value tile

__device__ __forceinline__ bf16x8_t as_bf16x8(uint4 u) { return __builtin_bit_cast(bf16x8_t, u); }

// The rotated pair chunks (8 values each at d and d + 64) of one row at
// position pos, as bf16 words: lo = a cos - b sin, hi = b cos + a sin.
__device__ __forceinline__ void rotate_chunks(uint4 a8, uint4 b8, const float* cs, const float* sn, uint4& lo,
                                              uint4& hi) {
  const uint32_t aw[4] = {a8.x, a8.y, a8.z, a8.w}, bw[4] = {b8.x, b8.y, b8.z, b8.w};
  uint32_t lw[4], hw[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const float a0 = bf16_lo(aw[e]), a1 = bf16_hi(aw[e]);
    const float b0 = bf16_lo(bw[e]), b1 = bf16_hi(bw[e]);
    const float c0 = cs[2 * e], c1 = cs[2 * e + 1], s0 = sn[2 * e], s1 = sn[2 * e + 1];
    lw[e] = bf16x2_bits(__fsub_rn(__fmul_rn(a0, c0), __fmul_rn(b0, s0)), __fsub_rn(__fmul_rn(a1, c1), __fmul_rn(b1, s1)));
    hw[e] = bf16x2_bits(__fadd_rn(__fmul_rn(b0, c0), __fmul_rn(a0, s0)), __fadd_rn(__fmul_rn(b1, c1), __fmul_rn(a1, s1)));
  }
  lo = make_uint4(lw[0], lw[1], lw[2], lw[3]);
  hi = make_uint4(hw[0], hw[1], hw[2], hw[3]);
}

__global__ __launch_bounds__(kAttnWaves * 64) void stream_attention(const AttnArgs a) {
  __shared__ __align__(16) uint16_t l_k[kKeys * kD];          // rotated keys [key][d]
  __shared__ __align__(16) uint16_t l_vt[kD * kVtPitch];      // values transposed [d][key]
  __shared__ int l_pos[kKeys];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = blockIdx.y, hk = h / (a.H / a.Hkv);
  const int r16 = lane & 15, g = lane >> 4;
  const int P = a.n_pos;
  auto clamp_pos = [&](int p) { return p < 0 ? 0 : (p >= P ? P - 1 : p); };  // table reads stay in bounds

  // ---- this lane's query: rotated, as the B operand of S^T = K Q^T
  // (lane: query r16, d chunk 32 i + 8 g for MFMA i; chunks i and i + 2 are
  // a rotate-half pair)
  const int qi = blockIdx.x * kQPerBlock + wave * kQPerWave + r16;
  const bool q_ok = qi < a.Nq;
  const int pq = q_ok ? a.pos_q[qi] : INT_MIN;
  bf16x8_t qf[4];
  {
    const uint4* qrow = reinterpret_cast<const uint4*>(a.q + ((size_t)h * a.Nq + (q_ok ? qi : 0)) * kD);
    const int pc = clamp_pos(q_ok ? pq : 0);
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int d = 32 * i + 8 * g;  // < 64
      uint4 x0 = q_ok ? qrow[d / 8] : make_uint4(0, 0, 0, 0);
      uint4 x1 = q_ok ? qrow[(d + kHalf) / 8] : make_uint4(0, 0, 0, 0);
      uint4 lo, hi;
      rotate_chunks(x0, x1, a.rope_cos + (size_t)pc * kHalf + d, a.rope_sin + (size_t)pc * kHalf + d, lo, hi);
      qf[i] = as_bf16x8(lo);
      qf[i + 2] = as_bf16x8(hi);
    }
  }

  f32x4_t acc[kD / 16];
#pragma unroll
  for (int t = 0; t < kD / 16; ++t) acc[t] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float m = -INFINITY, lsum = 0.0f;
  const float sl2 = a.scale_log2e;

  const uint16_t* kbase = a.k + (size_t)hk * a.Nk * kD;
  const uint16_t* vbase = a.v + (size_t)hk * a.Nk * kD;
  // staging: thread tid handles key tid / 8 of the tile and the pair of
  // 8-element chunks (8 c, 64 + 8 c), c = tid % 8
  const int sj = tid >> 3, sc = tid & 7;
  for (int k0 = 0; k0 < a.Nk; k0 += kKeys) {
    {
      const int j = k0 + sj;
      const bool ok = j < a.Nk;
      const uint4* krow = reinterpret_cast<const uint4*>(kbase + (size_t)(ok ? j : 0) * kD);
      const uint4* vrow = reinterpret_cast<const uint4*>(vbase + (size_t)(ok ? j : 0) * kD);
      const int pj = ok ? a.pos_k[j] : INT_MAX;
      const int pc = clamp_pos(ok ? pj : 0);
      const uint4 z = make_uint4(0, 0, 0, 0);
      uint4 lo, hi;
      rotate_chunks(ok ? krow[sc] : z, ok ? krow[sc + 8] : z, a.rope_cos + (size_t)pc * kHalf + 8 * sc,
                    a.rope_sin + (size_t)pc * kHalf + 8 * sc, lo, hi);
      *reinterpret_cast<uint4*>(&l_k[sj * kD + 8 * sc]) = lo;
      *reinterpret_cast<uint4*>(&l_k[sj * kD + kHalf + 8 * sc]) = hi;
      const uint4 v0 = ok ? vrow[sc] : z, v1 = ok ? vrow[sc + 8] : z;
      const uint32_t w0[4] = {v0.x, v0.y, v0.z, v0.w}, w1[4] = {v1.x, v1.y, v1.z, v1.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        l_vt[(8 * sc + 2 * e) * kVtPitch + sj] = (uint16_t)(w0[e] & 0xFFFFu);
        l_vt[(8 * sc + 2 * e + 1) * kVtPitch + sj] = (uint16_t)(w0[e] >> 16);
        l_vt[(kHalf + 8 * sc + 2 * e) * kVtPitch + sj] = (uint16_t)(w1[e] & 0xFFFFu);
        l_vt[(kHalf + 8 * sc + 2 * e + 1) * kVtPitch + sj] = (uint16_t)(w1[e] >> 16);
      }
      if (sc == 0) l_pos[sj] = pj;
    }
    __syncthreads();

    // ---- S^T for keys 16 u + (4 g + r), u = 0, 1: lane holds query r16
    float s[2][4];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      f32x4_t c = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const bf16x8_t kf = as_bf16x8(*reinterpret_cast<const uint4*>(&l_k[(16 * u + r16) * kD + 32 * i + 8 * g]));
        c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[i], c, 0, 0, 0);
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const bool vis = l_pos[16 * u + 4 * g + r] <= pq;
        s[u][r] = vis ? c[r] * sl2 : -INFINITY;
      }
    }
    // ---- online softmax over this lane's query (its 8 keys here, then the
    // 4 lane groups holding the same query)
    float tmax = -INFINITY;
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int r = 0; r < 4; ++r) tmax = fmaxf(tmax, s[u][r]);
    tmax = fmaxf(tmax, __shfl_xor(tmax, 16, 64));
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
    const float mnew = fmaxf(m, tmax);
    const float alpha = mnew == m ? 1.0f : exp2f(m - mnew);  // also 1 while nothing is visible yet
    float p[2][4], psum = 0.0f;
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        p[u][r] = s[u][r] == -INFINITY ? 0.0f : exp2f(s[u][r] - mnew);
        psum += p[u][r];
      }
    lsum = lsum * alpha + psum;
    m = mnew;
    // weights as the B operand: element e of lane group g is key 4 g + e
    // (e < 4) or 16 + 4 g + (e - 4)
    const uint4 pw = make_uint4(bf16x2_bits(p[0][0], p[0][1]), bf16x2_bits(p[0][2], p[0][3]),
                                bf16x2_bits(p[1][0], p[1][1]), bf16x2_bits(p[1][2], p[1][3]));
    const bf16x8_t pb = as_bf16x8(pw);
    // ---- O^T += V^T P^T: A row d = 16 t + r16, the same 8 keys
#pragma unroll
    for (int t = 0; t < kD / 16; ++t) {
      const uint16_t* vr = &l_vt[(16 * t + r16) * kVtPitch];
      const uint2 va = *reinterpret_cast<const uint2*>(vr + 4 * g);
      const uint2 vb = *reinterpret_cast<const uint2*>(vr + 16 + 4 * g);
      const bf16x8_t vf = as_bf16x8(make_uint4(va.x, va.y, vb.x, vb.y));
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[t][r] *= alpha;
      acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pb, acc[t], 0, 0, 0);
    }
    __syncthreads();  // the next tile overwrites the staged keys and values
  }

  // ---- O = O^T / l: lane holds query r16, d = 16 t + 4 g + r
  lsum += __shfl_xor(lsum, 16, 64);
  lsum += __shfl_xor(lsum, 32, 64);
  if (!q_ok) return;
  const float inv = lsum > 0.0f ? __fdiv_rn(1.0f, lsum) : 0.0f;  // a query that sees no key gets 0
  uint16_t* orow = a.o + ((size_t)h * a.Nq + qi) * kD;
#pragma unroll
  for (int t = 0; t < kD / 16; ++t) {
    const uint2 w = make_uint2(bf16x2_bits(acc[t][0] * inv, acc[t][1] * inv), bf16x2_bits(acc[t][2] * inv, acc[t][3] * inv));
    *reinterpret_cast<uint2*>(orow + 16 * t + 4 * g) = w;
  }
}

}  // namespace

hipError_t launch_stream_attention(const AttnArgs& a, hipStream_t stream) {
  if (a.Nq == 0) return hipSuccess;
  const dim3 grid((unsigned)((a.Nq + kQPerBlock - 1) / kQPerBlock), (unsigned)a.H);
  stream_attention<<<grid, dim3(kAttnWaves * 64), 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace w4a8
