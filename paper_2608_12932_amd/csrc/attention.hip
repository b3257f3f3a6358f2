// Streaming prefill attention (FlashDrive Sec. 3.1 and Fig. 3).
//
// When the camera window advances by one frame, only the tokens of the
// frame that just arrived need fresh attention rows: they form the query
// set here, while the keys and values come from the whole window's cache
// (older frames kept from earlier steps plus the arrival, ordered view by
// view).  The cache stores keys without their rotary embedding; this
// kernel rotates each key at the position it occupies in the window now,
// so sliding the window changes only the position array.  Key j may be
// seen by query i exactly when pos_k[j] <= pos_q[i], i.e. causally in the
// view-major order of the window.
//
// A first kernel rotates the window's keys once per call, at the
// positions they occupy now (every query head of a kv head reads them),
// records each 32-key tile's smallest and largest position, and (one more
// workgroup) deals the attention's work items to workgroup ids so that the
// CUs get even shares: a query block late in the window sees many more key
// tiles than an early one.  Then one workgroup per (64 queries, head, key
// split); each of its 4 waves owns 16 queries.  Key tiles that none of its
// queries can see are skipped, and a split none of them sees ends the
// workgroup before its queries are rotated.  Per 32-key tile:
//   - the workgroup stages the rotated keys (bf16, [key][d]) and the values
//     transposed ([d][key]) in LDS;
//   - a wave forms S^T = K Q^T with v_mfma_f32_16x16x32_bf16 (its rotated
//     queries are the B operand, held in registers), so a lane holds one
//     query's scores for 8 keys;
//   - online softmax in fp32: base-2 hardware exponentials of
//     score * (scale log2 e) - running maximum as one fused multiply-add
//     (weights below 2^-126 of the largest may flush to 0), the per-score
//     position test only on tiles that straddle a query of the wave, and
//     row swaps across the lane groups of a query;
//   - the weights rounded to bf16 as the B operand of O^T += V^T P^T; the 8
//     keys a lane holds are the reduction indices of its lane group, and V^T
//     is read from LDS in the same key order.
// Rotations are fp32 IEEE operations rounded to bf16, as a bf16 model holds
// its rotated operands.
#include <climits>

#include "device.h"
#include "attention.h"
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
// LDS row pitches (bf16 elements), padded against bank conflicts: the key
// rows' 16-byte reads by 16 lanes (one per key) and the transposed value
// tile's dword writes (two keys of one d) and 8-byte reads
constexpr int kKPitch = kD + 8;
constexpr int kVtPitch = kKeys + 4;

__device__ __forceinline__ bf16x8_t as_bf16x8(uint4 u) { return __builtin_bit_cast(bf16x8_t, u); }

// Reductions over the lane pairs (l, l ^ 16) and (l, l ^ 32) with the gfx950
// row swaps (no LDS round trip): each swap hands a lane its partner's value
// in one of the two results and its own in the other.  Scores are never NaN.
__device__ __forceinline__ float max_xor16(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  const float a = __uint_as_float(r[0]), b = __uint_as_float(r[1]);
  return a > b ? a : b;
}
__device__ __forceinline__ float max_xor32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  const float a = __uint_as_float(r[0]), b = __uint_as_float(r[1]);
  return a > b ? a : b;
}

// The rotated pair chunks (8 values each at d and d + 64) of one row at
// position pos, as bf16 words: lo = a cos - b sin, hi = b cos + a sin.
__device__ __forceinline__ void rotate_chunks(uint4 a8, uint4 b8, const float* cs, const float* sn, uint4& lo,
                                              uint4& hi) {
  // three roundings per output (two products, then the sum), as in plain
  // fp32 arithmetic: no contraction into fused multiply-adds (the _rn
  // intrinsics are ordinary operators in their own scope and would be
  // contracted)
#pragma clang fp contract(off)
  const uint32_t aw[4] = {a8.x, a8.y, a8.z, a8.w}, bw[4] = {b8.x, b8.y, b8.z, b8.w};
  uint32_t lw[4], hw[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const float a0 = bf16_lo(aw[e]), a1 = bf16_hi(aw[e]);
    const float b0 = bf16_lo(bw[e]), b1 = bf16_hi(bw[e]);
    const float c0 = cs[2 * e], c1 = cs[2 * e + 1], s0 = sn[2 * e], s1 = sn[2 * e + 1];
    lw[e] = bf16x2_bits(a0 * c0 - b0 * s0, a1 * c1 - b1 * s1);
    hw[e] = bf16x2_bits(b0 * c0 + a0 * s0, b1 * c1 + a1 * s1);
  }
  lo = make_uint4(lw[0], lw[1], lw[2], lw[3]);
  hi = make_uint4(hw[0], hw[1], hw[2], hw[3]);
}

// Limits of the dispatch schedule (larger calls keep the plain order).
constexpr int kSchedMaxClasses = 256;  // (query block, split) pairs
constexpr int kSchedMaxTiles = 1024;   // 32-key tiles

// The order in which the attention's workgroups take their work items.
// Workgroup ids are dealt to the CUs in rounds of C consecutive ids (id mod
// C picks the CU while every workgroup is resident), so a CU runs one item
// of each round side by side.  The items are ranked by their number of
// visible key tiles (the same for every head of a (query block, split)
// pair) and dealt heaviest first, every second round in reverse: a CU that
// gets one of the heaviest items of a round gets one of the lightest of the
// next.  sched[id] = (query block * S + split) * H + head.
__device__ void build_schedule(const AttnArgs& a) {
  __shared__ int s_qmax[kSchedMaxClasses];
  __shared__ int s_tmin[kSchedMaxTiles];
  __shared__ int s_vis[kSchedMaxClasses];
  __shared__ int s_class_of_rank[kSchedMaxClasses];
  const int tid = threadIdx.x;
  const int X = (a.Nq + kQPerBlock - 1) / kQPerBlock, ntiles = (a.Nk + kKeys - 1) / kKeys;
  const int S = a.S, n = X * S, H = a.H;
  // each block's largest query position and each tile's smallest key
  // position: every thread sweeps the position arrays with independent
  // loads and folds them into LDS with atomics
  for (int x = tid; x < X; x += 256) s_qmax[x] = INT_MIN;
  for (int t = tid; t < ntiles; t += 256) s_tmin[t] = INT_MAX;
  __syncthreads();
  // both position arrays swept together, so that every thread's loads of
  // both go out before any of its atomics
  constexpr int kBatch = 16;  // loads in flight per array and thread
  const int span = max(a.Nq, a.Nk);
  for (int i0 = tid; i0 < span; i0 += 256 * kBatch) {
    int vq[kBatch], vk[kBatch];
#pragma unroll
    for (int b = 0; b < kBatch; ++b) {
      const int i = i0 + 256 * b;
      vq[b] = i < a.Nq ? a.pos_q[i] : INT_MIN;
      vk[b] = i < a.Nk ? a.pos_k[i] : INT_MAX;
    }
#pragma unroll
    for (int b = 0; b < kBatch; ++b) {
      const int i = i0 + 256 * b;
      if (i < a.Nq) atomicMax(&s_qmax[i / kQPerBlock], vq[b]);
      if (i < a.Nk) atomicMin(&s_tmin[i / kKeys], vk[b]);
    }
  }
  for (int c = tid; c < n; c += 256) s_vis[c] = 0;
  __syncthreads();
  // visible tiles of each (block, split) class, one (class, tile) pair per
  // thread and step (the counter a lane adds to depends on its index)
  const int tps = a.tiles_per_split;
  for (int i = tid; i < n * tps; i += 256) {
    const int c = i / tps, t = (c % S) * tps + (i - c * tps);
    if (t < ntiles && s_tmin[t] <= s_qmax[c / S]) atomicAdd(&s_vis[c], 1);
  }
  __syncthreads();
  // a block whose keys only one split sees: that split writes the output
  // itself and the merge skips the block's rows
  for (int x = tid; x < X; x += 256) {
    int only = -1, cnt = 0;
    for (int z = 0; z < S; ++z)
      if (s_vis[x * S + z] > 0) {
        ++cnt;
        only = z;
      }
    a.solo[x] = cnt == 1 ? only : -1;
  }
  // rank of each class: heavier first, ties in class order
  for (int c = tid; c < n; c += 256) {
    const int vc = s_vis[c];
    int r = 0;
#pragma unroll 8
    for (int c2 = 0; c2 < n; ++c2) {
      const int v2 = s_vis[c2];
      r += (v2 > vc || (v2 == vc && c2 < c)) ? 1 : 0;
    }
    s_class_of_rank[r] = c;
  }
  __syncthreads();
  // item k of the ranked list is class s_class_of_rank[k / H], head k % H
  const int G = n * H, C = a.sched_cus;
  for (int k = tid; k < G; k += 256) {
    const int r = k / H, h = k - r * H;
    const int round = k / C, p = k - round * C;
    const bool reversed = (round & 1) && (round + 1) * C <= G;  // a partial last round keeps its order
    a.sched[round * C + (reversed ? C - 1 - p : p)] = s_class_of_rank[r] * H + h;
  }
}

constexpr int kRotHeads = 2;  // kv heads per thread of the key rotation

// The keys rotated at their window positions: k_rot[hk][j] from k[hk][j]
// and pos_k[j], one 16-byte pair of chunks (d = 8 c .., 64 + 8 c ..) of
// kRotHeads kv heads per thread (one read of the table row), 32 keys per
// workgroup.  Rotating each key once here instead of in every workgroup
// that stages it (all query blocks of the kv head's query heads) took
// 21 us off the bench workload's 114 us.  The first row of workgroups also
// records each tile's key-position bounds, and one more workgroup, past
// the last tile, builds the dispatch schedule.
__global__ __launch_bounds__(256) void rotate_keys(const AttnArgs a) {
  const int tid = threadIdx.x, hk = blockIdx.y;
  if ((int)blockIdx.x * kKeys >= a.Nk) {  // the column past the last tile: the schedule
    if (hk == 0) build_schedule(a);
    return;
  }
  if (hk == 0 && tid < 64) {
    // the tile's smallest and largest key positions (keys past Nk count as
    // unseen), read by every workgroup of the attention for its skip and
    // mask tests
    const int jj = blockIdx.x * kKeys + (tid & (kKeys - 1));
    int mn = jj < a.Nk ? a.pos_k[jj] : INT_MAX, mx = mn;
#pragma unroll
    for (int off = kKeys / 2; off >= 1; off >>= 1) {
      mn = min(mn, __shfl_xor(mn, off, 64));
      mx = max(mx, __shfl_xor(mx, off, 64));
    }
    if (tid == 0) a.tile_bounds[blockIdx.x] = make_int2(mn, mx);
  }
  const int j = blockIdx.x * kKeys + (tid >> 3), c = tid & 7;
  if (j >= a.Nk) return;
  const int P = a.n_pos, p = a.pos_k[j];
  const int pc = p < 0 ? 0 : (p >= P ? P - 1 : p);  // table reads stay in bounds
  // kRotHeads kv heads per thread share one read of the table row
  const int h0 = hk * kRotHeads, nh = min(kRotHeads, a.Hkv - h0);
  uint4 x0[kRotHeads], x1[kRotHeads];
#pragma unroll
  for (int i = 0; i < kRotHeads; ++i)
    if (i < nh) {
      const uint16_t* src = a.k + ((size_t)(h0 + i) * a.Nk + j) * kD;
      x0[i] = *reinterpret_cast<const uint4*>(src + 8 * c);
      x1[i] = *reinterpret_cast<const uint4*>(src + kHalf + 8 * c);
    }
  float cs[8], sn[8];
  {
    const float4* cp = reinterpret_cast<const float4*>(a.rope_cos + (size_t)pc * kHalf + 8 * c);
    const float4* sp = reinterpret_cast<const float4*>(a.rope_sin + (size_t)pc * kHalf + 8 * c);
    const float4 c0 = cp[0], c1 = cp[1], s0 = sp[0], s1 = sp[1];
    cs[0] = c0.x; cs[1] = c0.y; cs[2] = c0.z; cs[3] = c0.w; cs[4] = c1.x; cs[5] = c1.y; cs[6] = c1.z; cs[7] = c1.w;
    sn[0] = s0.x; sn[1] = s0.y; sn[2] = s0.z; sn[3] = s0.w; sn[4] = s1.x; sn[5] = s1.y; sn[6] = s1.z; sn[7] = s1.w;
  }
#pragma unroll
  for (int i = 0; i < kRotHeads; ++i)
    if (i < nh) {
      uint4 lo, hi;
      rotate_chunks(x0[i], x1[i], cs, sn, lo, hi);
      uint16_t* dst = a.k_rot + ((size_t)(h0 + i) * a.Nk + j) * kD;
      *reinterpret_cast<uint4*>(dst + 8 * c) = lo;
      *reinterpret_cast<uint4*>(dst + kHalf + 8 * c) = hi;
    }
}

// Per-tile minimum key positions kept for the skip test (tiles beyond this
// count are never skipped).
constexpr int kMaxSkipTiles = 512;

// The occupancy hint (4 workgroups, i.e. 4 waves per SIMD) holds the kernel
// to 128 registers (it needs 110, without spills); LDS (39.3 KiB per
// workgroup) also fits 4.
__global__ __launch_bounds__(kAttnWaves * 64, 4) void stream_attention(const AttnArgs a) {
  // two stages of the key / value tile: the next visible tile is staged
  // while the current one is computed
  __shared__ __align__(16) uint16_t l_k[2][kKeys * kKPitch];     // rotated keys [key][d]
  __shared__ __align__(16) uint16_t l_vt[2][kD * kVtPitch];      // values transposed [d][key]
  __shared__ int l_pos[2][kKeys];
  __shared__ int l_tmin[kMaxSkipTiles];
  __shared__ int l_tmax[kMaxSkipTiles];
  __shared__ int l_qmax[kAttnWaves];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  int xb = blockIdx.x, h = blockIdx.y, split = blockIdx.z;  // this workgroup's item
  if (a.sched) {  // a 1-D grid dealt by the schedule
    const int code = a.sched[blockIdx.x], c = code / a.H;
    h = code % a.H;
    xb = c / a.S;
    split = c % a.S;
  }
  // this split alone sees keys of the block: it writes the output itself
  const bool final_out = a.S == 1 || (a.sched && a.solo[xb] == split);
  const int hk = h / (a.H / a.Hkv);
  const int r16 = lane & 15, g = lane >> 4;
  const int P = a.n_pos;
  auto clamp_pos = [&](int p) { return p < 0 ? 0 : (p >= P ? P - 1 : p); };  // table reads stay in bounds

  // ---- this lane's query: rotated, as the B operand of S^T = K Q^T
  // (lane: query r16, d chunk 32 i + 8 g for MFMA i; chunks i and i + 2 are
  // a rotate-half pair)
  const int qi = xb * kQPerBlock + wave * kQPerWave + r16;
  const bool q_ok = qi < a.Nq;
  const int pq = q_ok ? a.pos_q[qi] : INT_MIN;
  // Rows past Nq and keys past Nk are out-of-range buffer offsets, which
  // read zeros (selects of a loaded value against a zero vector had put the
  // zero in scratch memory, on the loop's critical path).
  const __amdgpu_buffer_rsrc_t qres = make_rsrc(a.q + (size_t)h * a.Nq * kD, (uint32_t)((size_t)a.Nq * kD * 2));
  uint4 qraw[2][2];  // chunks (32 i + 8 g, + 64), rotated once the block is known to see a key
  {
    const uint32_t qoff = q_ok ? (uint32_t)(qi * kD * 2) : kOOB;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int d = 32 * i + 8 * g;  // < 64
      qraw[i][0] = buf_load16(qres, qoff == kOOB ? kOOB : qoff + d * 2);
      qraw[i][1] = buf_load16(qres, qoff == kOOB ? kOOB : qoff + (d + kHalf) * 2);
    }
  }

  // ---- this workgroup's key tiles (its split of the key range) and the
  // skip test: a tile none of its queries can see (every key position above
  // the largest query position) is not staged
  const int ntiles_all = (a.Nk + kKeys - 1) / kKeys;
  const int t_begin = split * a.tiles_per_split;
  const int ntiles = min(ntiles_all, t_begin + a.tiles_per_split);  // one past the last tile
  const bool skipping = ntiles - t_begin <= kMaxSkipTiles;
  int wave_qmin;  // the wave's smallest query position (INT_MAX when it has no query)
  {
    int qm = pq, qn = q_ok ? pq : INT_MAX;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      qm = max(qm, __shfl_xor(qm, off, 64));
      qn = min(qn, __shfl_xor(qn, off, 64));
    }
    if (lane == 0) l_qmax[wave] = qm;
    wave_qmin = __builtin_amdgcn_readfirstlane(qn);
    // the split's tile bounds, one tile per thread
    if (skipping)
      for (int t = t_begin + tid; t < ntiles; t += kAttnWaves * 64) {
        const int2 bd = a.tile_bounds[t];
        l_tmin[t - t_begin] = bd.x;
        l_tmax[t - t_begin] = bd.y;
      }
  }
  __syncthreads();
  int wg_qmax = l_qmax[0];
#pragma unroll
  for (int w = 1; w < kAttnWaves; ++w) wg_qmax = max(wg_qmax, l_qmax[w]);
  auto next_visible = [&](int t) {
    if (skipping)
      while (t < ntiles && l_tmin[t - t_begin] > wg_qmax) ++t;
    return t;
  };
  int cur = next_visible(t_begin);
  if (a.S > 1 && cur >= ntiles) {
    // no query of the block sees a key of this split: an empty partial
    // (the merge reads only its maximum)
    if (q_ok && g == 0)
      *reinterpret_cast<float2*>(a.part_ml + (((size_t)split * a.H + h) * a.Nq + qi) * 2) = make_float2(-INFINITY, 0.0f);
    return;
  }

  bf16x8_t qf[4];
  {
    const int pc = clamp_pos(q_ok ? pq : 0);
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int d = 32 * i + 8 * g;
      uint4 lo, hi;
      rotate_chunks(qraw[i][0], qraw[i][1], a.rope_cos + (size_t)pc * kHalf + d, a.rope_sin + (size_t)pc * kHalf + d,
                    lo, hi);
      qf[i] = as_bf16x8(lo);
      qf[i + 2] = as_bf16x8(hi);
    }
  }

  f32x4_t acc[kD / 16];
#pragma unroll
  for (int t = 0; t < kD / 16; ++t) acc[t] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float m = -INFINITY, lsum = 0.0f;
  const float sl2 = a.scale_log2e;

  const __amdgpu_buffer_rsrc_t kres =
      make_rsrc(a.k_rot + (size_t)hk * a.Nk * kD, (uint32_t)((size_t)a.Nk * kD * 2));
  const __amdgpu_buffer_rsrc_t vres = make_rsrc(a.v + (size_t)hk * a.Nk * kD, (uint32_t)((size_t)a.Nk * kD * 2));
  // staging: for the keys, thread tid handles key tid / 8 of the tile and
  // the pair of 8-element chunks (8 c, 64 + 8 c), c = tid % 8; for the
  // values, keys 2 kp and 2 kp + 1 (kp = tid % 16) and d chunk tid / 16, so
  // that each transposed store is one dword.  The global loads of the next
  // tile are issued before the current tile's compute.
  const int sj = tid >> 3, sc = tid & 7;
  const int vkp = tid & 15, vc = tid >> 4;
  uint4 gk0, gk1, gv0, gv1;
  int gpj;
  auto load_tile = [&](int t) {
    const int j = t * kKeys + sj;
    const bool ok = j < a.Nk;
    const int jv0 = t * kKeys + 2 * vkp, jv1 = jv0 + 1;
    gpj = ok ? a.pos_k[j] : INT_MAX;
    const uint32_t ko = ok ? (uint32_t)((j * kD + 8 * sc) * 2) : kOOB;
    gk0 = buf_load16(kres, ko);
    gk1 = buf_load16(kres, ko == kOOB ? kOOB : ko + kHalf * 2);
    gv0 = buf_load16(vres, jv0 < a.Nk ? (uint32_t)((jv0 * kD + 8 * vc) * 2) : kOOB);
    gv1 = buf_load16(vres, jv1 < a.Nk ? (uint32_t)((jv1 * kD + 8 * vc) * 2) : kOOB);
  };
  auto store_tile = [&](int b) {
    *reinterpret_cast<uint4*>(&l_k[b][sj * kKPitch + 8 * sc]) = gk0;
    *reinterpret_cast<uint4*>(&l_k[b][sj * kKPitch + kHalf + 8 * sc]) = gk1;
    // row d of the transposed tile gets (v[2 kp][d], v[2 kp + 1][d]) as one dword
    const uint32_t w0[4] = {gv0.x, gv0.y, gv0.z, gv0.w}, w1[4] = {gv1.x, gv1.y, gv1.z, gv1.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      uint32_t* r0 = reinterpret_cast<uint32_t*>(&l_vt[b][(8 * vc + 2 * e) * kVtPitch + 2 * vkp]);
      uint32_t* r1 = reinterpret_cast<uint32_t*>(&l_vt[b][(8 * vc + 2 * e + 1) * kVtPitch + 2 * vkp]);
      *r0 = __builtin_amdgcn_perm(w1[e], w0[e], 0x05040100u);  // low halves: d = 8 vc + 2 e
      *r1 = __builtin_amdgcn_perm(w1[e], w0[e], 0x07060302u);  // high halves: d + 1
    }
    if (sc == 0) l_pos[b][sj] = gpj;
  };

  auto compute_tile = [&](int b, int t) {
    // ---- S^T for keys 16 u + (4 g + r), u = 0, 1: lane holds query r16
    // (raw scores; the scale is applied inside the exponent)
    float s[2][4];
    // the position test per score only where some key of the tile lies
    // beyond some query of the wave
    const bool full = skipping && l_tmax[t - t_begin] <= wave_qmin;
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      f32x4_t c = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const bf16x8_t kf = as_bf16x8(*reinterpret_cast<const uint4*>(&l_k[b][(16 * u + r16) * kKPitch + 32 * i + 8 * g]));
        c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[i], c, 0, 0, 0);
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) s[u][r] = c[r];
    }
    if (!full) {
#pragma unroll
      for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (l_pos[b][16 * u + 4 * g + r] > pq) s[u][r] = -INFINITY;
    }
    // ---- online softmax over this lane's query (its 8 keys here, then the
    // 4 lane groups holding the same query), in scaled base-2 units: the
    // scale is positive, so the largest raw score gives the largest scaled one
    float tmax = -INFINITY;
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int r = 0; r < 4; ++r) tmax = fmaxf(tmax, s[u][r]);
    tmax = max_xor32(max_xor16(tmax)) * sl2;
    const float mnew = fmaxf(m, tmax);
    // exponent offset: while nothing is visible yet the masked scores
    // (-inf) must still give 0
    const float mb = mnew == -INFINITY ? 0.0f : mnew;
    const float alpha = __builtin_amdgcn_exp2f(m - mb);  // 0 while m is -inf (the sums are 0 then)
    float p[2][4], psum = 0.0f;
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        p[u][r] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[u][r], sl2, -mb));
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
      const uint16_t* vr = &l_vt[b][(16 * t + r16) * kVtPitch];
      const uint2 va = *reinterpret_cast<const uint2*>(vr + 4 * g);
      const uint2 vb = *reinterpret_cast<const uint2*>(vr + 16 + 4 * g);
      const bf16x8_t vf = as_bf16x8(make_uint4(va.x, va.y, vb.x, vb.y));
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[t][r] *= alpha;
      acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pb, acc[t], 0, 0, 0);
    }
  };

  // One barrier per tile: stage b is computed while stage b ^ 1 is filled;
  // stage b ^ 1 was last read before the previous barrier.
  if (cur < ntiles) {
    load_tile(cur);
    store_tile(0);
  }
  __syncthreads();
  int b = 0;
  while (cur < ntiles) {
    const int nxt = next_visible(cur + 1);
    if (nxt < ntiles) load_tile(nxt);
    compute_tile(b, cur);
    if (nxt < ntiles) store_tile(b ^ 1);
    __syncthreads();
    b ^= 1;
    cur = nxt;
  }

  // ---- O = O^T / l: lane holds query r16, d = 16 t + 4 g + r
  lsum += __shfl_xor(lsum, 16, 64);
  lsum += __shfl_xor(lsum, 32, 64);
  if (!q_ok) return;
  if (!final_out) {
    // a split's partial result: the unnormalized sum, its running maximum
    // (base 2, scaled scores) and weight total; attn_combine merges them
    const size_t row = ((size_t)split * a.H + h) * a.Nq + qi;
    float* po = a.part_o + row * kD;
    if (m != -INFINITY)  // the merge reads no sum of a split that saw nothing
#pragma unroll
      for (int t = 0; t < kD / 16; ++t)
        *reinterpret_cast<float4*>(po + 16 * t + 4 * g) = make_float4(acc[t][0], acc[t][1], acc[t][2], acc[t][3]);
    if (g == 0) *reinterpret_cast<float2*>(a.part_ml + row * 2) = make_float2(m, lsum);
    return;
  }
  const float inv = lsum > 0.0f ? __fdiv_rn(1.0f, lsum) : 0.0f;  // a query that sees no key gets 0
  uint16_t* orow = a.o + ((size_t)h * a.Nq + qi) * kD;
#pragma unroll
  for (int t = 0; t < kD / 16; ++t) {
    const uint2 w = make_uint2(bf16x2_bits(acc[t][0] * inv, acc[t][1] * inv), bf16x2_bits(acc[t][2] * inv, acc[t][3] * inv));
    *reinterpret_cast<uint2*>(orow + 16 * t + 4 * g) = w;
  }
}


// Merge of the splits' partial results: thread per (head, query, 8 of d).
__global__ __launch_bounds__(256) void attn_combine(const AttnArgs a) {
  const size_t idx = (size_t)blockIdx.x * 256 + threadIdx.x;
  const size_t rows = (size_t)a.H * a.Nq;
  if (idx >= rows * (kD / 8)) return;
  const size_t row = idx / (kD / 8);
  const int c = (int)(idx % (kD / 8));
  if (a.sched && a.solo[(int)(row % (size_t)a.Nq) / kQPerBlock] >= 0) return;  // written by its only split
  float mmax = -INFINITY;
  for (int s = 0; s < a.S; ++s) mmax = fmaxf(mmax, a.part_ml[((size_t)s * rows + row) * 2]);
  float o[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f}, l = 0.0f;
  if (mmax != -INFINITY) {
    for (int s = 0; s < a.S; ++s) {
      const float2 ml = *reinterpret_cast<const float2*>(a.part_ml + ((size_t)s * rows + row) * 2);
      if (ml.x == -INFINITY) continue;  // the split saw no key of this query
      const float wgt = exp2f(ml.x - mmax);
      l += ml.y * wgt;
      const float4* po = reinterpret_cast<const float4*>(a.part_o + ((size_t)s * rows + row) * kD + 8 * c);
      const float4 u0 = po[0], u1 = po[1];
      o[0] += u0.x * wgt; o[1] += u0.y * wgt; o[2] += u0.z * wgt; o[3] += u0.w * wgt;
      o[4] += u1.x * wgt; o[5] += u1.y * wgt; o[6] += u1.z * wgt; o[7] += u1.w * wgt;
    }
  }
  const float inv = l > 0.0f ? __fdiv_rn(1.0f, l) : 0.0f;
  *reinterpret_cast<uint4*>(a.o + row * kD + 8 * c) =
      make_uint4(bf16x2_bits(o[0] * inv, o[1] * inv), bf16x2_bits(o[2] * inv, o[3] * inv),
                 bf16x2_bits(o[4] * inv, o[5] * inv), bf16x2_bits(o[6] * inv, o[7] * inv));
}

}  // namespace

// Key-range splits (at most 8, at least 8 tiles each): the heaviest
// workgroups, whose queries see the whole window, otherwise run every tile
// in series.
int stream_attention_splits(int H, int Nq, int Nk) {
  const long blocks = (long)((Nq + kQPerBlock - 1) / kQPerBlock) * H;
  const int ntiles = (Nk + kKeys - 1) / kKeys;
  // split until the grid would outgrow one round of resident workgroups
  // (4 per CU at 128 registers per lane, on 256 CUs): a second round costs
  // more than the longer serial key loop it saves
  constexpr long kResident = 4 * 256;
  int S = 1;
  while (S < 8 && blocks * S * 2 <= kResident && ntiles / (S * 2) >= 8) S *= 2;
  return S;
}

// Workspace, past the counter region shared with the linear calls'
// workspaces (left untouched here): the rotated keys (room for H kv heads,
// the most a call with H query heads has), then the split partials.
size_t rotated_keys_bytes(int H, int Nk) { return ((size_t)H * Nk * kD * 2 + 255) / 256 * 256; }
size_t tile_bounds_bytes(int Nk) { return ((size_t)(Nk + kKeys - 1) / kKeys * sizeof(int2) + 255) / 256 * 256; }
// The splits a call uses (the split rule, without empty trailing splits).
int used_splits(int H, int Nq, int Nk, int* tiles_per_split) {
  const int ntiles = (Nk + kKeys - 1) / kKeys;
  const int S = stream_attention_splits(H, Nq, Nk);
  const int tps = (ntiles + S - 1) / S;
  if (tiles_per_split) *tiles_per_split = tps;
  return (ntiles + tps - 1) / tps;
}
// Bytes of the dispatch schedule (0 for calls past its limits).
size_t schedule_bytes(int H, int Nq, int Nk) {
  const long classes = (long)((Nq + kQPerBlock - 1) / kQPerBlock) * used_splits(H, Nq, Nk, nullptr);
  if (classes > kSchedMaxClasses || (Nk + kKeys - 1) / kKeys > kSchedMaxTiles) return 0;
  const size_t blocks = (size_t)(Nq + kQPerBlock - 1) / kQPerBlock;
  return (((size_t)classes * H + blocks) * sizeof(int) + 255) / 256 * 256;  // the schedule, then the solo table
}
size_t stream_attention_workspace(int H, int Nq, int Nk) {
  const int S = stream_attention_splits(H, Nq, Nk);
  return kCounterRegionBytes + rotated_keys_bytes(H, Nk) + tile_bounds_bytes(Nk) + schedule_bytes(H, Nq, Nk) +
         (S > 1 ? (size_t)S * H * Nq * (kD + 2) * sizeof(float) : 0);
}

// Compute units of the current device (looked up once per device).
int compute_units() {
  static int cus[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cus[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cus[dev] = n;
  }
  return cus[dev];
}

hipError_t launch_stream_attention(const AttnArgs& a0, hipStream_t stream) {
  if (a0.Nq == 0) return hipSuccess;
  AttnArgs a = a0;
  const int ntiles = (a.Nk + kKeys - 1) / kKeys;
  a.S = used_splits(a.H, a.Nq, a.Nk, &a.tiles_per_split);
  uint8_t* ws = static_cast<uint8_t*>(a.workspace) + kCounterRegionBytes;
  a.k_rot = reinterpret_cast<uint16_t*>(ws);
  a.tile_bounds = reinterpret_cast<int2*>(ws + rotated_keys_bytes(a.H, a.Nk));
  const size_t sched_bytes = schedule_bytes(a.H, a.Nq, a.Nk);
  a.sched = sched_bytes ? reinterpret_cast<int*>(ws + rotated_keys_bytes(a.H, a.Nk) + tile_bounds_bytes(a.Nk)) : nullptr;
  a.sched_cus = compute_units();
  a.solo = a.sched ? a.sched + (size_t)((a.Nq + kQPerBlock - 1) / kQPerBlock) * a.S * a.H : nullptr;
  if (a.S > 1) {
    a.part_o = reinterpret_cast<float*>(ws + rotated_keys_bytes(a.H, a.Nk) + tile_bounds_bytes(a.Nk) + sched_bytes);
    a.part_ml = a.part_o + (size_t)a.S * a.H * a.Nq * kD;
  }
  rotate_keys<<<dim3((unsigned)(ntiles + (a.sched ? 1 : 0)), (unsigned)((a.Hkv + kRotHeads - 1) / kRotHeads)), dim3(256), 0,
                stream>>>(a);
  const unsigned X = (unsigned)((a.Nq + kQPerBlock - 1) / kQPerBlock);
  // scheduled calls (at most kSchedMaxClasses x 4096 items) take a 1-D grid
  const dim3 grid = a.sched ? dim3(X * (unsigned)a.H * (unsigned)a.S) : dim3(X, (unsigned)a.H, (unsigned)a.S);
  stream_attention<<<grid, dim3(kAttnWaves * 64), 0, stream>>>(a);
  if (a.S > 1) {
    const size_t threads = (size_t)a.H * a.Nq * (kD / 8);
    attn_combine<<<dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, stream>>>(a);
  }
  return hipGetLastError();
}

}  // namespace w4a8
