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
//   - with bf16 input and a narrow column group over a long K, the
//     per-token quantize is fused in front: every workgroup reads the whole
//     token rows for the absmax (shuffles and one LDS atomic per row) and
//     quantizes its own split into LDS, issuing the weight stages in between,
//     and the waves then read the codes from LDS.  Otherwise a separate
//     quantize kernel has written the codes, which the waves load per stage.
// The epilogue applies the per-token and per-channel (or per-group) scales.
// SWIGLU instances serve the fused gate+up projection with its gated
// activation merged in (FlashDrive Sec. 3.5, Kernel Fusion): a workgroup's
// NT tiles are NT / 2 gate tiles and the NT / 2 up tiles of the same
// columns, and it writes silu(gate) * up, half the columns of the GEMM.
#include <cmath>
#include <cstdio>

#include "device.h"
#include "kernels.h"

namespace w4a8 {

namespace {

constexpr int kWaves = kSmallMWaves;
constexpr int kThreads = kWaves * 64;
constexpr int kXCache = 16;       // fused quantize: x chunks held per thread
// Registers for in-flight weight (+ activation) stages.  Narrow column
// groups (NT <= 2) get more, so a long K split (K = 12288: 12 blocks per
// wave) fits in one block of stages; wider groups already hold a whole
// K = 4096 split, and a deeper ring only costs them registers.  Group mode
// also holds the fp32 sums and the stage scales.
constexpr int kOperandVgprsNarrow = 152;
constexpr int kOperandVgprs = 128;
constexpr int kOperandVgprsFused = 112;  // the fused path also holds the x chunks
constexpr int kLdsHeader = 256;   // per-row absmax / s / inv / mode
constexpr int kMaxTilesPerWave = 12;
constexpr int kMaxFusedTiles = 2;  // fused quantize pays off up to this many tiles
constexpr int kFusedMinKB = 256;   // ... and from this many 128-k blocks (K >= 32768) on
// LDS words per wave tile of partial sums in the reduction: 256 plus a
// 16-word skew, so that consecutive tiles start 16 banks apart
constexpr int kRedTile = 272;

// How the activations reach the MFMA A operand.
enum QMode {
  kQNone = 0,  // int8 codes from memory (x_scale given)
  kQLds = 1,   // bf16 in; codes made in LDS
};

// Weight stages in flight per wave (used by the kernels and the planner).
// Gated kernels hold a second set of epilogue scales and sums: they keep
// the base budget, less 16 registers in group mode.
constexpr int stage_depth(int MT, int NT, int QM, bool GROUP, bool SW) {
  int per = NT * 4 + (QM == kQLds ? 0 : MT * 8);
  int budget = QM == kQLds ? kOperandVgprsFused : !GROUP && !SW && NT <= 2 ? kOperandVgprsNarrow : kOperandVgprs;
  if (SW && GROUP) budget -= 16;
  int d = budget / per;
  return d < 1 ? 1 : (d > 16 ? 16 : d);
}

// Output of one element from its reduced accumulator.
struct Emit {
  const SmallMArgs& a;
  // per-channel: v = 16 * acc
  __device__ void channel(int row, int n, int v, float sx, float sw) const {
    const size_t o = (size_t)row * a.N + n;
    const int acc = v >> 4;
    if (a.out_kind == kOutI32) {
      static_cast<int*>(a.y)[o] = acc;
      return;
    }
    const float y32 = __fmul_rn(__fmul_rn((float)acc, sx), sw);
    if (a.out_kind == kOutF32)
      static_cast<float*>(a.y)[o] = y32;
    else
      static_cast<uint16_t*>(a.y)[o] = (uint16_t)f32_to_bf16(y32);
  }
  // group: t = sum_g p_g * s_g
  __device__ void group(int row, int n, float t, float sx) const {
    const size_t o = (size_t)row * a.N + n;
    const float y32 = __fmul_rn(t, sx);
    if (a.out_kind == kOutF32)
      static_cast<float*>(a.y)[o] = y32;
    else
      static_cast<uint16_t*>(a.y)[o] = (uint16_t)f32_to_bf16(y32);
  }
  // gated output column f from the fp32 gate and up values (the values the
  // plain linear would round to bf16): silu(g) * u, with
  // silu(g) = g / (1 + e^-g)
  __device__ void gated(int row, int f, float g, float u) const {
    const size_t o = (size_t)row * a.F + f;
    const float y32 = __fmul_rn(__fdiv_rn(g, __fadd_rn(1.0f, __expf(-g))), u);
    if (a.out_kind == kOutF32)
      static_cast<float*>(a.y)[o] = y32;
    else
      static_cast<uint16_t*>(a.y)[o] = (uint16_t)f32_to_bf16(y32);
  }
  __device__ float channel_value(int v, float sx, float sw) const {
    return __fmul_rn(__fmul_rn((float)(v >> 4), sx), sw);
  }
};

template <int MT, int NT, bool GROUP, int QM, bool EXACT, bool SWIGLU>
__global__ __launch_bounds__(kThreads) void smallm(const SmallMArgs a) {
  static_assert(!SWIGLU || NT % 2 == 0, "gated instances pair gate and up tiles");
  constexpr int HT = SWIGLU ? NT / 2 : NT;  // output column tiles per workgroup
  constexpr bool FUSED = QM != kQNone;
  constexpr int D = stage_depth(MT, NT, QM, GROUP, SWIGLU);
  extern __shared__ __align__(16) uint8_t lds[];
  uint32_t* l_amax = reinterpret_cast<uint32_t*>(lds);
  float* l_s = reinterpret_cast<float*>(lds + 64);
  float* l_inv = reinterpret_cast<float*>(lds + 128);
  int* l_mode = reinterpret_cast<int*>(lds + 192);
  uint8_t* l_body = lds + kLdsHeader;
  __shared__ int l_last;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  // Workgroups are dealt to the 8 XCDs round robin; renumber them so that
  // each XCD gets a contiguous range of column groups (its output rows then
  // share cache lines only at the 7 range boundaries, and its weight tiles
  // are one contiguous range).
  int bidx = blockIdx.x;
  if ((gridDim.x & 7) == 0) bidx = (bidx & 7) * (int)(gridDim.x >> 3) + (bidx >> 3);
  const int gid = bidx / a.S, split = bidx % a.S;
  const int M = a.M, N = a.N, K = a.K, KB = a.KB;
  const int ntiles = N / 16;
  const int nt0 = gid * NT;
  // Tile t < HT of this group is weight tile t0 + t; gated instances take
  // tile t >= HT (the up half) from the same columns F / 16 tiles on.
  const int t0 = gid * HT;
  const int u0 = SWIGLU ? a.F / 16 + t0 : t0 + HT;
  const int kb_begin = split * a.kbs;
  const int kb_end = min(KB, kb_begin + a.kbs);
  const int nkb = kb_end - kb_begin;
  // Uniform trip count (blocks per wave, rounded up): a wave's blocks past
  // the split read zeros; whole stages past it are skipped.
  const int iters = (nkb + kWaves - 1) / kWaves;
  const int r16 = lane & 15, g4 = lane >> 4;
  const int ldq = nkb * 128 + 16;  // fused: LDS row stride of the codes

  // The NT tiles of this group are contiguous in the packed layout; tiles
  // past N fall outside the resource and read as zeros.
  const int tiles_here = SWIGLU ? NT : min(NT, ntiles - nt0);
  const __amdgpu_buffer_rsrc_t wres = make_rsrc(a.wp + (size_t)t0 * KB * kBlockBytes,
                                                (uint32_t)((SWIGLU ? HT : tiles_here) * KB * kBlockBytes));
  const __amdgpu_buffer_rsrc_t wres_u =
      SWIGLU ? make_rsrc(a.wp + (size_t)u0 * KB * kBlockBytes, (uint32_t)(HT * KB * kBlockBytes)) : wres;
  const __amdgpu_buffer_rsrc_t sres =
      GROUP ? make_rsrc(static_cast<const uint16_t*>(a.w_scale) + t0 * 16,
                        (uint32_t)(((size_t)KB * N - t0 * 16) * 2))
            : wres;
  const __amdgpu_buffer_rsrc_t sres_u =
      GROUP && SWIGLU ? make_rsrc(static_cast<const uint16_t*>(a.w_scale) + u0 * 16,
                                  (uint32_t)(((size_t)KB * N - u0 * 16) * 2))
                      : sres;
  const __amdgpu_buffer_rsrc_t xres = make_rsrc(a.x, (uint32_t)((size_t)M * K * (FUSED ? 2 : 1)));

  // ---- fused quantize: load this thread's x chunks first, so that waiting
  // for them later does not wait for the weight stream issued after them.
  // Thread tid owns row tid / tpr and, of that row's K/8 16-byte chunks,
  // c8 = tid % tpr + tpr * j; chunks past the row read as zeros.
  // Every workgroup reads the rows in the same order: concurrent requests
  // for the same line then merge in L2.
  uint4 xc[QM == kQLds ? kXCache : 1];
  const int tpr = QM == kQLds ? a.tpr : 1;
  const int xrow = tid / tpr, xcol = tid % tpr;
  const int nchunk = K / 8;                  // a multiple of tpr (host-side condition)
  const int cpt = nchunk / tpr;              // chunk slots used per thread (<= kXCache)
  auto xchunk = [&](int j) { return xcol + tpr * j; };
  if constexpr (QM == kQLds) {
    // one vector offset per thread; the chunk step goes in the scalar offset
    const uint32_t xbase = xrow < M ? (uint32_t)((xrow * nchunk + xcol) * 16) : kOOB;
#pragma unroll
    for (int j = 0; j < kXCache; ++j)
      xc[j] = buf_load16s(xres, j < cpt ? xbase : kOOB, (uint32_t)(j * tpr * 16));
    if (tid < 16) l_amax[tid] = 0u;
  }

  // ---- weight stream, D stages deep
  uint4 wb[D][NT];
  uint4 ab[FUSED ? 1 : D][MT][2];
  uint16_t sgb[GROUP ? D : 1][NT];
  // Stage i of this wave covers block kb_begin + wave + 8 i of the split.
  auto stage_kb = [&](int i) { return kb_begin + wave + i * kWaves; };
  // The wave-uniform part of each offset (tile, block) goes in the scalar
  // offset; the lane part, or an out-of-range value, in the vector offset.
  auto load_stage = [&](int slot, int i) {
    const int kb = stage_kb(i);
    const bool ok = kb < kb_end;
    const uint32_t wv = ok ? (uint32_t)(lane * 16) : kOOB;
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const bool up = SWIGLU && t >= HT;
      const int tt = up ? t - HT : t;
      wb[slot][t] = buf_load16s<kCacheStream>(up ? wres_u : wres, wv, (uint32_t)((tt * KB + (ok ? kb : 0)) * kBlockBytes));
      if constexpr (GROUP)
        sgb[slot][t] = buf_load2s(up ? sres_u : sres, ok ? (uint32_t)((tt * 16 + r16) * 2) : kOOB,
                                  (uint32_t)((size_t)(ok ? kb : 0) * N * 2));
    }
    if constexpr (!FUSED) {
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const int row = mt * 16 + r16;
        const uint32_t off = ok && row < M ? (uint32_t)(row * K + g4 * 32) : kOOB;
        const uint32_t so = (uint32_t)((ok ? kb : 0) * 128);
        ab[slot][mt][0] = buf_load16s(xres, off, so);
        ab[slot][mt][1] = buf_load16s(xres, off == kOOB ? kOOB : off + 16, so);
      }
    }
  };
  // Without the LDS-mode quantize the whole prologue is issued at once.
  // Stages past this wave's last block are not issued (nor computed below):
  // with a short split, D can exceed the blocks a wave owns.  Group mode
  // issues them (they read zeros): guarding its loads made the compiler
  // spill the stage registers.
  // Issue order across the waves: the CU serves vector-memory requests
  // roughly in issue order, so a wave that issues its whole prologue at
  // once gets all of its blocks before the next wave gets any, and the last
  // waves then compute after the stream has ended.  A workgroup barrier
  // after stage s sends every wave's copy of stages 0 .. s ahead of the
  // rest.  Measured, us per call on int8 codes (none / after every stage /
  // after stage 0): down M = 1 6.35 / 6.30 / 6.46; O group M = 1
  // 5.28 / 4.84 / 5.24; qkv group M = 16 6.58 / 6.55 / 6.40; gate+up group
  // M = 1 10.9 / 10.9 / 10.16, M = 16 11.6 / 11.46 / 11.04; gate+up
  // channel M = 16 10.87 / 11.27 / 11.03.  So one column tile per wave takes
  // a barrier after every stage, the other group instances one after stage
  // 0, and the other per-channel instances none.
  constexpr int kIssueBarriers = NT == 1 ? D - 1 : (GROUP ? 1 : 0);
  if constexpr (QM != kQLds) {
#pragma unroll
    for (int s = 0; s < D; ++s) {
      if (EXACT || GROUP || s < iters) load_stage(s, s);
      if (s < kIssueBarriers) __builtin_amdgcn_s_barrier();
    }
  }

  // ---- epilogue scales, fetched now so their latency hides under the
  // weight stream.  Thread tid finishes outputs o = tid + q * threads.
  // Gated instances finish HT tiles of output columns, each from a gate
  // and an up column.
  constexpr int kOut = MT * 16 * HT * 16;
  constexpr int kOPT = (kOut + kThreads - 1) / kThreads;
  const bool scaled = a.out_kind != kOutI32;
  const __amdgpu_buffer_rsrc_t swres = make_rsrc(static_cast<const float*>(a.w_scale) + t0 * 16,
                                                 !GROUP && scaled ? (uint32_t)((SWIGLU ? HT : tiles_here) * 64) : 0u);
  const __amdgpu_buffer_rsrc_t swres_u =
      make_rsrc(static_cast<const float*>(a.w_scale) + u0 * 16, !GROUP && SWIGLU ? (uint32_t)(HT * 64) : 0u);
  const __amdgpu_buffer_rsrc_t sxres = make_rsrc(a.x_scale, !FUSED && scaled ? (uint32_t)(M * 4) : 0u);
  float swp[kOPT], sxp[kOPT], swu[SWIGLU ? kOPT : 1];
#pragma unroll
  for (int q = 0; q < kOPT; ++q) {
    const int o = tid + q * kThreads;
    const int row = o / (HT * 16), col = o % (HT * 16);
    const bool ok = o < kOut && row < M;
    swp[q] = __uint_as_float(buf_load4(swres, ok ? (uint32_t)(col * 4) : kOOB));
    if constexpr (SWIGLU) swu[q] = __uint_as_float(buf_load4(swres_u, ok ? (uint32_t)(col * 4) : kOOB));
    sxp[q] = __uint_as_float(buf_load4(sxres, ok ? (uint32_t)(row * 4) : kOOB));
  }

  // ---- LDS-mode quantize: absmax over the full rows, codes for this split
  if constexpr (QM == kQLds) {
    lds_barrier();  // l_amax initialised
    uint32_t pm = 0;
#pragma unroll
    for (int j = 0; j < kXCache; ++j) pm = absmax_chunk(pm, xc[j]);
    uint32_t v = fold_pair_max(pm);
    const int width = tpr < 64 ? tpr : 64;  // lanes of one row within a wave
    for (int off = width / 2; off >= 1; off >>= 1) {
      const uint32_t o = (uint32_t)__shfl_xor((int)v, off, 64);
      v = v > o ? v : o;
    }
    if (xrow < M && (lane & (width - 1)) == 0) atomicMax(&l_amax[xrow], v);
    lds_barrier();
    if (tid < M) {
      const QScale q = qscale_from_absmax(bf16_lo(l_amax[tid]));
      l_s[tid] = q.s;
      l_inv[tid] = q.inv;
      l_mode[tid] = q.mode;
    }
    lds_barrier();
    // The activation rows came in alone (the weight stream would have
    // queued them behind it).  Now start the weight stream one stage at a
    // time, quantizing a share of the chunks between stages: a wave that
    // issued its whole prologue at once would sit blocked on the memory
    // pipeline with its quantize work still ahead of it.
    const float qs = xrow < M ? l_s[xrow] : 0.0f, qinv = xrow < M ? l_inv[xrow] : 0.0f;
    const int qmode = xrow < M ? l_mode[xrow] : 0;
    const int k_lo = kb_begin * 128, k_hi = kb_end * 128;
    uint8_t* dst = l_body + min(xrow, M - 1) * ldq - k_lo;
    constexpr int kPer = (kXCache + D - 1) / D;  // chunks quantized after each stage
#pragma unroll
    for (int st = 0; st < D; ++st) {
      if (EXACT || GROUP || st < iters) load_stage(st, st);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int jj = 0; jj < kPer; ++jj) {
        const int j = st * kPer + jj;
        if (j < kXCache) {
          const int k = xchunk(j) * 8;
          if (xrow < M && j < cpt && k >= k_lo && k < k_hi)  // k < K since j < cpt
            *reinterpret_cast<uint2*>(dst + k) = quant_chunk(xc[j], qs, qinv, qmode);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
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

  // Stage s of the block at base: compute block i = base + s from slot s.
  // Group mode issues every tile's two MFMAs first and then the rescales,
  // so the MFMAs run back to back and the rescales of one tile do not wait
  // on the MFMA latency of the next.  Its partial sums are kept 16x too
  // large (the unpacked weights' factor, taken out exactly in the
  // epilogue), so the fp16 scale feeds the FMA directly: one
  // v_fma_mix_f32 per value, with no conversion or multiply of the scale.
  auto compute_stage = [&](int s, int i) {
    v4i alo[MT], ahi[MT];
    v4i pg[GROUP ? MT : 1][GROUP ? NT : 1];
    if constexpr (QM == kQLds) {
      // Rows past M and stages past the split read clamped LDS addresses:
      // their weights are zero, and rows past M are never stored.
      const int kb = min(stage_kb(i), kb_end - 1);
      const uint8_t* p = l_body + min(r16, M - 1) * ldq + (kb - kb_begin) * 128 + g4 * 32;
      alo[0] = *reinterpret_cast<const v4i*>(p);
      ahi[0] = *reinterpret_cast<const v4i*>(p + 16);
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
          pg[mt][t] = mfma16(alo[mt], blo, zero4);
          pg[mt][t] = mfma16(ahi[mt], bhi, pg[mt][t]);
        } else {
          acc[mt][t] = mfma16(alo[mt], blo, acc[mt][t]);
          acc[mt][t] = mfma16(ahi[mt], bhi, acc[mt][t]);
        }
      }
    }
    if constexpr (GROUP) {
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        const float sg = f16_to_f32(sgb[s][t]);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
          for (int r = 0; r < 4; ++r) facc[mt][t][r] = __fmaf_rn((float)pg[mt][t][r], sg, facc[mt][t][r]);
      }
    }
  };
  // Blocks with a successor refill each slot right after computing it; the
  // last block (its slots hold stages base .. base + D - 1) only computes.
  // Stages at or past iters are not computed, and in channel mode not
  // loaded either (wave-uniform branches): they would only read and
  // multiply zeros, which cost 9-14 % where D exceeds a wave's blocks
  // (K = 4096 at NT <= 2, K = 12288).
  // EXACT instances (the host picks them when every wave's block count is a
  // multiple of D, e.g. gate+up: 4 blocks per wave, 4 stages) run the loop
  // without the branches, which split the compiler's scheduling regions and
  // cost ~2 % there.
  int base = 0;
  for (; base + D < iters; base += D) {
#pragma unroll
    for (int s = 0; s < D; ++s) {
      compute_stage(s, base + s);
      if (EXACT || GROUP || base + s + D < iters) load_stage(s, base + s + D);
    }
  }
#pragma unroll
  for (int s = 0; s < D; ++s)
    if (EXACT || base + s < iters) compute_stage(s, base + s);

  // ---- reduce the waves' partial sums through LDS.  The partials get their
  // own region (past the codes in fused mode), so no barrier is needed
  // before writing them: one placed here was hoisted by the compiler into
  // the middle of the last stages' MFMAs, which cost 0.66 us on gate+up.
  uint32_t* red = reinterpret_cast<uint32_t*>(
      l_body + (QM == kQLds ? ((size_t)M * (a.kbs * 128 + 16) + 15) / 16 * 16 : 0));
  // Lane l holds rows 4 (l >> 4) + i (i < 4) of column l & 15 of each 16 x
  // 16 tile; value i goes to word i 64 + l of the wave's tile, so that the
  // reads below (one row, consecutive columns across the lanes) are
  // consecutive words, and the skewed tile pitch spreads neighbouring tiles
  // over the banks.  (Each lane's four values as one 16-byte write left
  // every column four words apart and every tile on the same banks: 4-way
  // conflicts on every read of the reduction.)
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      uint32_t* dst = red + ((wave * MT + mt) * NT + t) * kRedTile + lane;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        if constexpr (GROUP)
          dst[i * 64] = __float_as_uint(facc[mt][t][i]);
        else
          dst[i * 64] = (uint32_t)acc[mt][t][i];
      }
    }
  lds_barrier();

  const Emit emit{a};
  auto wave_sum_f = [&](int mt, int t, int src) {
    float v = 0.0f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) v += __uint_as_float(red[((w * MT + mt) * NT + t) * kRedTile + src]);
    return v * 0.0625f;  // every partial and sum above is 16x the true one: exact barring underflow
  };
  auto wave_sum_i = [&](int mt, int t, int src) {
    int v = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) v += (int)red[((w * MT + mt) * NT + t) * kRedTile + src];
    return v;
  };
#pragma unroll
  for (int q = 0; q < kOPT; ++q) {
    const int o = tid + q * kThreads;
    const int row = o / (HT * 16), col = o % (HT * 16);
    const int mt = row >> 4, rr = row & 15, t = col >> 4, cc = col & 15;
    if (o >= kOut || row >= M || t >= tiles_here) continue;
    if constexpr (FUSED) sxp[q] = l_s[row];
    const int src = (rr & 3) * 64 + (rr >> 2) * 16 + cc;
    const int n = (t0 + t) * 16 + cc;      // (gate) column
    const int nu = (u0 + t) * 16 + cc;     // up column (gated instances)
    if constexpr (GROUP) {
      const float v = wave_sum_f(mt, t, src);
      const float vu = SWIGLU ? wave_sum_f(mt, t + HT, src) : 0.0f;
      if (a.S == 1) {
        if constexpr (SWIGLU)
          emit.gated(row, n, __fmul_rn(v, sxp[q]), __fmul_rn(vu, sxp[q]));
        else
          emit.group(row, n, v, sxp[q]);
      } else {
        float* part = static_cast<float*>(a.partial) + ((size_t)split * M + row) * N;
        part[n] = v;
        if constexpr (SWIGLU) part[nu] = vu;
      }
    } else {
      const int v = wave_sum_i(mt, t, src);
      const int vu = SWIGLU ? wave_sum_i(mt, t + HT, src) : 0;
      if (a.S == 1) {
        if constexpr (SWIGLU)
          emit.gated(row, n, emit.channel_value(v, sxp[q], swp[q]), emit.channel_value(vu, sxp[q], swu[q]));
        else
          emit.channel(row, n, v, sxp[q], swp[q]);
      } else {
        int* part = static_cast<int*>(a.partial) + ((size_t)split * M + row) * N;
        part[n] = v;
        if constexpr (SWIGLU) part[nu] = vu;
      }
    }
  }
  if (a.S == 1) return;

  // ---- split-K: the last workgroup of this column group finishes.
  // One agent-scope acquire-release RMW per workgroup, by one thread: the
  // barrier before it orders every wave's partial stores before the release,
  // and the barrier after it orders the acquire before every wave's reads.
  // (A device-scope fence in every wave instead made each call 40-100 us
  // slower: each one writes back or invalidates the whole L2 of its XCD.)
  __syncthreads();
  if (tid == 0) {
    const unsigned prev = __hip_atomic_fetch_add(&a.counters[gid], 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
    l_last = prev == (unsigned)(a.S - 1);
  }
  __syncthreads();
  if (!l_last) return;
#pragma unroll
  for (int q = 0; q < kOPT; ++q) {
    const int o = tid + q * kThreads;
    const int row = o / (HT * 16), col = o % (HT * 16);
    const int t = col >> 4, cc = col & 15;
    if (o >= kOut || row >= M || t >= tiles_here) continue;
    const int n = (t0 + t) * 16 + cc;
    const int nu = (u0 + t) * 16 + cc;
    if constexpr (GROUP) {
      const float* part = static_cast<const float*>(a.partial);
      float v = 0.0f, vu = 0.0f;
      for (int s = 0; s < a.S; ++s) {
        v += part[((size_t)s * M + row) * N + n];
        if constexpr (SWIGLU) vu += part[((size_t)s * M + row) * N + nu];
      }
      if constexpr (SWIGLU)
        emit.gated(row, n, __fmul_rn(v, sxp[q]), __fmul_rn(vu, sxp[q]));
      else
        emit.group(row, n, v, sxp[q]);
    } else {
      const int* part = static_cast<const int*>(a.partial);
      int v = 0, vu = 0;
      for (int s = 0; s < a.S; ++s) {
        v += part[((size_t)s * M + row) * N + n];
        if constexpr (SWIGLU) vu += part[((size_t)s * M + row) * N + nu];
      }
      if constexpr (SWIGLU)
        emit.gated(row, n, emit.channel_value(v, sxp[q], swp[q]), emit.channel_value(vu, sxp[q], swu[q]));
      else
        emit.channel(row, n, v, sxp[q], swp[q]);
    }
  }
  if (tid == 0) __hip_atomic_store(&a.counters[gid], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

typedef void (*SmallMKernel)(const SmallMArgs);

// MT * NT is capped at 12 (kMaxTilesPerWave): beyond it the accumulators
// and in-flight operands no longer fit in 256 registers.  Group kernels
// have no EXACT form (the planner never asks for one); gated kernels need
// an even NT.
template <int MT, int NT, bool GROUP, int QM, bool SW>
SmallMKernel instance(bool exact) {
  if constexpr (MT * NT > kMaxTilesPerWave || (QM != kQNone && MT != 1) || (SW && NT % 2))
    return nullptr;
  else if constexpr (GROUP)
    return exact ? nullptr : smallm<MT, NT, GROUP, QM, false, SW>;
  else
    return exact ? smallm<MT, NT, GROUP, QM, true, SW> : smallm<MT, NT, GROUP, QM, false, SW>;
}

template <int MT, bool GROUP, int QM, bool SW>
SmallMKernel pick_nt(int NT, bool exact) {
  switch (NT) {
    case 1: return instance<MT, 1, GROUP, QM, SW>(exact);
    case 2: return instance<MT, 2, GROUP, QM, SW>(exact);
    case 3: return instance<MT, 3, GROUP, QM, SW>(exact);
    case 4: return instance<MT, 4, GROUP, QM, SW>(exact);
    case 6: return instance<MT, 6, GROUP, QM, SW>(exact);
    default: return nullptr;
  }
}

template <bool GROUP, bool SW>
SmallMKernel pick_group(const SmallMPlan& p) {
  if (p.qmode == kQLds) return pick_nt<1, GROUP, kQLds, SW>(p.NT, p.exact);
  switch (p.MT) {
    case 1: return pick_nt<1, GROUP, kQNone, SW>(p.NT, p.exact);
    case 2: return pick_nt<2, GROUP, kQNone, SW>(p.NT, p.exact);
    case 4: return pick_nt<4, GROUP, kQNone, SW>(p.NT, p.exact);
    default: return nullptr;
  }
}

SmallMKernel pick(const SmallMPlan& p) {
  if (p.swiglu) return p.group ? pick_group<true, true>(p) : pick_group<false, true>(p);
  return p.group ? pick_group<true, false>(p) : pick_group<false, false>(p);
}

}  // namespace

// Plan cost model.  Candidates (column tiles per workgroup NT, K splits S)
// are compared on
//   (rounds - 1) * kRoundUs
//   + max(all bytes / kHbmGBs, rounds * bytes per workgroup / kCuGBs)
//   + kSplitUs if K is split,
// where rounds = workgroup rounds over the 256 CUs and a workgroup's bytes
// are its packed weights plus half of the activation codes it reads.  The
// whole chip streams ~6.5 TB/s, one workgroup at most ~60 GB/s; a second
// round of workgroups costs its own ramp-up and drain; a K split adds a
// serial chain (partial stores, the arrival counter, the finishing
// workgroup's reads).  With the layer shapes this keeps S = 1 (the
// partial-sum handoff never pays off below ~400 KB of weights per
// workgroup) and picks the narrowest column group that still fits one
// round; the split choices were checked on the GPU at K = 65536.
// The launch's estimated time (SmallMPlan::model_us, shown by the plan
// description) adds what every candidate pays alike, or what was measured
// only without a split:
//   kFixedUs (dispatch, the first bytes' latency, the wave reduction and
//   epilogue, the drain) + the workgroup's codes / kActGBs (read from L2
//   beyond the weight stream) + kGroupUs with group scales (their
//   scattered loads and the rescale).
// Against the kernel-trace averages of the layer shapes (gate+up, qkv, O,
// down at M = 1, 4, 16, both scale modes) the estimate is within ~13 %.
constexpr double kRoundUs = 1.5;
constexpr double kHbmGBs = 6500.0;
constexpr double kCuGBs = 60.0;
constexpr double kSplitUs = 5.0;
constexpr double kFixedUs = 3.2;
constexpr double kActGBs = 70.0;
constexpr double kGroupUs = 1.0;

SmallMPlan plan_smallm(int M, int N, int K, bool group, bool bf16_in, bool swiglu) {
  SmallMPlan p{};
  p.MT = M <= 16 ? 1 : (M <= 32 ? 2 : 4);
  p.group = group;
  p.swiglu = swiglu;
  const int ntiles = N / 16, KB = K / 128;
  const int nts[] = {1, 2, 3, 4, 6};
  const int ss[] = {1, 2, 4, 8};
  const double all_bytes = (double)N * K / 2;
  double best = 1e30;
  for (int nt : nts) {
    // a gated group pairs nt / 2 gate tiles with the up tiles of the same columns
    if (ntiles % nt || p.MT * nt > kMaxTilesPerWave || (swiglu && nt % 2)) continue;
    for (int s : ss) {
      if (s > KB) continue;
      const int kbs = (KB + s - 1) / s;
      const long wgs = (long)(ntiles / nt) * s;
      const long rounds = (wgs + 255) / 256;
      // weights, plus the activation codes every workgroup reads (from L2,
      // counted at half weight)
      const double codes = (double)M * kbs * 128;
      const double wg_bytes = (double)nt * kbs * kBlockBytes + 0.5 * codes;
      double us = (double)(rounds - 1) * kRoundUs +
                  fmax(all_bytes / (kHbmGBs * 1e3), (double)rounds * wg_bytes / (kCuGBs * 1e3));
      if (s > 1) us += kSplitUs;
      if (us < best - 1e-9) {
        best = us;
        p.NT = nt;
        p.S = s;
        p.groups = ntiles / nt;
        p.model_us = us + kFixedUs + codes / (kActGBs * 1e3) + (group ? kGroupUs : 0.0);
      }
    }
  }
  const int kbs = (KB + p.S - 1) / p.S;
  int mp = 1;
  while (mp < M) mp *= 2;
  p.tpr = kThreads / (mp < 16 ? mp : 16);
  // Fused quantize only for narrow column groups over a very long K.  Every
  // workgroup reads the whole token rows before its weight stream starts,
  // and that read alone takes ~3.5 us (a timeline of the down projection,
  // K = 12288, M = 1: rows in at 3.6 us, weights issued from 4.3 us); a
  // separate quantize launch costs ~3 us, the launch floor being ~2.4 us.
  // Measured down projection, us per call: M = 1: fused 10.4, separate
  // 9.5; M = 4: 10.4 against 9.7.  With NT >= 3 the deeper weight prologue
  // also stalls the waves at issue while the quantize work is still ahead.
  p.qmode = kQNone;
  if (bf16_in && p.MT == 1 && p.NT <= kMaxFusedTiles && KB >= kFusedMinKB && (K / 8) % p.tpr == 0 &&
      (K / 8) / p.tpr <= kXCache && (size_t)M * (kbs * 128 + 16) <= 96 * 1024)
    p.qmode = kQLds;
  p.fused = p.qmode != kQNone;
  // Every split's waves own a multiple of D blocks: the loop needs no
  // guards (the last split may be shorter).  Group kernels always take the
  // guarded loop, which measured faster for them even where no stage is
  // skipped (gate+up, M = 1 and 16).
  {
    const int D = stage_depth(p.MT, p.NT, p.qmode, group, swiglu);
    const int last = KB - (p.S - 1) * kbs;
    const int it_full = (kbs + kWaves - 1) / kWaves, it_last = (last + kWaves - 1) / kWaves;
    p.exact = !group && it_full % D == 0 && it_last % D == 0;
  }
  const size_t red = (size_t)kWaves * p.MT * p.NT * kRedTile * 4;
  const size_t codes = p.qmode == kQLds ? ((size_t)M * (kbs * 128 + 16) + 15) / 16 * 16 : 0;
  p.lds_bytes = kLdsHeader + codes + red;
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
  static thread_local char buf[128];
  static const char* modes[] = {"int8-in", "fused-quant"};
  snprintf(buf, sizeof buf, "smallm<MT=%d,NT=%d,%s,%s%s> S=%d groups=%d model=%.1fus", p.MT, p.NT,
           p.group ? "group" : "channel", modes[p.qmode], p.swiglu ? ",swiglu" : "", p.S, p.groups, p.model_us);
  return buf;
}

}  // namespace w4a8
