// Large-M W4A8 GEMM kernel template (streaming prefill of new-frame tokens,
// M > 64), included by gemm_largem.hip (per-channel scales) and
// gemm_largem_group.hip (group scales; built with VGPR-form MFMAs).
//
// At large M the layer is bound by the INT8 contraction (FlashDrive
// Sec. 4.2: prefill gains from the INT8 matrix units), so the kernels keep
// the matrix cores fed:
//   - a BM x BN output tile per workgroup, 128 k per step (one scale group);
//     tile sizes are picked on the host so that the tile count fills the 256
//     CUs in whole waves;
//   - each step's int8 activation tile and packed int4 weight tile travel
//     from HBM straight into one stage of a 4-deep LDS ring
//     (buffer_load_dwordx4 ... lds: no registers, no VALU).  Right after the
//     barrier of step kb, step kb + 4 refills step kb's stage, whose operands
//     are already in registers, so three steps of MFMA work cover the load
//     latency;
//   - every load instruction writes 1 KiB of LDS contiguously; activation
//     rows land XOR-swizzled (16-byte chunk c of row r at c ^ ((r >> 1) & 7))
//     because each lane fetches the global chunk that belongs at its LDS
//     position.  ds_read_b128 serves 16 lanes (256 bytes of banks) per
//     clock; with 128-byte rows, the 16 rows an operand read touches in one
//     clock then fall on 16 distinct 16-byte bank groups (a swizzle on r & 7
//     left rows r and r + 8 on the same banks and halved the read rate).
//     Weight chunks keep the packed order, already conflict free;
//   - the ring keeps the activation tiles of its 4 stages together, then
//     their weight tiles, then their scales, and the step loop is unrolled
//     over the 4 stages: every operand read is one per-lane address plus
//     the stage's immediate offset, with no address arithmetic in the loop
//     (3-9 % faster than per-stage blocks with the stage added per read);
//   - the operands of step kb + 1 are read from LDS into a second register
//     set between the MFMAs of step kb (v_mfma_i32_32x32x32_i8), and every
//     other instruction of a step (stage fill, LDS reads, nibble unpack) is
//     dealt out evenly between the MFMAs;
//   - workgroups are renumbered so that the tiles given to one XCD (the
//     hardware deals workgroups to the 8 XCDs round robin) share their
//     weight columns in that XCD's L2.
// The epilogue applies per-token and per-channel scales (or, in group mode,
// each step's int32 partial is rescaled by its fp16 group scale into an
// fp32 accumulator), stages the output tile in the idle LDS ring and writes
// it as 16-byte row chunks.
// SW (gated) instances serve the fused gate+up projection with its gated
// activation merged in (FlashDrive Sec. 3.5, Kernel Fusion): of a wave's WN
// (even) 32-column blocks, the first WN / 2 hold gate columns and the rest
// the up columns of the same outputs, and the tile writes silu(g) * u,
// BN / 2 columns of y.
#pragma once
#include <type_traits>

#include "device.h"
#include "kernels.h"

namespace w4a8 {

namespace {

// The tile menu: BM = 32 WM GM rows, BN = 32 WN GN columns, ring = LDS
// stages in flight.  The small tiles' stages are small, so they keep more of
// them in flight to cover the L2 latency.
struct TileCfg {
  int WM, WN, GM, GN, ring;
  int ks;          // k groups of GM x GN waves (each with ring / ks stages)
  double quality;  // relative efficiency of the tile shape (operand reuse)
  bool group_ok;   // fits the registers with group-mode accumulators
  bool plain_ok;   // serves the plain output (its fp32 tile fits the LDS ring)
  bool gated_ok;   // serves the gated output (an even number of blocks per wave)
};
// The weights come from plan sweeps of the layer shapes at M = 256..2048 in
// both scale modes.  A 64 x 96 tile (two waves) lost to 64 x 64 wherever it
// was chosen (group qkv at M = 256: 23.4 against 16.4 us) and was dropped.
// 128 x 256 serves only the gated output: its plain fp32 tile (133 KB)
// would not fit the 128 KB ring, the gated one (64 KB) does.
constexpr TileCfg kMenu[] = {
    {2, 3, 2, 2, 4, 1, 1.00, false, true, false},  // 128 x 192, 4 waves
    {2, 2, 2, 2, 4, 1, 0.95, true, true, true},    // 128 x 128, 4 waves
    {1, 1, 2, 2, 4, 1, 0.80, true, true, false},   // 64 x 64, 4 waves
    {2, 4, 2, 2, 4, 1, 1.05, false, false, true},  // 128 x 256, 4 waves (gated)
    // 64 x 64 with two k groups (8 waves, two per SIMD, an 8-deep ring):
    // taken in place of entry 2 when the tiles fill at most one round, i.e.
    // one workgroup per CU, where a single wave per SIMD leaves the SIMD
    // idle between its MFMA and VALU bursts
    {1, 1, 2, 2, 8, 2, 0.80, false, false, false},
};
constexpr int kMenuKSplit = 4;  // the k-split form of entry 2
constexpr int kMenuSize = sizeof(kMenu) / sizeof(kMenu[0]);

template <int WM, int WN, int GM, int GN, bool GROUP, int kRing, bool SW, int KS = 1>
__global__ __launch_bounds__(GM * GN * 64 * KS) void largem(const LargeMArgs a) {
  static_assert(!SW || WN % 2 == 0, "gated tiles pair gate and up blocks per wave");
  // KS k groups of GM x GN waves: group wk takes the steps kb = KS i + wk
  // with its own kRing / KS stages of the ring (stage KS s + wk), and the
  // groups' sums meet in LDS at the end
  constexpr int kThreads = GM * GN * 64;  // threads of one k group
  constexpr int kWaves = GM * GN;         // waves of one k group
  constexpr int kOwnRing = kRing / KS;    // ring stages of one k group
  static_assert(kRing % KS == 0, "every k group owns whole ring stages");
  constexpr int BM = 32 * WM * GM, BN = 32 * WN * GN;
  constexpr int kABytes = BM * 128, kBBytes = BN / 16 * kBlockBytes;
  constexpr int kSBytes = GROUP ? kWaves * 256 : 0;  // group scales: 256 B per wave
  constexpr int kStage = kABytes + kBBytes + kSBytes;
  // LDS: the activation tiles of all ring stages first, then the weight
  // tiles, then the group scales, so that an operand read is one per-lane
  // address plus the stage's immediate offset (the activation region of a
  // 4-deep ring of 128-row tiles is exactly 64 KiB, the immediate's range).
  constexpr int kAReg = kRing * kABytes, kBReg = kRing * kBBytes;
  static_assert(kOwnRing == 4, "the step loop is unrolled over a k group's 4 ring stages");
  constexpr int kACh = kABytes / 16 / kThreads, kBCh = kBBytes / 16 / kThreads;  // loads per thread per stage
  static_assert(kACh * kThreads * 16 == kABytes, "A tile must split evenly over the threads");
  static_assert(kBCh * kThreads * 16 == kBBytes, "B tile must split evenly over the threads");
  constexpr int kSPerWave = BN / kWaves;                 // group scales each wave fetches
  static_assert(!GROUP || (kSPerWave * kWaves == BN && kSPerWave % 2 == 0 && kSPerWave <= 128),
                "group scales must split evenly, two per lane");
  constexpr int kPerStage = kACh + kBCh + (GROUP ? 1 : 0);  // vector-memory instructions per stage
  extern __shared__ __align__(16) uint8_t lds[];

  int bid = blockIdx.x;
  const int total = (int)gridDim.x;  // tiles_m * tiles_n (the host keeps it below 2^31)
  if (a.xcd_remap) bid = (bid & 7) * (total >> 3) + (bid >> 3);
  const int tm = bid % a.tiles_m, tn = bid / a.tiles_m;
  // Gated tiles: tile columns [0, BN/2) are gate columns f0 .., [BN/2, BN)
  // the up columns F + f0 ..; output columns f0 .. f0 + BN/2.
  constexpr int OBN = SW ? BN / 2 : BN;  // output columns per tile
  const int m0 = tm * BM, n0 = tn * BN, nt0 = n0 / 16;
  const int f0 = tn * OBN, ft0 = f0 / 16, fu0 = a.F / 16 + ft0;
  const int tid = (int)threadIdx.x % kThreads, lane = tid & 63;  // within the k group
  const int wk = __builtin_amdgcn_readfirstlane((int)threadIdx.x / kThreads);
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave % GM, wn = wave / GM;
  const int M = a.M, N = a.N, K = a.K, KB = a.KB;
  const int ntiles = N / 16;
  const int l32 = lane & 31, g2 = lane >> 5;

  // Per-tile buffer descriptors: rows past M and tiles past N lie outside
  // them and read as zeros (no branch, no traffic).
  const int rows_here = min(BM, M - m0);
  // (gated: per half, the tiles and columns inside [0, F))
  const int tiles_here = SW ? min(OBN / 16, a.F / 16 - ft0) : min(BN / 16, ntiles - nt0);
  const int cols_here = SW ? min(OBN, a.F - f0) : min(BN, N - n0);
  const u32x4 ares = make_rsrc_words(a.xq + (size_t)m0 * K, (uint32_t)(rows_here * K));
  const u32x4 bres = make_rsrc_words(a.wp + (size_t)(SW ? ft0 : nt0) * KB * kBlockBytes,
                                     (uint32_t)(tiles_here * KB * kBlockBytes));
  const u32x4 bres_u =
      SW ? make_rsrc_words(a.wp + (size_t)fu0 * KB * kBlockBytes, (uint32_t)(tiles_here * KB * kBlockBytes)) : bres;
  const int sc0 = SW ? f0 : n0, scu = SW ? a.F + f0 : n0;  // first scale column of each half
  const u32x4 sres = make_rsrc_words(static_cast<const uint16_t*>(a.w_scale) + sc0,
                                     GROUP ? (uint32_t)(((size_t)KB * N - sc0) * 2) : 0u);
  const u32x4 sres_u = SW ? make_rsrc_words(static_cast<const uint16_t*>(a.w_scale) + scu,
                                            GROUP ? (uint32_t)(((size_t)KB * N - scu) * 2) : 0u)
                          : sres;
  const uint32_t lds_base = (uint32_t)(uintptr_t)lds;

  // Load j of this thread for the A part covers LDS chunk p = j * threads +
  // tid of the stage, i.e. row p / 8, physical chunk p % 8, which holds the
  // logical chunk (p % 8) ^ (row % 8).  Each wave instruction fills 1 KiB.
  uint32_t a_voff[kACh];
#pragma unroll
  for (int j = 0; j < kACh; ++j) {
    const int p = j * kThreads + tid;
    const int row = p >> 3, ch = (p & 7) ^ ((row >> 1) & 7);
    a_voff[j] = (uint32_t)(row * K + ch * 16);
  }
  // group scales: wave w fetches columns [w kSPerWave, +kSPerWave), two per
  // lane (4 bytes); lanes past that and columns past N read zeros.  Gated
  // tiles: the waves of the second half fetch the up columns.
  const bool s_up = SW && wave * kSPerWave >= OBN;
  const int scol = wave * kSPerWave - (s_up ? OBN : 0) + 2 * lane;
  const uint32_t s_voff = GROUP && 2 * lane < kSPerWave && scol < cols_here ? (uint32_t)(scol * 2) : kOOB;

  // Vector-memory instruction d of step kb's stage fill (A loads, then B
  // loads, then the group scales).  Past the end the loads read zeros
  // without traffic, so every step issues the same kPerStage instructions.
  // Gated tiles: blocks [0, BN/32) of the stage are gate tiles, the rest the
  // up tiles of the same columns.
  uint32_t b_voff[kBCh];
  bool b_up[kBCh];
#pragma unroll
  for (int j = 0; j < kBCh; ++j) {
    const int blk = j * kWaves + wave;
    b_up[j] = SW && blk >= BN / 32;
    b_voff[j] = (uint32_t)(lane * 16 + (blk - (b_up[j] ? BN / 32 : 0)) * KB * kBlockBytes);
  }
  // A step past the end gets the scalar offset kOOB: every lane's offset
  // then lies past the descriptor's range (no vector select needed).
  auto issue_one = [&](int kb, int stage, int d) {
    const bool ok = kb < KB;
    if (d < kACh) {
      lds_dma16(ares, lds_base + (uint32_t)((KS * stage + wk) * kABytes + (d * kWaves + wave) * 1024), a_voff[d],
                ok ? kb * 128 : kOOB);
    } else if (d < kACh + kBCh) {
      const int blk = (d - kACh) * kWaves + wave;
      lds_dma16_nt(b_up[d - kACh] ? bres_u : bres, lds_base + (uint32_t)(kAReg + (KS * stage + wk) * kBBytes + blk * 1024),
                   b_voff[d - kACh], ok ? kb * kBlockBytes : kOOB);
    } else if constexpr (GROUP) {
      lds_dma4(s_up ? sres_u : sres, lds_base + (uint32_t)(kAReg + kBReg + (KS * stage + wk) * kSBytes + wave * 256), s_voff,
               ok ? (uint32_t)((size_t)kb * N * 2) : kOOB);
    }
  };

  // LDS read offsets of this lane's MFMA operands: activation row
  // wm 32 WM + 32 i + l32 (its chunks c sit at c ^ ((row >> 1) & 7)), weight column
  // wn 32 WN + 32 j + l32 of the stage's weight tiles (gated: column
  // (j >= WN/2) BN/2 + 32 (WN/2) wn + 32 (j mod WN/2) + l32: blocks below
  // WN/2 in the gate half, the rest in the up half).
  constexpr int HW = SW ? WN / 2 : WN;  // blocks per wave in each half
  auto tile_col = [&](int j) {
    return SW ? (j >= HW ? BN / 2 : 0) + wn * 32 * HW + (j % HW) * 32 + l32 : wn * 32 * WN + j * 32 + l32;
  };
  const int swz = (l32 >> 1) & 7;
  uint32_t a_rd[WM], b_rd[WN];
#pragma unroll
  for (int i = 0; i < WM; ++i) a_rd[i] = (uint32_t)(wk * kABytes + (wm * 32 * WM + i * 32 + l32) * 128);
#pragma unroll
  for (int j = 0; j < WN; ++j) {
    const int col = tile_col(j);
    b_rd[j] = (uint32_t)(kAReg + wk * kBBytes + (col >> 4) * kBlockBytes + (col & 15) * 16);
  }
  // MFMA k half tp covers the 64 k of chunk group g = 2 tp + g2: activation
  // chunks 2 g and 2 g + 1, weight chunk g (low nibbles, then high nibbles).
  uint32_t a_ch[4];
#pragma unroll
  for (int tp = 0; tp < 2; ++tp) {
    const int g = 2 * tp + g2;
    a_ch[2 * tp] = (uint32_t)(((2 * g) ^ swz) << 4);
    a_ch[2 * tp + 1] = (uint32_t)(((2 * g + 1) ^ swz) << 4);
  }
  uint32_t a_addr[WM][4];
#pragma unroll
  for (int i = 0; i < WM; ++i)
#pragma unroll
    for (int c = 0; c < 4; ++c) a_addr[i][c] = a_rd[i] + a_ch[c];
  uint32_t s_rd[GROUP ? WN : 1];
#pragma unroll
  for (int j = 0; j < (GROUP ? WN : 1); ++j) {
    const int col = tile_col(j);
    s_rd[j] = (uint32_t)(kAReg + kBReg + wk * kSBytes + (col / kSPerWave) * 256 + (col % kSPerWave) * 2);
  }

  // One step's MFMA operands, held in registers so that the LDS reads of
  // step kb + 1 overlap the MFMAs of step kb.
  struct Ops {
    v4i a[WM][4];             // activation chunks of both k halves
    uint4 b[WN][2];           // packed weight chunk of both k halves
    v4i lo0[WN], hi0[WN];     // k half 0's weight nibbles, unpacked ahead of the step
    v4i lo1[GROUP ? WN : 1], hi1[GROUP ? WN : 1];  // group mode: k half 1's too
    float sg[GROUP ? WN : 1];
  };
  constexpr int kReadsTp = 2 * WM + WN;
  constexpr int kReads = 2 * kReadsTp + (GROUP ? WN : 0);  // LDS reads per step
  // LDS read r of step kb's operands: per k half the weight chunks first
  // (half 0's are unpacked while the previous step still runs), then the
  // activation chunks; the group scales last.
  // (stage_c: the ring stage, a compile-time constant, so that its offset
  // is the instruction's immediate)
  auto read_one = [&](auto stage_c, int r, Ops& o) {
    constexpr int S = decltype(stage_c)::value;
    if (r < 2 * kReadsTp) {
      const int tp = r / kReadsTp, u = r % kReadsTp;
      if (u < WN)
        o.b[u][tp] = *reinterpret_cast<const uint4*>(lds + S * KS * kBBytes + b_rd[u] + (2 * tp + g2) * 256);
      else if constexpr (GROUP) {
        // Group mode reads the activation operands straight into AGPRs
        // (only the MFMA reads them), which leaves the VGPRs to the int32
        // partial sums the rescale reads.  They are used in the next step,
        // whose barrier waits for every outstanding LDS read.
        const uint32_t addr = lds_base + a_addr[(u - WN) / 2][2 * tp + ((u - WN) & 1)];
        v4i t;
        asm volatile("ds_read_b128 %0, %1 offset:%2" : "=a"(t) : "v"(addr), "i"(S * KS * kABytes) : "memory");
        o.a[(u - WN) / 2][2 * tp + ((u - WN) & 1)] = t;
      } else {
        o.a[(u - WN) / 2][2 * tp + ((u - WN) & 1)] =
            *reinterpret_cast<const v4i*>(lds + S * KS * kABytes + a_addr[(u - WN) / 2][2 * tp + ((u - WN) & 1)]);
      }
    } else if constexpr (GROUP) {
      const int j = r - 2 * kReadsTp;
      o.sg[j] = f16_to_f32(*reinterpret_cast<const uint16_t*>(lds + S * KS * kSBytes + s_rd[j])) * 0.0625f;
    }
  };

  // The epilogue's scales: four consecutive rows' token scales per 16-byte
  // load (rows 8 q + 4 g2 + e of block i), one channel scale per column
  // block.  Channel mode fetches them now, so that their latency hides
  // behind the main loop; group mode, short of registers, after it.
  const bool scaled = a.out_kind != kOutI32;
  const __amdgpu_buffer_rsrc_t xsres =
      make_rsrc(uniform_ptr(a.x_scale + m0), uniform_u32(scaled ? (uint32_t)(rows_here * 4) : 0u));
  const __amdgpu_buffer_rsrc_t wsres = make_rsrc(uniform_ptr(static_cast<const float*>(a.w_scale) + sc0),
                                                 uniform_u32((!GROUP && scaled) ? (uint32_t)(cols_here * 4) : 0u));
  const __amdgpu_buffer_rsrc_t wsres_u = make_rsrc(uniform_ptr(static_cast<const float*>(a.w_scale) + scu),
                                                   uniform_u32((SW && !GROUP) ? (uint32_t)(cols_here * 4) : 0u));
  float swv[WN];
#pragma unroll
  for (int j = 0; j < WN; ++j)
    swv[j] = SW ? __uint_as_float(buf_load4(j >= HW ? wsres_u : wsres, (uint32_t)((wn * 32 * HW + (j % HW) * 32 + l32) * 4)))
                : __uint_as_float(buf_load4(wsres, (uint32_t)((wn * 32 * WN + j * 32 + l32) * 4)));
  uint4 sx4[WM][4];
  auto load_sx = [&]() {
#pragma unroll
    for (int i = 0; i < WM; ++i)
#pragma unroll
      for (int q = 0; q < 4; ++q)
        sx4[i][q] = buf_load16(xsres, (uint32_t)((wm * 32 * WM + i * 32 + 8 * q + 4 * g2) * 4));
  };
  if constexpr (!GROUP) load_sx();

  // Channel mode accumulates every step into acc[0].  Group mode rescales
  // each step's int32 partial into facc: with the 64 x 64 tile the steps
  // alternate between two accumulator sets so that the rescale of one
  // overlaps the MFMAs of the next; the larger tiles use one set (see
  // step1 below).
  v16i acc[GROUP ? 2 : 1][WM][WN];
  float facc[GROUP ? WM : 1][GROUP ? WN : 1][16];
#pragma unroll
  for (int h = 0; h < (GROUP ? 2 : 1); ++h)
#pragma unroll
    for (int i = 0; i < WM; ++i)
#pragma unroll
      for (int j = 0; j < WN; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[h][i][j][r] = 0;
  if constexpr (GROUP)
#pragma unroll
    for (int i = 0; i < WM; ++i)
#pragma unroll
      for (int j = 0; j < WN; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) facc[i][j][r] = 0.0f;

  // Unpacking one 4-byte word of packed weights into its low- and
  // high-nibble MFMA operand words.
  // Written as assembly so that the compiler keeps each unpack in the MFMA
  // slot it is dealt to instead of gathering them in front of their first
  // use.
  auto unpack_word = [](const uint4& c, int e, v4i& lo, v4i& hi) {
    const uint32_t w = e == 0 ? c.x : e == 1 ? c.y : e == 2 ? c.z : c.w;
    int l, h;
    asm volatile(
        "v_lshlrev_b32 %0, 4, %2\n\t"
        "v_and_b32 %0, 0xf0f0f0f0, %0\n\t"
        "v_and_b32 %1, 0xf0f0f0f0, %2"
        : "=&v"(l), "=&v"(h)
        : "v"(w));
    lo[e] = l;
    hi[e] = h;
  };
  auto unpack0 = [&](Ops& o, int u) {  // word u of k half 0
    unpack_word(o.b[u / 4][0], u % 4, o.lo0[u / 4], o.hi0[u / 4]);
  };

  // Step kb: wait for stage kb + 1 (this wave's loads: at most kRing - 2
  // younger stages outstanding); barrier: every wave's loads of stage kb + 1
  // are visible, and every wave has finished reading step kb's operands out
  // of stage kb (the fence waits for its LDS reads).  Then the step's MFMAs
  // run from registers, one per slot, and every other instruction of the
  // step is dealt out evenly over the slots so that the matrix core never
  // waits on a burst: the refill of stage kb with step kb + kRing, the LDS
  // reads of step kb + 1's operands, the unpacking of this step's second k
  // half (first half of the slots) and of step kb + 1's first k half
  // (second half of the slots), and in group mode the rescale of the
  // previous step's partial sums.  Past the last step the reads fetch
  // values that are never used.
  constexpr int kMfma = 4 * WM * WN;  // MFMAs per step
  constexpr int kHalf = kMfma / 2;
  constexpr int kUnits = 4 * WN;      // weight words per k half
  constexpr int kRescale = WM * WN * 16;
  static_assert(kRescale % kMfma == 0, "rescale work must split evenly over the MFMA slots");
  float sg_prev[GROUP ? WN : 1];
#pragma unroll
  for (int j = 0; j < (GROUP ? WN : 1); ++j) sg_prev[j] = 0.0f;
  auto step = [&](auto stage_c, int kb, const Ops& cur, Ops& nxt, v16i (&c)[WM][WN], v16i (&prev)[WM][WN]) {
    constexpr int S = decltype(stage_c)::value;
    wait_vmcnt<(kOwnRing - 2) * kPerStage>();
    lds_barrier();
    v4i lo1[WN], hi1[WN];
#pragma unroll
    for (int q = 0; q < kMfma; ++q) {
      // MFMA q: k half tp, nibble half h, block (i, j)
      const int tp = q / (2 * WM * WN), h = (q / (WM * WN)) % 2, i = (q / WN) % WM, j = q % WN;
      const v4i& bop = tp == 0 ? (h ? cur.hi0[j] : cur.lo0[j]) : (h ? hi1[j] : lo1[j]);
      // group mode: a step's first MFMA into a block starts from zero (an
      // inline constant), so the rescaled partial needs no clearing
      if (GROUP && tp == 0 && h == 0)
        c[i][j] = mfma32(cur.a[i][2 * tp + h], bop, v16i{});
      else
        c[i][j] = mfma32(cur.a[i][2 * tp + h], bop, c[i][j]);
#pragma unroll
      for (int d = 0; d < kPerStage; ++d)
        if (d * kMfma / kPerStage == q) issue_one(kb + kRing, S, d);
#pragma unroll
      for (int r = 0; r < kReads; ++r)
        if (r * kMfma / kReads == q) read_one(std::integral_constant<int, (S + 1) % kOwnRing>{}, r, nxt);
#pragma unroll
      for (int u = 0; u < kUnits; ++u) {
        if (q < kHalf && u * kHalf / kUnits == q) unpack_word(cur.b[u / 4][1], u % 4, lo1[u / 4], hi1[u / 4]);
        if (q >= kHalf && u * kHalf / kUnits == q - kHalf) unpack0(nxt, u);
      }
      if constexpr (GROUP) {
#pragma unroll
        for (int t = 0; t < kRescale / kMfma; ++t) {
          const int e = q * (kRescale / kMfma) + t;
          const int ri = e / (WN * 16), rj = (e / 16) % WN, rr = e % 16;
          facc[ri][rj][rr] = __fmaf_rn((float)prev[ri][rj][rr], sg_prev[rj], facc[ri][rj][rr]);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    if constexpr (GROUP)
#pragma unroll
      for (int j = 0; j < WN; ++j) sg_prev[j] = cur.sg[j];
  };

  // Group mode with at least 12 MFMAs per step: one accumulator set.  A
  // block's four MFMAs run back to back (block t in slots 4t .. 4t + 3, the
  // first from a zero operand), and its 16 partials are rescaled over the
  // kW slots from 4t + 5 on; those that fall past the step's last slot are
  // done early in the next step, before that step's first MFMA into the
  // block (slot 4t), with the scale of the step they belong to.  The next
  // step's weights are unpacked whole during this one (k half 0 from 3/16
  // of the slots on, k half 1 from 10/16, after their LDS reads land).
  constexpr int kW = kMfma >= 16 ? 8 : kMfma - 5;
  auto rescale_slot = [&](int q, bool wrapped, const v16i (&c)[WM][WN], const float (&sg)[GROUP ? WN : 1]) {
#pragma unroll
    for (int t = 0; t < WM * WN; ++t)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int slot = 4 * t + 5 + e * kW / 16;
        if ((!wrapped && slot == q) || (wrapped && slot - kMfma == q)) {
          const int i = t / WN, j = t % WN;
          facc[i][j][e] = __fmaf_rn((float)c[i][j][e], sg[j], facc[i][j][e]);
        }
      }
  };
  float sg_last[GROUP ? WN : 1];
#pragma unroll
  for (int j = 0; j < (GROUP ? WN : 1); ++j) sg_last[j] = 0.0f;
  auto step1 = [&](auto stage_c, int kb, const Ops& cur, Ops& nxt, v16i (&c)[WM][WN]) {
    constexpr int S = decltype(stage_c)::value;
    wait_vmcnt<(kOwnRing - 2) * kPerStage>();
    lds_barrier();
#pragma unroll
    for (int q = 0; q < kMfma; ++q) {
      const int t = q / 4, sub = q % 4, tp = sub / 2, h = sub % 2, i = t / WN, j = t % WN;
      rescale_slot(q, true, c, sg_last);  // before this step overwrites the block
      const v4i& bop = tp == 0 ? (h ? cur.hi0[j] : cur.lo0[j]) : (h ? cur.hi1[j] : cur.lo1[j]);
      if (sub == 0)
        c[i][j] = mfma32(cur.a[i][2 * tp + h], bop, v16i{});
      else
        c[i][j] = mfma32(cur.a[i][2 * tp + h], bop, c[i][j]);
#pragma unroll
      for (int d = 0; d < kPerStage; ++d)
        if (d * kMfma / kPerStage == q) issue_one(kb + kRing, S, d);
#pragma unroll
      for (int r = 0; r < kReads; ++r)
        if (r * kMfma / kReads == q) read_one(std::integral_constant<int, (S + 1) % kOwnRing>{}, r, nxt);
#pragma unroll
      for (int u = 0; u < kUnits; ++u) {
        if (q == kMfma * 3 / 16 + u * (kMfma * 6 / 16) / kUnits)
          unpack_word(nxt.b[u / 4][0], u % 4, nxt.lo0[u / 4], nxt.hi0[u / 4]);
        if (q == kMfma * 10 / 16 + u * (kMfma * 6 / 16) / kUnits)
          unpack_word(nxt.b[u / 4][1], u % 4, nxt.lo1[u / 4], nxt.hi1[u / 4]);
      }
      rescale_slot(q, false, c, cur.sg);
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int j = 0; j < (GROUP ? WN : 1); ++j) sg_last[j] = cur.sg[j];
  };

  const int NS = (KB + KS - 1) / KS;  // steps per k group (a trailing one past K reads zeros)
#pragma unroll
  for (int st = 0; st < kOwnRing; ++st)
#pragma unroll
    for (int d = 0; d < kPerStage; ++d) issue_one(KS * st + wk, st, d);
  Ops o0, o1;
  wait_vmcnt<(kOwnRing - 1) * kPerStage>();  // stage 0 (and the scales, issued before it)
  lds_barrier();
#pragma unroll
  for (int r = 0; r < kReads; ++r) read_one(std::integral_constant<int, 0>{}, r, o0);
#pragma unroll
  for (int u = 0; u < kUnits; ++u) unpack0(o0, u);
  if constexpr (GROUP && kMfma >= 12) {
#pragma unroll
    for (int u = 0; u < kUnits; ++u) unpack_word(o0.b[u / 4][1], u % 4, o0.lo1[u / 4], o0.hi1[u / 4]);
    for (int i = 0; i < NS; i += kOwnRing) {
      step1(std::integral_constant<int, 0>{}, KS * i + wk, o0, o1, acc[0]);
      if (i + 1 < NS) step1(std::integral_constant<int, 1>{}, KS * (i + 1) + wk, o1, o0, acc[0]);
      if (i + 2 < NS) step1(std::integral_constant<int, 2>{}, KS * (i + 2) + wk, o0, o1, acc[0]);
      if (i + 3 < NS) step1(std::integral_constant<int, 3>{}, KS * (i + 3) + wk, o1, o0, acc[0]);
    }
    // the last step's rescales that fall past its last slot
#pragma unroll
    for (int q = 0; q < kMfma; ++q) rescale_slot(q, true, acc[0], sg_last);
  } else {
    for (int i = 0; i < NS; i += kOwnRing) {
      step(std::integral_constant<int, 0>{}, KS * i + wk, o0, o1, acc[0], acc[GROUP ? 1 : 0]);
      if (i + 1 < NS) step(std::integral_constant<int, 1>{}, KS * (i + 1) + wk, o1, o0, acc[GROUP ? 1 : 0], acc[0]);
      if (i + 2 < NS) step(std::integral_constant<int, 2>{}, KS * (i + 2) + wk, o0, o1, acc[0], acc[GROUP ? 1 : 0]);
      if (i + 3 < NS) step(std::integral_constant<int, 3>{}, KS * (i + 3) + wk, o1, o0, acc[GROUP ? 1 : 0], acc[0]);
    }
  }
  if constexpr (GROUP && kMfma < 12) {
    // the last step's partial sums (the set of step KB - 1)
    auto rescale_last = [&](v16i (&last)[WM][WN]) {
#pragma unroll
      for (int i = 0; i < WM; ++i)
#pragma unroll
        for (int j = 0; j < WN; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) facc[i][j][r] = __fmaf_rn((float)last[i][j][r], sg_prev[j], facc[i][j][r]);
    };
    if (NS & 1)
      rescale_last(acc[0]);
    else
      rescale_last(acc[1]);
  }
  if constexpr (GROUP) load_sx();
  wait_vmcnt<0>();  // the stages issued past the end (and group mode's token scales)
  lds_barrier();    // every wave is done with the ring
  if constexpr (KS > 1) {
    // the k groups' sums (fp32 in group mode, int32 otherwise) meet in the
    // idle ring; group 0 keeps the total
    static_assert((KS - 1) * kWaves * WM * WN * 16 * 64 * 4 <= kRing * kStage, "merge must fit the ring");
    static_assert(!SW, "gated tiles take one k group");
    float* red = reinterpret_cast<float*>(lds);
    int* redi = reinterpret_cast<int*>(lds);
    auto slot = [&](int g, int i, int j, int r) { return ((((g * kWaves + wave) * WM + i) * WN + j) * 16 + r) * 64 + lane; };
    if (wk > 0)
#pragma unroll
      for (int i = 0; i < WM; ++i)
#pragma unroll
        for (int j = 0; j < WN; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            if constexpr (GROUP)
              red[slot(wk - 1, i, j, r)] = facc[i][j][r];
            else
              redi[slot(wk - 1, i, j, r)] = acc[0][i][j][r];
          }
    lds_barrier();
    if (wk == 0)
      for (int g = 1; g < KS; ++g)
#pragma unroll
        for (int i = 0; i < WM; ++i)
#pragma unroll
          for (int j = 0; j < WN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
              if constexpr (GROUP)
                facc[i][j][r] = __fadd_rn(facc[i][j][r], red[slot(g - 1, i, j, r)]);
              else
                acc[0][i][j][r] += redi[slot(g - 1, i, j, r)];
            }
    lds_barrier();
  }

  // ---- epilogue.  Lane holds column l32 and rows 8 q + 4 g2 + e (r = 4 q + e)
  // of each 32 x 32 block.  The scaled tile is staged in the idle LDS ring
  // and leaves as 16-byte row chunks, so every store writes whole cache
  // lines.  bf16 results are first paired across adjacent lanes (columns
  // 2 p and 2 p + 1; the even lane takes row r, the odd lane row r + 1) so
  // that every LDS write is a whole dword.
  auto result = [&](int i, int j, int r) -> float {
    const uint4 s4 = sx4[i][r >> 2];
    const float sx = __uint_as_float((r & 3) == 0 ? s4.x : (r & 3) == 1 ? s4.y : (r & 3) == 2 ? s4.z : s4.w);
    if constexpr (GROUP) {
      return __fmul_rn(facc[i][j][r], sx);
    } else {
      return __fmul_rn(__fmul_rn((float)(acc[0][i][j][r] >> 4), sx), swv[j]);
    }
  };
  // The output tile: OWN 32-column blocks per wave (gated: WN / 2, each the
  // activation of a gate block and its up block).
  constexpr int OWN = SW ? WN / 2 : WN;
  auto out_value = [&](int i, int j, int r) -> float {
    if constexpr (SW) {
      const float g = result(i, j, r), u = result(i, j + OWN, r);
      return __fmul_rn(__fdiv_rn(g, __fadd_rn(1.0f, __expf(-g))), u);
    } else {
      return result(i, j, r);
    }
  };
  const int ldy = SW ? a.F : N, oc0 = SW ? f0 : n0;  // output row stride, first output column
  auto store_tile = [&](auto es_tag) {
    constexpr int es = decltype(es_tag)::value;  // output element bytes
    // Row pitch: one half-wave's writes (bf16: rows R and R + 1 of 64 bytes;
    // 4-byte kinds: one 128-byte row) cover all 32 banks once.
    constexpr int kPitch = es == 2 ? OBN * 2 + 64 : OBN * 4 + 16;
    static_assert(BM * kPitch <= kRing * kStage, "output tile must fit the LDS ring");
    if constexpr (es == 2) {
      // NaN results become the canonical quiet NaN (sign and payload of a NaN
      // product vary), which the hardware conversion (round to nearest even,
      // bit-identical to f32_to_bf16 for every other input) turns into 0x7FC0.
      // A lane converts rows r and r + 1 of its column into one word, swaps
      // words with its neighbour and keeps the two halves of its row: the
      // even lane bytes {own 0-1, partner 0-1}, the odd lane {partner 2-3,
      // own 2-3}.
      const bool odd = lane & 1;
      const uint32_t sel = odd ? 0x03020706u : 0x05040100u;
      if (wk == 0)
#pragma unroll
      for (int i = 0; i < WM; ++i)
#pragma unroll
        for (int j = 0; j < OWN; ++j)
#pragma unroll
          for (int rp = 0; rp < 8; ++rp) {
            const uint32_t pair =
                bf16x2_bits(canonical_nan(out_value(i, j, 2 * rp)), canonical_nan(out_value(i, j, 2 * rp + 1)));
            const uint32_t recv = (uint32_t)__builtin_amdgcn_mov_dpp((int)pair, 0xB1, 0xF, 0xF, false);
            const uint32_t word = __builtin_amdgcn_perm(recv, pair, sel);
            const int r = 2 * rp + (odd ? 1 : 0);
            const int row = wm * 32 * WM + i * 32 + 8 * (r >> 2) + 4 * g2 + (r & 3);
            const int col = wn * 32 * OWN + j * 32 + (l32 & ~1);
            *reinterpret_cast<uint32_t*>(lds + row * kPitch + col * 2) = word;
          }
    } else {
      if (wk == 0)
#pragma unroll
      for (int i = 0; i < WM; ++i)
#pragma unroll
        for (int j = 0; j < OWN; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int row = wm * 32 * WM + i * 32 + 8 * (r >> 2) + 4 * g2 + (r & 3);
            const int col = wn * 32 * OWN + j * 32 + l32;
            uint32_t v;
            if constexpr (GROUP || SW)
              v = __float_as_uint(out_value(i, j, r));
            else
              v = a.out_kind == kOutI32 ? (uint32_t)(acc[0][i][j][r] >> 4) : __float_as_uint(result(i, j, r));
            *reinterpret_cast<uint32_t*>(lds + row * kPitch + col * 4) = v;
          }
    }
    lds_barrier();
    constexpr int kRowChunks = OBN * es / 16;
    constexpr int kChunks = BM * kRowChunks;
    static_assert(kChunks % (kThreads * KS) == 0, "output chunks must split evenly over the threads");
#pragma unroll
    for (int it = 0; it < kChunks / (kThreads * KS); ++it) {
      const int p = it * kThreads * KS + (int)threadIdx.x;
      const int row = p / kRowChunks, cc = p % kRowChunks;
      const uint4 v = *reinterpret_cast<const uint4*>(lds + row * kPitch + cc * 16);
      // N is a multiple of 16 and a chunk holds 4 or 8 columns, so a chunk
      // is either wholly inside the output or wholly past its last column
      if (row < rows_here && cc * (16 / es) < cols_here)
        *reinterpret_cast<uint4*>(static_cast<uint8_t*>(a.y) + ((size_t)(m0 + row) * ldy + oc0) * es + cc * 16) = v;
    }
  };
  if (a.out_kind == kOutBF16)
    store_tile(std::integral_constant<int, 2>{});
  else
    store_tile(std::integral_constant<int, 4>{});
}

// The instance of menu entry C (SW: the gated form).
template <int C, bool GROUP, bool SW = false>
constexpr LargeMKernelFn menu_kernel() {
  return largem<kMenu[C].WM, kMenu[C].WN, kMenu[C].GM, kMenu[C].GN, GROUP, kMenu[C].ring, SW, kMenu[C].ks>;
}

}  // namespace

}  // namespace w4a8
