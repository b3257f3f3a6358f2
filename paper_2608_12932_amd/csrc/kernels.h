// Internal launch interface between the C ABI (api.cpp) and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace w4a8 {

enum OutKind { kOutBF16 = 0, kOutF32 = 1, kOutI32 = 2 };

// Every workspace starts with this region of arrival counters, at the same
// offsets for every call shape, and everything else a call keeps there
// (partial sums, codes) lies beyond it: counters return to zero at the end
// of each call, so one zero-filled workspace serves calls of any shape.
constexpr size_t kCounterRegionBytes = 64 * 1024;
constexpr int kMaxCounters = (int)(kCounterRegionBytes / sizeof(unsigned));

// ---- activation quantize (quantize.hip)
hipError_t launch_quantize(const uint16_t* x, int M, int K, int8_t* q, float* scale,
                           hipStream_t stream);
// RMSNorm (gain gamma, eps > 0) of each row, then the quantize of the fp32 result
hipError_t launch_rmsnorm_quantize(const uint16_t* x, const uint16_t* gamma, float eps, int M, int K, int8_t* q,
                                   float* scale, hipStream_t stream);

// ---- weight pack (pack.hip); `err` is a device word set to 1 on a range error
hipError_t launch_pack(const int8_t* w, int N, int K, uint8_t* out, unsigned* err,
                       hipStream_t stream);
hipError_t pack_error_word(unsigned** err);  // per-device status word

// ---- small-M GEMM (gemm_smallm.hip)
struct SmallMArgs {
  const void* x;         // bf16 [M][K] (fused quantize) or int8 codes [M][K]
  const float* x_scale;  // [M] (int8 input)
  const uint8_t* wp;     // packed weights
  const void* w_scale;   // fp32 [N] or fp16 [K/128][N]
  void* y;               // [M][N]
  void* partial;         // [S][M][N] int32 or fp32 (S > 1)
  unsigned* counters;    // [groups] arrival counters (S > 1)
  int M, N, K, KB;
  int S, kbs;            // K splits and 128-k blocks per split
  int tpr;               // fused quantize: threads per token row
  int out_kind;
  int F;                 // gated output: gate width (N / 2); y is [M][F]
};
struct SmallMPlan {
  int MT, NT;            // 16-row tiles, 16-column tiles per workgroup
  int S;                 // K splits over workgroups
  bool fused;            // quantize inside the GEMM
  int qmode;             // 0 int8 codes in, 1 quantize fused, codes made in LDS
  bool group;            // group-wise scales
  int groups;            // workgroups along N
  int tpr;               // fused quantize: threads per token row
  bool exact;            // every wave's block count is a multiple of the stage depth
  bool swiglu;           // gated output silu(gate) * up (gate columns [0, N/2), up [N/2, N))
  size_t lds_bytes;
  double model_us;       // the cost model's time for the GEMM launch (int8 codes in)
};
SmallMPlan plan_smallm(int M, int N, int K, bool group, bool bf16_in, bool swiglu);
hipError_t launch_smallm(const SmallMPlan& p, const SmallMArgs& a, hipStream_t stream);
constexpr int kSmallMWaves = 8;
constexpr int kSmallMMaxM = 64;

// ---- large-M GEMM (gemm_largem.hip)
struct LargeMArgs {
  const int8_t* xq;
  const float* x_scale;
  const uint8_t* wp;
  const void* w_scale;
  void* y;
  int M, N, K, KB;
  int out_kind;
  int tiles_m, tiles_n;
  int xcd_remap;
  int F;                 // gated output: gate width (N / 2); y is [M][F]
};
struct LargeMPlan {
  int cfg;               // index into the tile menu
  int BM, BN, threads;
  bool group;
  bool swiglu;           // gated output (the 128 x 128 tile; a tile covers BN / 2 output columns)
  int tiles_m, tiles_n;
  int64_t tiles;         // tiles_m * tiles_n, the grid size
  size_t lds_bytes;
};
// Largest grid a launch takes (one workgroup per tile).
constexpr int64_t kMaxGrid = 0x7FFFFFFF;
LargeMPlan plan_largem(int M, int N, int K, bool group, bool swiglu);
hipError_t launch_largem(const LargeMPlan& p, const LargeMArgs& a, hipStream_t stream);
typedef void (*LargeMKernelFn)(const LargeMArgs);
// group-scale instance of tile-menu entry cfg (gemm_largem_group.hip), or
// nullptr where the tile does not fit the group accumulators (or, gated,
// for any tile but the gated one)
LargeMKernelFn largem_group_kernel(int cfg, bool swiglu);

// ---- flow-matching Euler step with the velocity cache (flow.hip)
// v == nullptr: a reused step (x += dt * cache); otherwise cache = v after
// x += dt * v, and, with stats, stats[b] = (sum v c, sum v v, sum c c,
// sum (v - c)^2) against the cache before the step; the update is applied
// `repeat` times (consecutive steps with the same velocity).  One workgroup
// per row.
hipError_t launch_flow_step(float* x, const uint16_t* v, uint16_t* cache, int B, int n, float dt, int repeat,
                            double* stats, hipStream_t stream);

// ---- library-owned scratch of w4a8_linear_noalloc (noalloc.hip)
// Size of the per-device scratch array; the caller-workspace layout of
// w4a8_linear (counter region first) is laid over it.
constexpr size_t kNoAllocScratchBytes = size_t(32) << 20;
// Device address of this device's scratch array (looked up once per device).
hipError_t noalloc_scratch(void** ptr);
// Zero words [0, n) of p with a kernel on `stream`.
hipError_t launch_clear_words(unsigned* p, int n, hipStream_t stream);

const char* smallm_kernel_name(const SmallMPlan& p);
const char* largem_kernel_name(const LargeMPlan& p);

}  // namespace w4a8
