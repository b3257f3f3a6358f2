// Large-M W4A8 GEMM: tile planning, the per-channel kernel instances and the
// launch.  The kernel template is in largem_kernel.h; the group-scale
// instances are built in gemm_largem_group.hip.
#include <cstdio>

#include "largem_kernel.h"

namespace w4a8 {

namespace {

LargeMKernelFn channel_kernel(int cfg, bool swiglu) {
  if (swiglu) {
    switch (cfg) {
      case 1: return menu_kernel<1, false, true>();
      case 3: return menu_kernel<3, false, true>();
      default: return nullptr;
    }
  }
  switch (cfg) {
    case 0: return menu_kernel<0, false>();
    case 1: return menu_kernel<1, false>();
    case 2: return menu_kernel<2, false>();
    case kMenuKSplit: return menu_kernel<kMenuKSplit, false>();
    default: return nullptr;
  }
}

}  // namespace

// Gated plans (swiglu) take the tiles whose waves hold an even number of
// blocks (gate and up halves): a tile covers BN / 2 output columns.
LargeMPlan plan_largem(int M, int N, int K, bool group, bool swiglu) {
  (void)K;
  LargeMPlan p{};
  p.group = group;
  p.swiglu = swiglu;
  double best = -1.0;
  for (int c = 0; c < kMenuSize; ++c) {
    const TileCfg& t = kMenu[c];
    if (group && !t.group_ok) continue;
    if (t.ks > 1) continue;  // the k-split form replaces entry 2 below
    if (swiglu ? !t.gated_ok : !t.plain_ok) continue;
    const int BM = 32 * t.WM * t.GM, BN = 32 * t.WN * t.GN;
    const int tm = (M + BM - 1) / BM, tn = swiglu ? (N / 2 + BN / 2 - 1) / (BN / 2) : (N + BN - 1) / BN;
    const int64_t tiles = (int64_t)tm * tn;
    const int64_t rounds = (tiles + 255) / 256;
    const double eff = (double)M * N / ((double)rounds * 256.0 * BM * BN);
    const double score = eff * t.quality;
    if (score > best + 1e-9) {
      best = score;
      p.cfg = c;
      p.BM = BM;
      p.BN = BN;
      p.threads = 64 * t.GM * t.GN * t.ks;
      p.tiles_m = tm;
      p.tiles_n = tn;
      p.tiles = tiles;
    }
  }
  // 64 x 64 tiles that fill at most one round: two k groups per tile
  // (measured at M = 256, group scales: o 12.4 -> 10.8 us, down 31.8 -> 24.4
  // us; channel scales: down 24.0 -> 21.7 us, o unchanged; with more tiles,
  // one 8-wave workgroup per CU loses to three 4-wave ones)
  if (!swiglu && p.cfg == 2 && p.tiles <= 256) {
    p.cfg = kMenuKSplit;
    p.threads = 64 * kMenu[p.cfg].GM * kMenu[p.cfg].GN * kMenu[p.cfg].ks;
  }
  const TileCfg& c = kMenu[p.cfg];
  p.lds_bytes = (size_t)c.ring * ((size_t)p.BM * 128 + (size_t)p.BN / 16 * kBlockBytes +
                                  (group ? (size_t)(c.GM * c.GN) * 256 : 0));
  return p;
}

hipError_t launch_largem(const LargeMPlan& p, const LargeMArgs& a, hipStream_t stream) {
  LargeMKernelFn k = p.group ? largem_group_kernel(p.cfg, p.swiglu) : channel_kernel(p.cfg, p.swiglu);
  if (!k || p.tiles < 1 || p.tiles > kMaxGrid) return hipErrorInvalidValue;
  const unsigned grid = (unsigned)p.tiles;
  hipLaunchKernelGGL(k, dim3(grid), dim3(p.threads), p.lds_bytes, stream, a);
  return hipGetLastError();
}

const char* largem_kernel_name(const LargeMPlan& p) {
  static thread_local char buf[96];
  snprintf(buf, sizeof buf, "largem<%dx%d,%s%s%s> tiles=%dx%d", p.BM, p.BN, p.group ? "group" : "channel",
           p.swiglu ? ",swiglu" : "", kMenu[p.cfg].ks > 1 ? ",ksplit" : "", p.tiles_m, p.tiles_n);
  return buf;
}

}  // namespace w4a8
