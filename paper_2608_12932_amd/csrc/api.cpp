// C ABI of the W4A8 linear layer (declared in include/w4a8.h): argument
// validation, the choice of kernel path and tiling, workspace layout and
// launches.  Every check runs before anything is enqueued, so a rejected
// call has no effect and touches no HIP state.
#include "w4a8.h"

#include <cstdio>
#include <mutex>

#include "attention.h"
#include "kernels.h"

using namespace w4a8;

namespace {

constexpr int64_t kNMax = int64_t(1) << 24;
static_assert(W4A8_NOALLOC_SCRATCH_BYTES == kNoAllocScratchBytes, "header and library agree on the scratch size");

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }
size_t round_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

bool valid_nk(int64_t N, int64_t K) {
  return N >= 16 && N % 16 == 0 && N <= kNMax && K >= W4A8_GROUP_SIZE && K % W4A8_GROUP_SIZE == 0 &&
         K <= W4A8_K_MAX;
}

// Everything w4a8_linear decides from the shapes and modes alone.
struct Plan {
  bool small_m = false;
  bool separate_quant = false;  // bf16 input quantized by its own kernel first
  SmallMPlan sm{};
  LargeMPlan lm{};
  // workspace layout (bytes)
  size_t off_counters = 0, off_partial = 0, off_xq = 0, off_sx = 0, total = 0;
  bool counters_fit = true;  // the split's counters fit the counter region
  bool grid_fits = true;     // the large-M tile count fits one launch
};

Plan make_plan(int64_t M, int64_t N, int64_t K, bool group, bool bf16_in, bool swiglu = false) {
  Plan p;
  p.small_m = M <= kSmallMMaxM;
  if (p.small_m) {
    p.sm = plan_smallm((int)M, (int)N, (int)K, group, bf16_in, swiglu);
    p.separate_quant = bf16_in && !p.sm.fused;
  } else {
    p.lm = plan_largem((int)M, (int)N, (int)K, group, swiglu);
    p.separate_quant = bf16_in;
    p.grid_fits = p.lm.tiles >= 1 && p.lm.tiles <= kMaxGrid;
  }
  // counters at offset 0 of the shared counter region, the rest beyond it
  const bool split = p.small_m && p.sm.S > 1;
  p.counters_fit = !split || p.sm.groups <= kMaxCounters;
  size_t off = split || p.separate_quant ? kCounterRegionBytes : 0;
  if (split) {
    p.off_counters = 0;
    p.off_partial = off;
    off = round_up(off + (size_t)p.sm.S * M * N * 4, 256);
  }
  if (p.separate_quant) {
    p.off_xq = off;
    off = round_up(off + (size_t)M * K, 256);
    p.off_sx = off;
    off = round_up(off + (size_t)M * sizeof(float), 256);
  }
  p.total = off;
  return p;
}

std::mutex g_pack_mutex;

bool valid_modes(int scale_mode, int in_kind) {
  return (scale_mode == W4A8_SCALE_CHANNEL_F32 || scale_mode == W4A8_SCALE_GROUP_F16) &&
         (in_kind == W4A8_IN_BF16 || in_kind == W4A8_IN_I8);
}

// Shapes the gated entry points take: an even number of 16-column tiles
// (gate and up halves of whole tiles).
bool gated_shape(int64_t N) { return N % 32 == 0; }

// Both linear entry points after their own checks: the rest of the
// validation, the plan, and the launches.
// noalloc: the workspace is this device's library-owned scratch array
// (workspace and workspace_bytes are ignored); its split-K counters are
// cleared by a kernel before use.
w4a8_status run_linear(const void* x, int in_kind, const float* x_scale, int64_t M, int64_t K,
                       const uint8_t* w_packed, const void* w_scale, int scale_mode, int64_t N, void* y,
                       int out_kind, void* workspace, size_t workspace_bytes, hipStream_t stream,
                       bool swiglu, bool noalloc = false) {
  if (M < 0 || M > W4A8_M_MAX || !valid_nk(N, K)) return W4A8_EINVAL;
  if (!valid_modes(scale_mode, in_kind)) return W4A8_EINVAL;
  if (out_kind != W4A8_OUT_BF16 && out_kind != W4A8_OUT_F32 && out_kind != W4A8_OUT_I32_ACC)
    return W4A8_EINVAL;
  if (swiglu && (out_kind == W4A8_OUT_I32_ACC || N % 32)) return W4A8_EINVAL;
  if (M == 0) return W4A8_OK;
  // 32-bit buffer offsets: the group-scale array (N*K/64 bytes) stays below 2 GiB
  if ((uint64_t)N * (uint64_t)K >= (uint64_t(1) << 37)) return W4A8_EUNSUPPORTED;
  if (!x || !aligned(x, 16) || !w_packed || !aligned(w_packed, 16) || !y || !aligned(y, 16))
    return W4A8_EINVAL;
  if (in_kind == W4A8_IN_I8 && (!x_scale || !aligned(x_scale, 4))) return W4A8_EINVAL;
  if (out_kind != W4A8_OUT_I32_ACC &&
      (!w_scale || !aligned(w_scale, scale_mode == W4A8_SCALE_CHANNEL_F32 ? 4 : 2)))
    return W4A8_EINVAL;

  // The integer accumulator does not depend on the scales, so the raw
  // accumulator output always takes the per-channel kernels.
  const bool group = scale_mode == W4A8_SCALE_GROUP_F16 && out_kind != W4A8_OUT_I32_ACC;
  const bool bf16_in = in_kind == W4A8_IN_BF16;
  const Plan p = make_plan(M, N, K, group, bf16_in, swiglu);
  if (!p.counters_fit || !p.grid_fits) return W4A8_EUNSUPPORTED;
  if (noalloc) {
    if (p.total > kNoAllocScratchBytes) return W4A8_EUNSUPPORTED;
    workspace = nullptr;
    if (p.total) {
      if (noalloc_scratch(&workspace) != hipSuccess) return W4A8_EHIP;
      if (p.small_m && p.sm.S > 1 &&
          launch_clear_words(static_cast<unsigned*>(workspace), p.sm.groups, stream) != hipSuccess)
        return W4A8_EHIP;
    }
  } else {
    if (workspace_bytes < p.total) return W4A8_EINVAL;
    if (p.total && (!workspace || !aligned(workspace, 256))) return W4A8_EINVAL;
  }

  uint8_t* ws = static_cast<uint8_t*>(workspace);
  const void* xin = x;
  const float* sx = x_scale;
  if (p.separate_quant) {
    int8_t* xq = reinterpret_cast<int8_t*>(ws + p.off_xq);
    float* s = reinterpret_cast<float*>(ws + p.off_sx);
    if (launch_quantize(static_cast<const uint16_t*>(x), (int)M, (int)K, xq, s, stream) != hipSuccess)
      return W4A8_EHIP;
    xin = xq;
    sx = s;
  }

  hipError_t e;
  if (p.small_m) {
    SmallMArgs a{};
    a.x = xin;
    a.x_scale = sx;
    a.wp = w_packed;
    a.w_scale = w_scale;
    a.y = y;
    a.partial = p.sm.S > 1 ? ws + p.off_partial : nullptr;
    a.counters = p.sm.S > 1 ? reinterpret_cast<unsigned*>(ws + p.off_counters) : nullptr;
    a.M = (int)M;
    a.N = (int)N;
    a.K = (int)K;
    a.KB = (int)(K / W4A8_GROUP_SIZE);
    a.S = p.sm.S;
    a.kbs = (a.KB + p.sm.S - 1) / p.sm.S;
    a.tpr = p.sm.tpr;
    a.out_kind = out_kind;
    a.F = swiglu ? (int)(N / 2) : 0;
    e = launch_smallm(p.sm, a, stream);
  } else {
    LargeMArgs a{};
    a.xq = static_cast<const int8_t*>(xin);
    a.x_scale = sx;
    a.wp = w_packed;
    a.w_scale = w_scale;
    a.y = y;
    a.M = (int)M;
    a.N = (int)N;
    a.K = (int)K;
    a.KB = (int)(K / W4A8_GROUP_SIZE);
    a.out_kind = out_kind;
    a.tiles_m = p.lm.tiles_m;
    a.tiles_n = p.lm.tiles_n;
    a.xcd_remap = p.lm.tiles % 8 == 0;
    a.F = swiglu ? (int)(N / 2) : 0;
    e = launch_largem(p.lm, a, stream);
  }
  return e == hipSuccess ? W4A8_OK : W4A8_EHIP;
}

size_t workspace_bytes(int64_t M, int64_t N, int64_t K, int scale_mode, int in_kind, bool swiglu) {
  if (M < 0 || M > W4A8_M_MAX || !valid_nk(N, K) || !valid_modes(scale_mode, in_kind)) return 0;
  if (M == 0 || (uint64_t)N * (uint64_t)K >= (uint64_t(1) << 37)) return 0;
  if (swiglu && !gated_shape(N)) return 0;
  const Plan p = make_plan(M, N, K, scale_mode == W4A8_SCALE_GROUP_F16, in_kind == W4A8_IN_BF16, swiglu);
  return p.counters_fit && p.grid_fits ? p.total : 0;
}

const char* describe(int64_t M, int64_t N, int64_t K, int scale_mode, int in_kind, int out_kind, bool swiglu) {
  static thread_local char buf[256];
  if (M <= 0 || M > W4A8_M_MAX || !valid_nk(N, K)) return "invalid shape";
  if (swiglu && !gated_shape(N)) return "invalid shape";
  const bool group = scale_mode == W4A8_SCALE_GROUP_F16 && out_kind != W4A8_OUT_I32_ACC;
  const Plan p = make_plan(M, N, K, group, in_kind == W4A8_IN_BF16, swiglu);
  if (!p.counters_fit || !p.grid_fits) return "unsupported shape";
  snprintf(buf, sizeof buf, "%s%s workspace=%zu", p.separate_quant ? "quantize_rows + " : "",
           p.small_m ? smallm_kernel_name(p.sm) : largem_kernel_name(p.lm), p.total);
  return buf;
}

}  // namespace

extern "C" {

const char* w4a8_status_string(w4a8_status s) {
  switch (s) {
    case W4A8_OK: return "ok";
    case W4A8_EINVAL: return "invalid argument";
    case W4A8_EUNSUPPORTED: return "unsupported shape";
    case W4A8_ERANGE: return "weight value outside [-8, 7]";
    case W4A8_EHIP: return "HIP runtime error";
  }
  return "unknown status";
}

size_t w4a8_packed_weight_bytes(int64_t N, int64_t K) {
  if (!valid_nk(N, K)) return 0;
  return (size_t)N * (size_t)K / 2;
}

w4a8_status w4a8_pack_weights(const int8_t* w, int64_t N, int64_t K, uint8_t* w_packed,
                              hipStream_t stream) {
  if (!valid_nk(N, K)) return W4A8_EINVAL;
  if (!w || !w_packed || !aligned(w, 16) || !aligned(w_packed, 16)) return W4A8_EINVAL;
  std::lock_guard<std::mutex> lk(g_pack_mutex);
  unsigned* err = nullptr;
  if (pack_error_word(&err) != hipSuccess) return W4A8_EHIP;
  if (launch_pack(w, (int)N, (int)K, w_packed, err, stream) != hipSuccess) return W4A8_EHIP;
  unsigned flag = 0;
  if (hipMemcpyAsync(&flag, err, sizeof flag, hipMemcpyDeviceToHost, stream) != hipSuccess) return W4A8_EHIP;
  if (hipStreamSynchronize(stream) != hipSuccess) return W4A8_EHIP;
  return flag ? W4A8_ERANGE : W4A8_OK;
}

w4a8_status w4a8_quantize_act(const uint16_t* x, int64_t M, int64_t K, int8_t* x_q, float* x_scale,
                              hipStream_t stream) {
  if (M < 0 || M > W4A8_M_MAX) return W4A8_EINVAL;
  if (K < W4A8_GROUP_SIZE || K % W4A8_GROUP_SIZE || K > W4A8_K_MAX) return W4A8_EINVAL;
  if (M == 0) return W4A8_OK;
  if (!x || !x_q || !x_scale || !aligned(x, 16) || !aligned(x_q, 16) || !aligned(x_scale, 4))
    return W4A8_EINVAL;
  return launch_quantize(x, (int)M, (int)K, x_q, x_scale, stream) == hipSuccess ? W4A8_OK : W4A8_EHIP;
}

w4a8_status w4a8_rmsnorm_quantize_act(const uint16_t* x, const uint16_t* gamma, float eps, int64_t M, int64_t K,
                                      int8_t* x_q, float* x_scale, hipStream_t stream) {
  if (M < 0 || M > W4A8_M_MAX) return W4A8_EINVAL;
  if (K < W4A8_GROUP_SIZE || K % W4A8_GROUP_SIZE || K > W4A8_K_MAX) return W4A8_EINVAL;
  if (!(eps > 0.0f) || !(eps <= 3.4e38f)) return W4A8_EINVAL;  // also rejects NaN and inf
  if (M == 0) return W4A8_OK;
  if (!x || !gamma || !x_q || !x_scale || !aligned(x, 16) || !aligned(gamma, 16) || !aligned(x_q, 16) ||
      !aligned(x_scale, 4))
    return W4A8_EINVAL;
  return launch_rmsnorm_quantize(x, gamma, eps, (int)M, (int)K, x_q, x_scale, stream) == hipSuccess ? W4A8_OK
                                                                                                  : W4A8_EHIP;
}

w4a8_status w4a8_flow_schedule(int64_t n_steps, int64_t n_reuse, int32_t* fresh) {
  if (n_steps < 1 || n_steps > 4096 || n_reuse < 0 || n_reuse >= n_steps || !fresh) return W4A8_EINVAL;
  const int64_t head = (n_steps - n_reuse + 1) / 2;
  for (int64_t i = 0; i < n_steps; ++i) fresh[i] = (i < head || i >= head + n_reuse) ? 1 : 0;
  return W4A8_OK;
}

w4a8_status w4a8_flow_step(float* x, const uint16_t* v_new, uint16_t* v_cache, int64_t B, int64_t n, float dt,
                           int64_t repeat, double* stats, hipStream_t stream) {
  if (B < 0 || B > (int64_t(1) << 24) || n < 1 || n > (int64_t(1) << 26)) return W4A8_EINVAL;
  if (repeat < 1 || repeat > 4096) return W4A8_EINVAL;
  if (!(dt == dt) || dt > 3.4e38f || dt < -3.4e38f) return W4A8_EINVAL;  // finite
  if (!v_new && stats) return W4A8_EINVAL;
  if (B == 0) return W4A8_OK;
  if (!x || !v_cache || !aligned(x, 16) || !aligned(v_cache, 16) || (v_new && !aligned(v_new, 16)) ||
      (stats && !aligned(stats, 8)))
    return W4A8_EINVAL;
  const uintptr_t xs = reinterpret_cast<uintptr_t>(x), cs = reinterpret_cast<uintptr_t>(v_cache);
  const uintptr_t xb = uintptr_t(B * n * 4), hb = uintptr_t(B * n * 2);
  auto overlap = [](uintptr_t a, uintptr_t na, uintptr_t b, uintptr_t nb) { return a < b + nb && b < a + na; };
  if (overlap(xs, xb, cs, hb)) return W4A8_EINVAL;
  if (v_new) {
    const uintptr_t vs = reinterpret_cast<uintptr_t>(v_new);
    if (overlap(xs, xb, vs, hb) || (vs != cs && overlap(vs, hb, cs, hb))) return W4A8_EINVAL;
    if (stats) {
      const uintptr_t ss = reinterpret_cast<uintptr_t>(stats), sb = uintptr_t(B * 32);
      if (overlap(ss, sb, xs, xb) || overlap(ss, sb, vs, hb) || overlap(ss, sb, cs, hb)) return W4A8_EINVAL;
    }
  }
  return launch_flow_step(x, v_new, v_cache, (int)B, (int)n, dt, (int)repeat, stats, stream) == hipSuccess
             ? W4A8_OK
             : W4A8_EHIP;
}

size_t w4a8_stream_attention_workspace_bytes(int64_t H, int64_t Nq, int64_t Nk) {
  constexpr int64_t kMax = int64_t(1) << 22;
  if (H < 1 || H > 4096 || Nq < 1 || Nq > kMax || Nk < 1 || Nk > kMax) return 0;
  return stream_attention_workspace((int)H, (int)Nq, (int)Nk);
}

w4a8_status w4a8_stream_attention(const uint16_t* q, const uint16_t* k, const uint16_t* v, const int32_t* pos_q,
                                  const int32_t* pos_k, const float* rope_cos, const float* rope_sin, int64_t n_pos,
                                  int64_t H, int64_t Hkv, int64_t Nq, int64_t Nk, int64_t D, float scale, uint16_t* o,
                                  void* workspace, size_t workspace_bytes, hipStream_t stream) {
  constexpr int64_t kMax = int64_t(1) << 22;  // 32-bit buffer offsets over a head's [N][128] rows
  if (D != 128) return W4A8_EUNSUPPORTED;
  if (H < 1 || Hkv < 1 || H % Hkv || H > 4096 || Nq < 0 || Nq > kMax || Nk < 1 || Nk > kMax || n_pos < 1 ||
      n_pos > kMax)
    return W4A8_EINVAL;
  if (!(scale == scale) || scale > 3.4e38f || scale < -3.4e38f) return W4A8_EINVAL;  // finite
  if (Nq == 0) return W4A8_OK;
  if (!q || !k || !v || !pos_q || !pos_k || !rope_cos || !rope_sin || !o || !aligned(q, 16) || !aligned(k, 16) ||
      !aligned(v, 16) || !aligned(o, 16) || !aligned(pos_q, 4) || !aligned(pos_k, 4) || !aligned(rope_cos, 16) ||
      !aligned(rope_sin, 16))
    return W4A8_EINVAL;
  const size_t need = stream_attention_workspace((int)H, (int)Nq, (int)Nk);
  if (workspace_bytes < need || !workspace || !aligned(workspace, 256)) return W4A8_EINVAL;
  AttnArgs a{};
  a.workspace = workspace;
  a.q = q;
  a.k = k;
  a.v = v;
  a.pos_q = pos_q;
  a.pos_k = pos_k;
  a.rope_cos = rope_cos;
  a.rope_sin = rope_sin;
  a.o = o;
  a.H = (int)H;
  a.Hkv = (int)Hkv;
  a.Nq = (int)Nq;
  a.Nk = (int)Nk;
  a.n_pos = (int)n_pos;
  a.scale_log2e = scale * 1.4426950408889634f;
  return launch_stream_attention(a, stream) == hipSuccess ? W4A8_OK : W4A8_EHIP;
}

size_t w4a8_linear_workspace_bytes(int64_t M, int64_t N, int64_t K, int scale_mode, int in_kind) {
  return workspace_bytes(M, N, K, scale_mode, in_kind, false);
}

const char* w4a8_linear_describe(int64_t M, int64_t N, int64_t K, int scale_mode, int in_kind,
                                 int out_kind) {
  return describe(M, N, K, scale_mode, in_kind, out_kind, false);
}

w4a8_status w4a8_linear(const void* x, int in_kind, const float* x_scale, int64_t M, int64_t K,
                        const uint8_t* w_packed, const void* w_scale, int scale_mode, int64_t N,
                        void* y, int out_kind, void* workspace, size_t workspace_bytes,
                        hipStream_t stream) {
  return run_linear(x, in_kind, x_scale, M, K, w_packed, w_scale, scale_mode, N, y, out_kind, workspace,
                    workspace_bytes, stream, false);
}

w4a8_status w4a8_linear_noalloc(const void* x, int in_kind, const float* x_scale, int64_t M, int64_t K,
                                const uint8_t* w_packed, const void* w_scale, int scale_mode, int64_t N,
                                void* y, int out_kind, hipStream_t stream) {
  return run_linear(x, in_kind, x_scale, M, K, w_packed, w_scale, scale_mode, N, y, out_kind, nullptr, 0,
                    stream, false, true);
}

size_t w4a8_linear_swiglu_workspace_bytes(int64_t M, int64_t N, int64_t K, int scale_mode, int in_kind) {
  return workspace_bytes(M, N, K, scale_mode, in_kind, true);
}

const char* w4a8_linear_swiglu_describe(int64_t M, int64_t N, int64_t K, int scale_mode, int in_kind) {
  return describe(M, N, K, scale_mode, in_kind, W4A8_OUT_BF16, true);
}

w4a8_status w4a8_linear_swiglu(const void* x, int in_kind, const float* x_scale, int64_t M, int64_t K,
                               const uint8_t* w_packed, const void* w_scale, int scale_mode, int64_t N,
                               void* y, int out_kind, void* workspace, size_t workspace_bytes,
                               hipStream_t stream) {
  return run_linear(x, in_kind, x_scale, M, K, w_packed, w_scale, scale_mode, N, y, out_kind, workspace,
                    workspace_bytes, stream, true);
}

}  // extern "C"
