/*
 * w4a8.h - C ABI of the MI355X (gfx950) W4A8 linear layer
 *
 *     y = dequant( quant8(x) . int4(W)^T )
 *
 * FlashDrive, Sec. 3.4 ("Quantization"): the backbone weights are held as
 * 4-bit integers, the activations entering each backbone linear layer are
 * cast to 8 bits, and the product runs on the integer matrix units; Sec. 4.2
 * ("Algorithm-level gains", on Table 1) attributes the decode gain to the 4x
 * smaller weight stream and the prefill gain to the INT8 contraction.  Sec.
 * 3.5 ("Kernel Fusion") fuses Q/K/V into one projection and gate/up into
 * another, which is why N can be 6144 or 24576 here.  The paper fixes no
 * scale granularity or rounding; this library implements:
 *   - per-token symmetric activation scale s_x[m] = max_k |x[m,k]| / 127 (fp32),
 *     codes q[m,k] = round_half_even(x[m,k] / s_x[m]) in [-127, 127];
 *     an all-zero token has s_x = 0 and q = 0;
 *   - weight integers W[n,k] in [-8, 7] with either one fp32 scale per output
 *     channel n, or one fp16 scale per 128 consecutive k per channel;
 *   - an exact int32 contraction acc[m,n] = sum_k q[m,k] W[n,k];
 *   - dequantization per channel: y = ((float)acc * s_x[m]) * s_w[n], two
 *     fp32 multiplies in that order; per group: y = s_x[m] * sum_g
 *     (float)p_g[m,n] * s_g[g][n] accumulated in fp32 (order unspecified);
 *     bf16 outputs are rounded to nearest even.
 *
 * Conventions for every call:
 *   - Matrices are dense and row-major (last index contiguous): x [M][K],
 *     W [N][K] (the nn.Linear weight layout, so y = x W^T), y [M][N].
 *   - Pointers named "device" are HIP device pointers; the caller allocates
 *     and owns every buffer; the library never allocates device memory on
 *     these calls and keeps no pointer after a call returns.
 *   - Work is enqueued on `stream` (0 = the null stream) and is asynchronous
 *     unless the call says otherwise; calls on different streams do not share
 *     state, except that concurrent w4a8_linear calls must not share one
 *     workspace.
 *   - Arguments are validated before anything is launched; an invalid call
 *     returns an error code and has no effect.  No call prints or aborts.
 *   - A HIP launch failure is reported as W4A8_EHIP.
 *
 * Shape of the interface, where it could have been drawn otherwise:
 *   - the group size is not an argument: W4A8_SCALE_GROUP_F16 fixes it at
 *     W4A8_GROUP_SIZE (128), the one group size the method uses here;
 *   - the workspace size queries take the input kind, because only a bf16
 *     input quantized by a separate kernel keeps codes in the workspace;
 *   - N need only be a multiple of 16, the output channels of one packed
 *     weight block, and K a multiple of 128, the k of one block.
 */
#ifndef W4A8_H_
#define W4A8_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  W4A8_OK = 0,
  W4A8_EINVAL = 1,       /* null/misaligned pointer, bad size, mode, or workspace too small */
  W4A8_EUNSUPPORTED = 2, /* well-formed but outside the supported shape range */
  W4A8_ERANGE = 3,       /* a weight value outside [-8, 7] */
  W4A8_EHIP = 4          /* the HIP runtime reported an error */
} w4a8_status;

/* weight scale granularity */
typedef enum {
  W4A8_SCALE_CHANNEL_F32 = 0, /* w_scale: fp32 [N] */
  W4A8_SCALE_GROUP_F16 = 1    /* w_scale: fp16 [K/128][N], group of 128 along k */
} w4a8_scale_mode;

/* activation input of w4a8_linear */
typedef enum {
  W4A8_IN_BF16 = 0, /* x: bf16 [M][K]; quantized inside the call */
  W4A8_IN_I8 = 1    /* x: int8 codes [M][K] with x_scale fp32 [M] (w4a8_quantize_act output) */
} w4a8_in_kind;

/* output of w4a8_linear */
typedef enum {
  W4A8_OUT_BF16 = 0,   /* y: bf16 [M][N] */
  W4A8_OUT_F32 = 1,    /* y: fp32 [M][N], the value before bf16 rounding */
  W4A8_OUT_I32_ACC = 2 /* y: int32 [M][N], the raw accumulator sum_k q W (scales unused) */
} w4a8_out_kind;

#define W4A8_GROUP_SIZE 128
#define W4A8_K_MAX 65536     /* 16 * 127 * 8 * K stays below 2^31 */
#define W4A8_M_MAX 1048576

/* Human-readable name of a status code (static string, never NULL). */
const char* w4a8_status_string(w4a8_status s);

/*
 * Size in bytes of the packed weight buffer for an N x K weight: N*K/2
 * (two 4-bit values per byte, the 4x reduction of Sec. 3.4's memory saving
 * against 16-bit weights).  Returns 0 if N or K is not a valid shape
 * (N % 16 != 0, K % 128 != 0, or out of range).
 */
size_t w4a8_packed_weight_bytes(int64_t N, int64_t K);

/*
 * Pack int4-range weights for w4a8_linear (one-time, off the hot path).
 *   w         device, int8 [N][K], every value in [-8, 7]
 *   N, K      N % 16 == 0, K % 128 == 0, 1 <= K <= W4A8_K_MAX
 *   w_packed  device, w4a8_packed_weight_bytes(N, K) bytes, 16-byte aligned;
 *             the layout is opaque (ordered for the matrix-core operand
 *             fragments) and only w4a8_linear reads it
 * Synchronizes `stream`.  Returns W4A8_ERANGE (w_packed then holds garbage)
 * if any value lies outside [-8, 7].  Calls from several host threads are
 * serialized internally.
 */
w4a8_status w4a8_pack_weights(const int8_t* w, int64_t N, int64_t K, uint8_t* w_packed,
                              hipStream_t stream);

/*
 * Per-token symmetric int8 quantization (the 8-bit activation cast of
 * Sec. 3.4), exactly as defined at the top of this header.
 *   x        device, bf16 bit patterns [M][K], finite values, 16-byte aligned
 *   M, K     0 <= M <= W4A8_M_MAX, K % 128 == 0, K <= W4A8_K_MAX; M == 0 is a no-op
 *   x_q      device, int8 [M][K], 16-byte aligned
 *   x_scale  device, fp32 [M], 4-byte aligned
 * Results are bit-identical to the IEEE-754 fp32 definition (division and
 * round-half-even).  Non-finite inputs give unspecified codes.
 */
w4a8_status w4a8_quantize_act(const uint16_t* x, int64_t M, int64_t K, int8_t* x_q,
                              float* x_scale, hipStream_t stream);

/*
 * The normalization prologue of a backbone linear: RMSNorm of each token row,
 * then the per-token quantize of w4a8_quantize_act applied to the fp32
 * normalized row, in one kernel.  FlashDrive, Sec. 3.5 ("Kernel Fusion"),
 * folds the pointwise and row-reduction work around the GEMMs into them,
 * without saying which ops those are; RMSNorm with a learned gain is this library's
 * reading of the normalization in front of the QKV and gate+up projections.
 * Per row m, with fp32 IEEE operations unless stated:
 *     ss = sum_k x[m,k]^2      (fp64, every square exact; any summation order)
 *     v  = fl32(ss / K)        (fp64 division rounded to fp32)
 *     r  = 1 / sqrt(v + eps)
 *     h[m,k] = (x[m,k] * r) * gamma[k]
 *     x_scale[m] = max_k |h[m,k]| / 127,
 *     x_q[m,k] = round_half_even(h[m,k] / x_scale[m])   (0 for an all-zero row)
 * The output feeds w4a8_linear / w4a8_linear_swiglu as W4A8_IN_I8.
 *   x        device, bf16 bit patterns [M][K], finite, 16-byte aligned
 *   gamma    device, bf16 gain [K], finite, 16-byte aligned
 *   eps      0 < eps < inf (W4A8_EINVAL otherwise); fl32(ss / K) must be finite
 *   M, K     0 <= M <= W4A8_M_MAX (0 is a no-op), K % 128 == 0, 128 <= K <= W4A8_K_MAX
 *   x_q      device, int8 [M][K], 16-byte aligned
 *   x_scale  device, fp32 [M], 4-byte aligned
 * Does not synchronize.  The fp64 sum is reduced in a fixed order, so a call
 * is deterministic; a different order can change v only where ss / K lies
 * within a few fp64 ulps of an fp32 rounding boundary.
 */
w4a8_status w4a8_rmsnorm_quantize_act(const uint16_t* x, const uint16_t* gamma, float eps, int64_t M, int64_t K,
                                      int8_t* x_q, float* x_scale, hipStream_t stream);

/*
 * Streaming prefill attention with pre-RoPE cached keys (FlashDrive, Sec.
 * 3.1 and Fig. 3).  As the window of camera frames advances, the arriving
 * frame's tokens take the last frame position of each view, in a cache
 * ordered view by view, and are the only rows whose attention is computed;
 * the keys and values of the older frames are reused from the cache.  Keys
 * sit in the cache without their rotary embedding and are rotated at the
 * positions they hold in the window now, and the mask lets a query see the
 * keys at or before its own window position, which keeps causality across
 * views.  This call computes, for every query head h and query i,
 *     o[h][i] = sum_j softmax_j(scale * RoPE(q[h][i], pos_q[i]) . RoPE(k[h'][j], pos_k[j])) v[h'][j]
 * over the keys j with pos_k[j] <= pos_q[i] (the causal order of the
 * window), h' = h / (H / Hkv) (grouped-query heads).
 *   RoPE: rotate-half pairs (d, d + 64) turned by the angles of the
 *   caller's tables: y_d = x_d cos - x_{d+64} sin, y_{d+64} = x_{d+64} cos +
 *   x_d sin, with cos = rope_cos[p][d], sin = rope_sin[p][d]; fp32 IEEE
 *   operations, rounded to bf16.  Scores, softmax and the weighted sum run
 *   in fp32 (bf16 MFMA operands: the rotated q and k, v and the softmax
 *   weights); the output is rounded to bf16.
 *   q            device, bf16 [H][Nq][D], 16-byte aligned
 *   k, v         device, bf16 [Hkv][Nk][D] (the window's cache, any slot
 *                order: positions carry the order), 16-byte aligned
 *   pos_q, pos_k device, int32 [Nq], [Nk], window positions in [0, n_pos)
 *                (positions outside are clamped for the table lookup)
 *   rope_cos, rope_sin  device, fp32 [n_pos][D/2], 16-byte aligned
 *   D            128 (W4A8_EUNSUPPORTED otherwise)
 *   H, Hkv       1 <= Hkv, H % Hkv == 0
 *   Nq, Nk       0 <= Nq (0 is a no-op), 1 <= Nk; both <= 2^22
 *   scale        finite (e.g. 1/sqrt(D))
 *   o            device, bf16 [H][Nq][D], 16-byte aligned
 *   workspace    device, >= w4a8_stream_attention_workspace_bytes(H, Nq, Nk)
 *                bytes, 256-byte aligned: the keys rotated at their
 *                positions (computed once per call, read by every query
 *                head of their kv head), each 32-key tile's smallest and
 *                largest position, the order in which workgroups take the
 *                work items, and the partial results of key-range
 *                splits, all written before read (no zero fill
 *                needed), past the first 64 KiB, which this call leaves
 *                untouched, so that it may share one buffer with
 *                w4a8_linear's workspace; concurrent calls must not share it
 * A query that sees no key gets 0.  Does not synchronize; enqueues kernels
 * only.
 */
w4a8_status w4a8_stream_attention(const uint16_t* q, const uint16_t* k, const uint16_t* v, const int32_t* pos_q,
                                  const int32_t* pos_k, const float* rope_cos, const float* rope_sin, int64_t n_pos,
                                  int64_t H, int64_t Hkv, int64_t Nq, int64_t Nk, int64_t D, float scale, uint16_t* o,
                                  void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Workspace bytes w4a8_stream_attention needs (0 for shapes it rejects;
 * every accepted shape needs some: the rotated keys). */
size_t w4a8_stream_attention_workspace_bytes(int64_t H, int64_t Nq, int64_t Nk);

/*
 * Bytes of device workspace w4a8_linear needs for this problem (0 if none).
 * The workspace holds split-K partial sums and arrival counters (and, when
 * bf16 input is quantized by its own kernel, the int8 codes and scales).
 * The caller must
 * zero-fill a workspace once before its first use; every call leaves its
 * counters at zero again, so the same workspace can be reused by later
 * calls on the same stream.  The counters of every shape sit in the first
 * 64 KiB, which nothing else writes, so calls of different shapes (and
 * w4a8_stream_attention) can share one workspace.  Returns 0 as well for invalid shapes.
 */
size_t w4a8_linear_workspace_bytes(int64_t M, int64_t N, int64_t K, int scale_mode, int in_kind);

/*
 * The W4A8 linear layer: y[M][N] = dequant(quant8(x) . W^T).
 *   x              device, bf16 [M][K] (in_kind W4A8_IN_BF16) or int8 codes
 *                  [M][K] (W4A8_IN_I8), 16-byte aligned
 *   x_scale        device, fp32 [M] (W4A8_IN_I8 only, else ignored)
 *   M, K           0 <= M <= W4A8_M_MAX (M == 0 is a no-op), K % 128 == 0,
 *                  128 <= K <= W4A8_K_MAX
 *   w_packed       device, from w4a8_pack_weights with the same N, K
 *   w_scale        device, fp32 [N] or fp16 [K/128][N] per scale_mode; unused
 *                  for W4A8_OUT_I32_ACC
 *   N              N % 16 == 0
 *   y              device, [M][N] of out_kind, 16-byte aligned
 *   workspace      device, >= w4a8_linear_workspace_bytes(...) bytes, 256-byte
 *                  aligned, zero-filled before its first use (may be NULL if
 *                  the size is 0)
 * Does not synchronize.  Deterministic: the same inputs give the same bits.
 * Enqueues kernels only (no allocation, memory set or copy), so a call can
 * be captured into a HIP graph on `stream` and replayed.
 */
w4a8_status w4a8_linear(const void* x, int in_kind, const float* x_scale, int64_t M, int64_t K,
                        const uint8_t* w_packed, const void* w_scale, int scale_mode, int64_t N,
                        void* y, int out_kind, void* workspace, size_t workspace_bytes,
                        hipStream_t stream);

/*
 * w4a8_linear for callers that cannot allocate device memory: code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation.  It
 * takes no workspace: the memory a call of w4a8_linear keeps in the caller's
 * workspace (split-K partial sums and arrival counters, the codes and scales
 * of a bf16 input quantized by a separate kernel) lives instead in a
 * library-owned device array of W4A8_NOALLOC_SCRATCH_BYTES per GPU, held from
 * the first call on a GPU until the process ends.  Arguments and results are
 * those of w4a8_linear (the same kernels, the same bits).
 *   - A problem whose w4a8_linear_workspace_bytes exceeds
 *     W4A8_NOALLOC_SCRATCH_BYTES returns W4A8_EUNSUPPORTED before anything
 *     is enqueued.
 *   - No call allocates or frees memory or sets memory with a memset; a split
 *     call clears its arrival counters with a small kernel, so the array
 *     needs no initial contents.
 *   - Every call on a GPU shares that GPU's array and finds the previous
 *     call's contents there: calls on one stream are ordered, but calls that
 *     can overlap on one GPU (different streams, or graphs replayed
 *     concurrently) race and must not be issued.
 *   - `stream` must belong to the current device.
 */
#define W4A8_NOALLOC_SCRATCH_BYTES (32u << 20)
w4a8_status w4a8_linear_noalloc(const void* x, int in_kind, const float* x_scale, int64_t M, int64_t K,
                                const uint8_t* w_packed, const void* w_scale, int scale_mode, int64_t N,
                                void* y, int out_kind, hipStream_t stream);

/*
 * Introspection for benchmarks and tests: a static, thread-local text
 * naming the kernels and tiling w4a8_linear would use for this problem and
 * its workspace size ("invalid shape" for a shape w4a8_linear rejects).
 * Enqueues nothing.
 */
const char* w4a8_linear_describe(int64_t M, int64_t N, int64_t K, int scale_mode, int in_kind,
                                 int out_kind);

/*
 * The fused gate+up projection with its gated activation merged into the
 * GEMM's epilogue.  FlashDrive, Sec. 3.5 ("Kernel Fusion"), runs the MLP's
 * gate and up projections as one GEMM and merges the element-wise
 * operations that follow into the kernels; the paper does not name the
 * activation, and this library takes SiLU (a reading: the usual gated-MLP
 * activation):
 *     y[m][f] = silu(g[m][f]) * u[m][f],   silu(g) = g / (1 + e^-g),
 * where g[m][f] and u[m][f] are the fp32 values w4a8_linear computes for
 * output columns f (gate) and N/2 + f (up) of the same call, before their
 * bf16 rounding.  silu and the product are evaluated in fp32 (e^-g with the
 * fast exponential), the result is rounded once to the output type.
 *   - W [N][K] holds the gate rows [0, N/2) followed by the up rows
 *     [N/2, N), packed by w4a8_pack_weights as one weight; w_scale covers
 *     all N columns in that order (fp32 [N] or fp16 [K/128][N]).
 *   - y is [M][N/2] of out_kind, W4A8_OUT_BF16 or W4A8_OUT_F32.
 *   - N % 32 == 0 (whole 16-column tiles in each half); other arguments and
 *     the workspace as for w4a8_linear, with its own size query below.
 *     W4A8_OUT_I32_ACC and N % 32 != 0 are W4A8_EINVAL; M == 0 is a no-op.
 *   - Every M the plain call takes: M <= 64 runs the small-M kernels,
 *     larger M the large-M kernel on its 128 x 128 tile.
 * Does not synchronize; enqueues kernels only (graph-capturable), like
 * w4a8_linear.
 */
w4a8_status w4a8_linear_swiglu(const void* x, int in_kind, const float* x_scale, int64_t M, int64_t K,
                               const uint8_t* w_packed, const void* w_scale, int scale_mode, int64_t N,
                               void* y, int out_kind, void* workspace, size_t workspace_bytes,
                               hipStream_t stream);

/* Workspace bytes w4a8_linear_swiglu needs (0 if none, and 0 for shapes it
 * rejects); the same zero-fill-once contract as w4a8_linear's workspace. */
size_t w4a8_linear_swiglu_workspace_bytes(int64_t M, int64_t N, int64_t K, int scale_mode, int in_kind);

/* The kernels w4a8_linear_swiglu would use, as w4a8_linear_describe. */
const char* w4a8_linear_swiglu_describe(int64_t M, int64_t N, int64_t K, int scale_mode, int in_kind);

/*
 * Which steps of an n_steps flow-matching solve evaluate the action network
 * and which reuse the cached velocity.  FlashDrive, Sec. 3.3 ("Adaptive
 * caching"): the first few and the last few steps are evaluated, and
 * n_reuse steps between them take the velocity of the last evaluated step.
 * The paper leaves the split of the evaluated steps between the two ends
 * open; this library's reading splits them evenly, the odd one at the
 * start: steps i < h and i >= h + n_reuse are evaluated, h = ceil((n_steps
 * - n_reuse) / 2).  The paper's 8 steps with 4 reused give 1 1 0 0 0 0 1 1.
 *   n_steps  1 <= n_steps <= 4096
 *   n_reuse  0 <= n_reuse < n_steps (step 0 is always evaluated)
 *   fresh    host, int32 [n_steps]: 1 evaluate, 0 reuse
 * Host-only: touches no device.
 */
w4a8_status w4a8_flow_schedule(int64_t n_steps, int64_t n_reuse, int32_t* fresh);

/*
 * One explicit Euler step x <- x + dt v of the flow-matching ODE of the
 * action head, with the velocity cache (FlashDrive, Sec. 3.3).  The action
 * network stays outside this library (the paper keeps it in BF16); its
 * velocity output is the input here.
 *   - Evaluated step (v_new != NULL): x[b,i] = fl32(x[b,i] + fl32(dt v_new[b,i])),
 *     then v_cache = v_new; with stats != NULL, per row b the sums behind
 *     the consecutive-velocity relative difference ||v - c|| / ||c|| and
 *     cosine v.c / (||v|| ||c||) that motivate the reuse, against the cache
 *     c before the step:
 *         stats[b] = (sum_i v c, sum_i v v, sum_i c c, sum_i (v - c)^2)
 *     each term formed in fp64 (exact for the products), summed in fp64
 *     in an unspecified order.
 *   - Reused step (v_new == NULL): x[b,i] = fl32(x[b,i] + fl32(dt v_cache[b,i]));
 *     the cache is unchanged, and stats must be NULL.
 * Both fp32 operations are rounded separately (no fused multiply-add), so
 * x and the cache are bit-exact functions of the inputs.
 * `repeat` applies the update that many times in the one call, each
 * rounded as a separate step: an evaluated step and the reused steps that
 * follow it (all with its velocity) take one call with repeat = 1 + the
 * number of reused steps, giving the bits of the step-by-step calls with
 * one pass over x.  The schedule 1 1 0 0 0 0 1 1 becomes four calls with
 * repeat 1, 5, 1, 1.
 *   x        device, fp32 [B][n] trajectory state, 16-byte aligned, updated in place
 *   v_new    device, bf16 [B][n] or NULL, 16-byte aligned
 *   v_cache  device, bf16 [B][n], 16-byte aligned (v_new may equal it;
 *            no other overlap among x, v_new and v_cache is allowed)
 *   B, n     0 <= B <= 2^24 (0 is a no-op), 1 <= n <= 2^26
 *   dt       finite (1 / n_steps for uniform steps)
 *   repeat   1 <= repeat <= 4096
 *   stats    device, fp64 [B][4] or NULL, 8-byte aligned
 * Does not synchronize.  One workgroup per row: rows of thousands of
 * elements and more reach HBM rates, the paper's trajectories (a few
 * hundred values per sample) are launch-bound.
 */
w4a8_status w4a8_flow_step(float* x, const uint16_t* v_new, uint16_t* v_cache, int64_t B, int64_t n, float dt,
                           int64_t repeat, double* stats, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* W4A8_H_ */
