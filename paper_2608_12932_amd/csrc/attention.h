// Launch interface of the streaming prefill attention (attention.hip) for
// the C ABI (api.cpp); kept apart from the GEMM interface in kernels.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace w4a8 {

struct AttnArgs {
  const uint16_t* q;      // bf16 [H][Nq][128], before the rotary embedding
  const uint16_t* k;      // bf16 [Hkv][Nk][128], before the rotary embedding
  const uint16_t* v;      // bf16 [Hkv][Nk][128]
  const int32_t* pos_q;   // [Nq] window positions
  const int32_t* pos_k;   // [Nk]
  const float* rope_cos;  // [n_pos][64]
  const float* rope_sin;  // [n_pos][64]
  uint16_t* o;            // bf16 [H][Nq][128]
  int H, Hkv, Nq, Nk, n_pos;
  float scale_log2e;      // score scale times log2(e)
  void* workspace;        // rotated keys and split partials (stream_attention_workspace bytes)
  // set by the launcher
  uint16_t* k_rot;        // bf16 [Hkv][Nk][128]: the keys rotated at their positions
  int2* tile_bounds;      // [ceil(Nk / 32)] smallest and largest key position of each 32-key tile
  int* sched;             // [items] work item of each workgroup id, or nullptr (plain order)
  int sched_cus;          // compute units the schedule deals to
  int* solo;              // [query blocks] the one split that sees keys of a block, else -1 (with sched)
  int S, tiles_per_split;
  float* part_o;          // [S][H][Nq][128] unnormalized partial sums
  float* part_ml;         // [S][H][Nq][2] running maximum (base 2) and weight total
};
hipError_t launch_stream_attention(const AttnArgs& a, hipStream_t stream);
int stream_attention_splits(int H, int Nq, int Nk);
size_t stream_attention_workspace(int H, int Nq, int Nk);

}  // namespace w4a8
