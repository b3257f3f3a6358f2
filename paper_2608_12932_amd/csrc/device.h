// Device helpers shared by the W4A8 kernels (gfx950 only).
//
// Packed weight layout (written by pack.hip, read by both GEMM paths).
//   The N x K int4 weight is cut into blocks of 16 output channels x 128 k
//   (one scale group), 1 KiB each, stored block-column-major:
//       block (t, b) at byte ((t * KB) + b) * 1024,  t = n / 16,  b = k / 128.
//   Inside a block, 16-byte chunk j = g * 16 + c (g = 0..3, c = 0..15) holds
//   channel 16 t + c, k in [128 b + 32 g, 128 b + 32 g + 32): byte i carries
//   k = 128 b + 32 g + i in its low nibble and k + 16 in its high nibble.
//   So a wave reading a block with lane l <- chunk l is one contiguous 1 KiB
//   load, and each lane's 16 bytes unpack into the B fragments of two int8
//   MFMAs without any shuffle.
//
// Nibble unpack: masking a nibble into the high half of a byte gives the
// signed byte 16 * w exactly for w in [-8, 7], so the MFMA accumulates
// 16 * acc; the factor is removed with an exact arithmetic shift (or folded
// into a power-of-two scale).  |16 * acc| <= 16 * 127 * 8 * K < 2^31 for
// K <= 65536.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <string.h>

namespace w4a8 {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));
typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));

constexpr int kGroup = 128;       // k per block and per group scale
constexpr int kNTile = 16;        // output channels per block
constexpr int kBlockBytes = 1024; // 16 x 128 x 4 bit

// Workgroup barrier that orders LDS traffic only: global loads still in
// flight stay in flight (a plain __syncthreads would wait for them).
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// MFMA operands from one packed 16-byte chunk: low nibbles (k .. k+15) and
// high nibbles (k+16 .. k+31), each as 16 signed bytes of value 16 * w.
__device__ __forceinline__ v4i nib_lo(uint4 c) {
  v4i r;
  r[0] = (int)((c.x << 4) & 0xF0F0F0F0u);
  r[1] = (int)((c.y << 4) & 0xF0F0F0F0u);
  r[2] = (int)((c.z << 4) & 0xF0F0F0F0u);
  r[3] = (int)((c.w << 4) & 0xF0F0F0F0u);
  return r;
}
__device__ __forceinline__ v4i nib_hi(uint4 c) {
  v4i r;
  r[0] = (int)(c.x & 0xF0F0F0F0u);
  r[1] = (int)(c.y & 0xF0F0F0F0u);
  r[2] = (int)(c.z & 0xF0F0F0F0u);
  r[3] = (int)(c.w & 0xF0F0F0F0u);
  return r;
}
__device__ __forceinline__ v4i as_v4i(uint4 c) {
  v4i r;
  r[0] = (int)c.x; r[1] = (int)c.y; r[2] = (int)c.z; r[3] = (int)c.w;
  return r;
}

__device__ __forceinline__ v4i mfma16(v4i a, v4i b, v4i c) {
  return __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ v16i mfma32(v4i a, v4i b, v16i c) {
  return __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float bf16_lo(uint32_t pair) { return __uint_as_float(pair << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t pair) { return __uint_as_float(pair & 0xFFFF0000u); }

// fp32 -> bf16 bits, round to nearest even; NaN -> 0x7FC0.
__device__ __forceinline__ uint32_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu)) return 0x7FC0u;
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}

// Two floats to bf16 with the hardware conversion (round to nearest even;
// bit-identical to f32_to_bf16 for every input but NaN, whose payload it
// keeps): low half from lo, high half from hi.
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float float2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t bf16x2_bits(float lo, float hi) {
  const float2_t v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}
// NaN (any sign or payload) replaced by the canonical quiet NaN; other
// values kept.
__device__ __forceinline__ float canonical_nan(float f) { return f != f ? __uint_as_float(0x7FC00000u) : f; }

__device__ __forceinline__ float f16_to_f32(uint16_t h) {
  _Float16 v;
  memcpy(&v, &h, 2);
  return (float)v;
}

// max(|a|) of the two bf16 values in each dword, as 16-bit magnitudes:
// for finite values the magnitude bit patterns order like the numbers.
__device__ __forceinline__ uint32_t absmax_pairs(uint32_t acc, uint32_t pair) {
  u16x2 a, p;
  memcpy(&a, &acc, 4);
  uint32_t m = pair & 0x7FFF7FFFu;
  memcpy(&p, &m, 4);
  u16x2 r = __builtin_elementwise_max(a, p);
  uint32_t o;
  memcpy(&o, &r, 4);
  return o;
}
__device__ __forceinline__ uint32_t absmax_chunk(uint32_t acc, uint4 c) {
  acc = absmax_pairs(acc, c.x);
  acc = absmax_pairs(acc, c.y);
  acc = absmax_pairs(acc, c.z);
  acc = absmax_pairs(acc, c.w);
  return acc;
}
__device__ __forceinline__ uint32_t fold_pair_max(uint32_t acc) {
  uint32_t lo = acc & 0xFFFFu, hi = acc >> 16;
  return lo > hi ? lo : hi;
}

__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    uint32_t o = (uint32_t)__shfl_xor((int)v, off, 64);
    v = v > o ? v : o;
  }
  return v;
}

// Per-token quantization parameters derived from the row's max |x|.
//   s = a / 127 and inv = 1 / s are IEEE fp32 divisions.  Codes are
//   round_half_even(fl(x / s)); for a >= 2^-96 fl(x / s) is obtained as
//   p = x * inv corrected by one Markstein step (two fmas), which an
//   exhaustive check over every pair of bf16 values (x, a) with |x| <= a and
//   a >= 2^-96 (tests/quant_exhaustive.c, run by tests/test_quant_proof.py)
//   shows to give the code of the correctly rounded quotient; below 2^-96
//   the residual can underflow, so those rows use the IEEE division directly.
struct QScale {
  float s, inv;
  int mode;  // 0: all-zero row, 1: reciprocal + correction, 2: IEEE division
};

__device__ __forceinline__ QScale qscale_from_absmax(float a) {
  QScale q;
  if (a == 0.0f) {
    q.s = 0.0f; q.inv = 0.0f; q.mode = 0;
  } else {
    q.s = a / 127.0f;
    q.inv = 1.0f / q.s;
    q.mode = a >= 0x1p-96f ? 1 : 2;
  }
  return q;
}

// Adding 1.5 * 2^23 rounds a value of magnitude < 2^22 to the nearest
// integer, ties to even, and leaves that integer (two's complement) in the
// low mantissa bits; the code is the low byte of the result.
__device__ __forceinline__ uint32_t qcode_fast(float x, float s, float inv) {
  float p = __fmul_rn(x, inv);
  float e = __fmaf_rn(-s, p, x);
  float r = __fmaf_rn(e, inv, p);
  return __float_as_uint(__fadd_rn(r, 12582912.0f));
}
__device__ __forceinline__ uint32_t qcode_div(float x, float s) {
  return __float_as_uint(__fadd_rn(__fdiv_rn(x, s), 12582912.0f));
}

// Pack the low bytes of four words into one word (byte i from word i).
__device__ __forceinline__ uint32_t pack4(uint32_t b0, uint32_t b1, uint32_t b2, uint32_t b3) {
  uint32_t lo = __builtin_amdgcn_perm(b1, b0, 0x0c0c0400u);
  uint32_t hi = __builtin_amdgcn_perm(b3, b2, 0x0c0c0400u);
  return __builtin_amdgcn_perm(hi, lo, 0x05040100u);
}

// Quantize 8 bf16 values (one 16-byte chunk) into 8 codes (two words).
// `mode` must be uniform across the wave (it is a per-token property).
__device__ __forceinline__ uint2 quant_chunk(uint4 c, float s, float inv, int mode) {
  uint2 o;
  if (mode == 1) {
    o.x = pack4(qcode_fast(bf16_lo(c.x), s, inv), qcode_fast(bf16_hi(c.x), s, inv),
                qcode_fast(bf16_lo(c.y), s, inv), qcode_fast(bf16_hi(c.y), s, inv));
    o.y = pack4(qcode_fast(bf16_lo(c.z), s, inv), qcode_fast(bf16_hi(c.z), s, inv),
                qcode_fast(bf16_lo(c.w), s, inv), qcode_fast(bf16_hi(c.w), s, inv));
  } else if (mode == 2) {
    o.x = pack4(qcode_div(bf16_lo(c.x), s), qcode_div(bf16_hi(c.x), s),
                qcode_div(bf16_lo(c.y), s), qcode_div(bf16_hi(c.y), s));
    o.y = pack4(qcode_div(bf16_lo(c.z), s), qcode_div(bf16_hi(c.z), s),
                qcode_div(bf16_lo(c.w), s), qcode_div(bf16_hi(c.w), s));
  } else {
    o.x = 0u;
    o.y = 0u;
  }
  return o;
}

// Streaming (non-temporal) 16-byte load: packed weights are read once per
// call, so they should not displace activations from the caches.
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 ldg_nt(const uint4* p) {
  const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  return make_uint4(v[0], v[1], v[2], v[3]);
}

// ---- buffer loads
// A raw buffer resource covers `bytes` bytes from `base`; a load whose
// offset lies at or beyond that range returns zeros without touching memory.
// Tails and padding are therefore expressed as out-of-range offsets instead
// of branches: a guarded load would otherwise become a branch whose join
// forces the wave to wait for the load right away, serializing the stream.
constexpr uint32_t kOOB = 0x80000000u;       // offset beyond any range used here
constexpr int kCacheDefault = 0;
constexpr int kCacheStream = 2;              // non-temporal: read once, do not keep

// A pointer the compiler may have placed in vector registers although it
// is the same in every lane, moved to scalar registers (so that a buffer
// descriptor built from it stays scalar).
template <class T>
__device__ __forceinline__ T* uniform_ptr(T* p) {
  const uint64_t v = (uint64_t)(uintptr_t)p;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v), hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  return reinterpret_cast<T*>((uintptr_t)(((uint64_t)hi << 32) | lo));
}
// The same for a 32-bit value.
__device__ __forceinline__ uint32_t uniform_u32(uint32_t v) { return __builtin_amdgcn_readfirstlane(v); }
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

template <int kAux = kCacheDefault>
__device__ __forceinline__ uint4 buf_load16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  const v4i v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, kAux);
  return make_uint4((uint32_t)v[0], (uint32_t)v[1], (uint32_t)v[2], (uint32_t)v[3]);
}

// Same with a wave-uniform scalar offset added to the address.  Range checks
// apply to the vector offset, so an out-of-range vector offset still reads
// zeros; in-range vector offsets are only ever paired with scalar offsets
// that keep the address inside the resource.
template <int kAux = kCacheDefault>
__device__ __forceinline__ uint4 buf_load16s(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
  const v4i v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, (int)soff, kAux);
  return make_uint4((uint32_t)v[0], (uint32_t)v[1], (uint32_t)v[2], (uint32_t)v[3]);
}
template <int kAux = kCacheDefault>
__device__ __forceinline__ uint16_t buf_load2s(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
  return (uint16_t)__builtin_amdgcn_raw_buffer_load_b16(r, (int)voff, (int)soff, kAux);
}

// ---- direct HBM -> LDS loads (LDS DMA)
// A raw buffer descriptor as four words (base, base_hi, bytes, format) for
// inline assembly; same range semantics as make_rsrc.
__device__ __forceinline__ u32x4 make_rsrc_words(const void* base, uint32_t bytes) {
  const uint64_t b = (uint64_t)(uintptr_t)base;
  u32x4 r;
  r[0] = (uint32_t)b;
  r[1] = (uint32_t)(b >> 32) & 0xFFFFu;  // stride 0
  r[2] = bytes;
  r[3] = 0x00020000u;
  return r;
}
// Each lane's 16 (or 4) bytes land at lds_addr + lane * 16 (or 4); the
// wave's instruction fills 1 KiB (256 B) of LDS contiguously.  Issued as
// assembly on purpose: the compiler, unable to tell which LDS stage such a
// load fills, would otherwise wait for every one of them before any LDS
// read and empty the prefetch ring.  Callers wait with s_waitcnt vmcnt.
// The descriptor, LDS address and scalar offset must be wave-uniform values
// the compiler keeps in scalar registers (the assembler rejects the
// instruction otherwise).
__device__ __forceinline__ void lds_dma16(u32x4 rsrc, uint32_t lds_addr, uint32_t voff, uint32_t soff) {
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
               :
               : "s"(lds_addr), "v"(voff), "s"(rsrc), "s"(soff)
               : "memory");
}
__device__ __forceinline__ void lds_dma16_nt(u32x4 rsrc, uint32_t lds_addr, uint32_t voff, uint32_t soff) {
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, %3 offen nt lds"
               :
               : "s"(lds_addr), "v"(voff), "s"(rsrc), "s"(soff)
               : "memory");
}
__device__ __forceinline__ void lds_dma4(u32x4 rsrc, uint32_t lds_addr, uint32_t voff, uint32_t soff) {
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dword %1, %2, %3 offen lds"
               :
               : "s"(lds_addr), "v"(voff), "s"(rsrc), "s"(soff)
               : "memory");
}
// s_waitcnt constraining only the vector-memory count (gfx9 encoding:
// vmcnt[3:0] | expcnt[6:4] | lgkmcnt[11:8] | vmcnt[5:4] << 14).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt is 6 bits");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | (0x7 << 4) | (0xF << 8) | ((N >> 4) << 14));
}

template <int kAux = kCacheDefault>
__device__ __forceinline__ uint16_t buf_load2(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return (uint16_t)__builtin_amdgcn_raw_buffer_load_b16(r, (int)off, 0, kAux);
}

template <int kAux = kCacheDefault>
__device__ __forceinline__ uint32_t buf_load4(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(r, (int)off, 0, kAux);
}

}  // namespace w4a8
