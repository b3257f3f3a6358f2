/*
 * w4a8_ceiling.h - measured ceilings of HBM reads and INT8 matrix cores on
 * the MI355X (gfx950), reported beside the published peaks (8 TB/s, 5.0
 * POPS dense INT8) that the W4A8 layer's roofline fractions use.  These are
 * measurement probes, not part of the layer (the layer's C ABI is w4a8.h);
 * they live in their own library, libw4a8_ceiling.so.
 *
 * Both calls enqueue one kernel on `stream` and return a hipError_t value
 * (0 = success); invalid arguments return hipErrorInvalidValue without a
 * launch.  Pointers are device pointers owned by the caller.
 */
#ifndef W4A8_CEILING_H_
#define W4A8_CEILING_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define W4A8_CEILING_READ_BLOCKS 256                 /* workgroups of 512 threads */
#define W4A8_CEILING_READ_SINK_WORDS (256 * 512)     /* one word per thread */
#define W4A8_CEILING_MAX_READ_BYTES ((1ull << 31) - (1ull << 24))
#define W4A8_CEILING_MFMA_BLOCKS 1024                /* workgroups of 256 threads (4 waves) */
#define W4A8_CEILING_MFMA_SINK_WORDS (1024 * 256)

/* Read `bytes` (a multiple of 16, at most W4A8_CEILING_MAX_READ_BYTES) of
 * `buf` once with 16-byte non-temporal loads.  Workgroup b reads the range
 * [b P, (b + 1) P) clipped to the buffer, with
 * P = 16 * ceil(bytes / (16 * W4A8_CEILING_READ_BLOCKS)); its thread i reads
 * the 16-byte chunks at i * 16 + j * 8192 (j = 0, 1, ...) of that range and
 * writes the XOR of all their 32-bit words to sink[b * 512 + i]
 * (W4A8_CEILING_READ_SINK_WORDS words). */
int w4a8_ceiling_stream_read(const void* buf, size_t bytes, uint32_t* sink, hipStream_t stream);

/* Run, on every wave of W4A8_CEILING_MFMA_BLOCKS x 4 waves, four independent
 * chains of `iters` v_mfma_i32_32x32x32_i8 (65536 int8 ops each) on all-one
 * operands.  Each thread writes the sum of its 64 accumulator words to
 * sink[t], which is 2048 * iters (mod 2^32); total work is
 * 1024 * 4 * 4 * iters * 65536 ops. */
int w4a8_ceiling_mfma_i8(int iters, int32_t* sink, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif  /* W4A8_CEILING_H_ */
