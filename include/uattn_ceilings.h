/*
 * uattn_ceilings -- measured ceilings for the roofline fractions of libuattn
 * (libuattn_ceilings.so).  Two microbenchmark kernels whose only purpose is
 * to measure, on the GPU at hand, what the attention kernels are compared
 * against besides the datasheet peaks:
 *
 *   uattn_ceiling_read   -- streaming HBM read bandwidth, either over one
 *                           contiguous buffer or over 16 KB blocks visited in
 *                           the order of a block table (the page-gathered
 *                           pattern of the paged-KV decode, where one
 *                           (page, kv head) is 64 keys x 128 dims x 2 bytes);
 *   uattn_ceiling_mfma   -- dense bf16 matrix-core throughput of
 *                           v_mfma_f32_16x16x32_bf16 with independent
 *                           accumulators and no memory traffic.
 *
 * Conventions as in uattn.h: device pointers, caller-owned buffers, calls
 * enqueue on `stream` and return; the caller times them (HIP events).
 * Errors are return codes (0 = OK, 1 = invalid argument, 4 = launch failed).
 */
#ifndef UATTN_CEILINGS_H
#define UATTN_CEILINGS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/*
 * Read `num_blocks` blocks of `block_bytes` bytes each and fold every 16-byte
 * piece into a per-workgroup XOR checksum.
 *
 *   src          base of the buffer, 16-byte aligned
 *   block_table  [num_blocks] int32 block indices into src (block i read at
 *                src + block_table[i] * block_bytes), or NULL for the
 *                identity order (one contiguous stream); entries are trusted
 *   block_bytes  a multiple of 16384
 *   flags        0, or 1 for loads with the non-temporal cache hint
 *   checksum     [grid] uint32 (written), grid = uattn_ceiling_read_grid()
 *
 * The XOR of all `grid` checksum words equals the XOR of every 32-bit word of
 * the blocks read, whatever the order.
 */
int32_t uattn_ceiling_read(const void* src, const int32_t* block_table, int64_t num_blocks, int64_t block_bytes,
                           int32_t flags, uint32_t* checksum, void* stream);

/* Workgroups uattn_ceiling_read launches on the current device. */
int32_t uattn_ceiling_read_grid(void);

/*
 * `waves` wavefronts each issue `iters` x 8 independent
 * v_mfma_f32_16x16x32_bf16 (16 x 16 x 32 x 2 = 16384 FLOP each), with no
 * memory traffic in the loop; each wave writes one float (the sum of its
 * accumulators) to out[wave] so that the work cannot be removed.
 *   FLOP of a call = waves * iters * 8 * 16384.
 */
int32_t uattn_ceiling_mfma(int32_t waves, int32_t iters, float* out, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* UATTN_CEILINGS_H */
