/*
 * kvattn probes: rate measurements for the rooflines of the attention
 * kernels (decode is bound by HBM, chunked prefill by the bf16 matrix
 * units). Each probe runs in the launch shape of the kernel it stands beside
 * and does none of its arithmetic, so that the kernel's rate can be set
 * against what this chip sustains for the same resource as well as against
 * the published peak. They compute no attention and are not part of the
 * attention path; errors and streams as in kvattn.h.
 */
#ifndef KVATTN_PROBES_H
#define KVATTN_PROBES_H

#include <stddef.h>
#include <stdint.h>

#include "kvattn.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Threads per workgroup of kvattn_probe_mfma (512: eight wavefronts, two per
 * SIMD, as the chunked-prefill kernel; like that kernel it reserves 96 KiB of
 * LDS, so one workgroup runs per CU). */
int kvattn_probe_mfma_threads(void);

/* Matrix-unit rate: num_workgroups workgroups, each wavefront issuing
 * 8 * iters v_mfma_f32_32x32x16_bf16 (32768 FLOP each) on four independent
 * fp32 accumulators, with pseudo-random bf16 operands in [-1, 1) (four A and
 * four B fragments per lane from a linear congruential sequence seeded by
 * the thread's global index h * 2654435761, stepped as x * 1664525 +
 * 1013904223 with A and B draws alternating; a draw x gives
 * ((x >> 8) & 0xffff) / 32768 - 1 rounded to bf16). Instruction m of an
 * iteration (m = 0 .. 7) adds A[m % 4] B[(m + m / 4) % 4] to accumulator
 * m % 4.
 *
 * out     device float [num_workgroups * kvattn_probe_mfma_threads()]: each
 *         thread's sum of its 64 accumulator elements.
 * clocks  NULL, or device uint64 [num_workgroups * 8 * 4]: wavefront w of
 *         workgroup b writes at 4 (8 b + w) the shader clock counter
 *         (s_memtime) before and after its loop, then the 100 MHz real-time
 *         counter (s_memrealtime) before and after; the ratio of the two
 *         differences, times 100 MHz, is the clock the wavefront ran at.
 * FLOP per call = num_workgroups * 8 wavefronts * 8 * iters * 32768.
 * KV_ERR_INVALID for num_workgroups <= 0, iters < 0 or a null out.
 * Asynchronous. */
int kvattn_probe_mfma(float* out, uint64_t* clocks, int num_workgroups, int iters,
                      void* stream);

/* Wavefronts of kvattn_probe_read_blocks for a batch: one per (kv head,
 * sequence, split of 1024 context tokens), ceil(max_seq_len / 1024) splits
 * per sequence; 0 for invalid sizes, -1 if it would not fit an int. */
int kvattn_probe_read_blocks_waves(int num_seqs, int num_kv_heads, int max_seq_len);

/* Memory rate for decode's access pattern: reads, through the block table,
 * the K tile and the V tile of kv head g of every block that holds a token
 * of sequence s (blocks 0 .. ceil(L_s / 16) - 1; ids outside
 * [0, num_blocks) are skipped), laid out as kvattn_decode reads them (same
 * layer layout, block_size 16, same grid order: kv head fastest, split
 * slowest, steps of 64 tokens whose loads are all issued before any is
 * used), with 16-byte non-temporal loads of 1 KiB per instruction: lane l
 * of a wavefront reads bytes [1024 c + 16 l, 1024 c + 16 l + 16) of each
 * tile, c = 0 .. 3.
 *
 * kv_layer, num_blocks, block_table, seq_lens, num_seqs, num_kv_heads,
 * head_dim, max_blocks_per_seq, max_seq_len: as for kvattn_decode (L_s is
 * seq_lens[s] clamped to [0, min(max_seq_len, 16 * max_blocks_per_seq)]);
 * the tile, 16 * head_dim elements of dtype, must be 4 KiB (bf16 with
 * head_dim 128, fp32 with head_dim 64; KV_ERR_UNSUPPORTED otherwise).
 * out   device uint32 [kvattn_probe_read_blocks_waves(...) * 64]: lane l of
 *       wavefront w writes out[64 w + l], the sum modulo 2^32 of the 32-bit
 *       words it read (0 for a wavefront whose split holds no token).
 * Asynchronous. */
int kvattn_probe_read_blocks(const void* kv_layer, int num_blocks, const int32_t* block_table,
                             const int32_t* seq_lens, int num_seqs, int num_kv_heads,
                             int head_dim, kv_dtype dtype, int max_blocks_per_seq,
                             int max_seq_len, uint32_t* out, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* KVATTN_PROBES_H */
