// Rate probes for the rooflines of the attention kernels. Each measures what
// this chip sustains for the resource a kernel is bound by, in that kernel's
// launch shape, so a kernel's rate can be set against the achievable rate as
// well as against the published peak. Neither computes attention.
//
//   * mfma_rate_kernel issues only v_mfma_f32_32x32x16_bf16 the way the
//     chunked-prefill kernel does: eight wavefronts per workgroup (two per
//     SIMD), four independent accumulators per wavefront, 32 x 16 and
//     16 x 32 bf16 fragments in registers. The operands are pseudo-random:
//     the matrix units' power, and with it the clock the chip holds, depends
//     on how many operand bits toggle, so constant operands overstate the
//     sustained rate.
//   * read_blocks_kernel reads, through a block table, the K and V tiles of
//     every block a decode batch reads, one wavefront per (kv head, sequence,
//     split of the context) in the decode kernel's grid order and, like that
//     kernel, in steps of 64 tokens (four blocks) whose 32 loads are all
//     issued before any is used: 16-byte non-temporal loads of 1 KiB per
//     instruction. It sums the words so that every load stays live. Its rate
//     is the memory system's for this pattern of 4 KiB tiles in randomly
//     placed blocks. (Reading block by block instead, eight loads in flight
//     per wavefront, measured 2.5% slower.)

#include <hip/hip_runtime.h>

#include "abi_internal.hpp"
#include "common.hpp"
#include "kvattn_probes.h"

namespace kvattn {

namespace {

constexpr int kProbeThreads = 512;    // eight wavefronts, as the prefill kernel
// LDS the matrix probe reserves: as the prefill kernel's, more than half of
// the 160 KiB of a CU, so that one workgroup runs per CU and two wavefronts
// per SIMD (its registers alone would let two workgroups share a CU)
constexpr int kProbeLdsBytes = 96 * 1024;
constexpr int kProbeBS = 16;          // tokens per block, as every kernel here
constexpr int kReadSplitTokens = 1024;
constexpr int kReadTileBytes = 4096;  // one (block, K/V, kv head) tile the read probe is built for
constexpr int kReadStepBlocks = 4;    // blocks per step (64 tokens), as the decode kernel

typedef float f32x16_t __attribute__((ext_vector_type(16)));

__global__ __attribute__((amdgpu_flat_work_group_size(kProbeThreads, kProbeThreads),
                          amdgpu_waves_per_eu(2, 2)))
void mfma_rate_kernel(float* __restrict__ out, unsigned long long* __restrict__ clocks,
                      int iters) {
  __shared__ float lds_pad[kProbeLdsBytes / 4];
  const int lane = threadIdx.x;
  // four A and four B fragments per lane from a linear congruential sequence
  // seeded by the thread's global index, values in [-1, 1)
  bf16x8_t a[4], b[4];
  uint32_t h = (blockIdx.x * (uint32_t)kProbeThreads + lane) * 2654435761u;
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      h = h * 1664525u + 1013904223u;
      a[j][i] = (__bf16)((float)((h >> 8) & 0xffff) / 32768.f - 1.f);
      h = h * 1664525u + 1013904223u;
      b[j][i] = (__bf16)((float)((h >> 8) & 0xffff) / 32768.f - 1.f);
    }
  f32x16_t acc[4];
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[j][i] = 0.f;
  // the shader clock counter and the 100 MHz real-time counter around the
  // loop: their ratio is the clock the chip ran the wavefront at
  const unsigned long long t0 = __builtin_amdgcn_s_memtime();
  const unsigned long long r0 = __builtin_amdgcn_s_memrealtime();
  // per iteration 8 instructions, two per accumulator, each pairing A
  // fragment m % 4 with B fragment (m + m / 4) % 4
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int m = 0; m < 8; ++m)
      acc[m % 4] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[m % 4], b[(m + m / 4) % 4],
                                                           acc[m % 4], 0, 0, 0);
  }
  const unsigned long long t1 = __builtin_amdgcn_s_memtime();
  const unsigned long long r1 = __builtin_amdgcn_s_memrealtime();
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int i = 0; i < 16; ++i) s += acc[j][i];
  // the sum passes through the reserved LDS, which keeps it allocated
  lds_pad[lane] = s;
  __syncthreads();
  out[(size_t)blockIdx.x * kProbeThreads + lane] = lds_pad[lane];
  if (clocks != nullptr && lane % kWave == 0) {
    unsigned long long* c = clocks + ((size_t)blockIdx.x * (kProbeThreads / kWave) + lane / kWave) * 4;
    c[0] = t0;
    c[1] = t1;
    c[2] = r0;
    c[3] = r1;
  }
}

__global__ __launch_bounds__(64) void read_blocks_kernel(
    const uint8_t* __restrict__ kv, int num_blocks, const int* __restrict__ block_table,
    const int* __restrict__ seq_lens, int num_seqs, int num_kv_heads, int max_blocks,
    int max_seq_len, uint32_t* __restrict__ out) {
  constexpr int kChunks = kReadTileBytes / 1024;
  const int wid = blockIdx.x;
  const int g = wid % num_kv_heads;
  const int s = (wid / num_kv_heads) % num_seqs;
  const int split = wid / (num_kv_heads * num_seqs);
  const int lane = threadIdx.x;
  int L = seq_lens[s];
  L = min(max(L, 0), min(max_seq_len, max_blocks * kProbeBS));
  uint32_t sum = 0;
  const int t0 = split * kReadSplitTokens;
  if (t0 < L) {
    const int t1 = min(L, t0 + kReadSplitTokens);
    const int* bt = block_table + (size_t)s * max_blocks;
    const size_t block_bytes = 2 * (size_t)num_kv_heads * kReadTileBytes;
    const size_t k_off = (size_t)g * kReadTileBytes;
    const size_t v_off = (size_t)(num_kv_heads + g) * kReadTileBytes;
    for (int tb = t0; tb < t1; tb += kReadStepBlocks * kProbeBS) {
      // the step's blocks that hold a token in [t0, t1) and have an id inside the layer
      int id[kReadStepBlocks];
#pragma unroll
      for (int j = 0; j < kReadStepBlocks; ++j) {
        id[j] = tb + j * kProbeBS < t1 ? bt[tb / kProbeBS + j] : -1;
        if ((unsigned)id[j] >= (unsigned)num_blocks) id[j] = -1;
      }
      uint4 x[kReadStepBlocks][2 * kChunks];
#pragma unroll
      for (int j = 0; j < kReadStepBlocks; ++j) {
        if (id[j] < 0) continue;
        const uint8_t* base = kv + (size_t)id[j] * block_bytes;
        const uint4* kp = reinterpret_cast<const uint4*>(base + k_off) + lane;
        const uint4* vp = reinterpret_cast<const uint4*>(base + v_off) + lane;
#pragma unroll
        for (int c = 0; c < kChunks; ++c) {
          x[j][c] = load_nt(kp + c * kWave);
          x[j][kChunks + c] = load_nt(vp + c * kWave);
        }
      }
#pragma unroll
      for (int j = 0; j < kReadStepBlocks; ++j) {
        if (id[j] < 0) continue;
#pragma unroll
        for (int c = 0; c < 2 * kChunks; ++c) sum += x[j][c].x + x[j][c].y + x[j][c].z + x[j][c].w;
      }
    }
  }
  out[(size_t)wid * kWave + lane] = sum;
}

int hip_fail(hipError_t e, const char* what) {
  return set_error(KV_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

}  // namespace

}  // namespace kvattn

using kvattn::clear_error;
using kvattn::set_error;

extern "C" int kvattn_probe_mfma_threads(void) { return kvattn::kProbeThreads; }

extern "C" int kvattn_probe_mfma(float* out, uint64_t* clocks, int num_workgroups, int iters,
                                 void* stream) {
  clear_error();
  if (num_workgroups <= 0 || iters < 0)
    return set_error(KV_ERR_INVALID, "kvattn_probe_mfma: %d workgroups, %d iterations",
                     num_workgroups, iters);
  if (!out) return set_error(KV_ERR_INVALID, "kvattn_probe_mfma: null output");
  hipLaunchKernelGGL(kvattn::mfma_rate_kernel, dim3(num_workgroups), dim3(kvattn::kProbeThreads),
                     0, static_cast<hipStream_t>(stream), out,
                     reinterpret_cast<unsigned long long*>(clocks), iters);
  const hipError_t e = hipGetLastError();
  return e == hipSuccess ? KV_OK : kvattn::hip_fail(e, "kvattn_probe_mfma launch");
}

extern "C" int kvattn_probe_read_blocks_waves(int num_seqs, int num_kv_heads, int max_seq_len) {
  if (num_seqs <= 0 || num_kv_heads <= 0 || max_seq_len <= 0) return 0;
  const long long splits = (max_seq_len + kvattn::kReadSplitTokens - 1) / kvattn::kReadSplitTokens;
  const long long w = splits * num_seqs * num_kv_heads;
  return w > 0x7fffffff ? -1 : (int)w;
}

extern "C" int kvattn_probe_read_blocks(const void* kv_layer, int num_blocks,
                                        const int32_t* block_table, const int32_t* seq_lens,
                                        int num_seqs, int num_kv_heads, int head_dim,
                                        kv_dtype dtype, int max_blocks, int max_seq_len,
                                        uint32_t* out, void* stream) {
  clear_error();
  if (num_seqs <= 0 || num_kv_heads <= 0 || num_blocks <= 0 || max_blocks <= 0 ||
      max_seq_len <= 0 || head_dim <= 0 || (dtype != KV_BF16 && dtype != KV_F32))
    return set_error(KV_ERR_INVALID,
                     "kvattn_probe_read_blocks: %d seqs, %d kv heads, %d blocks, %d table "
                     "columns, max_seq_len %d, head_dim %d, dtype %d",
                     num_seqs, num_kv_heads, num_blocks, max_blocks, max_seq_len, head_dim,
                     (int)dtype);
  const int elem_bytes = dtype == KV_BF16 ? 2 : 4;
  const long long tile = (long long)kvattn::kProbeBS * head_dim * elem_bytes;
  if (tile != kvattn::kReadTileBytes)
    return set_error(KV_ERR_UNSUPPORTED,
                     "kvattn_probe_read_blocks: built for 4 KiB tiles, not %lld bytes", tile);
  const int waves = kvattn_probe_read_blocks_waves(num_seqs, num_kv_heads, max_seq_len);
  if (waves <= 0) return set_error(KV_ERR_UNSUPPORTED, "kvattn_probe_read_blocks: grid too large");
  if (!kv_layer || !block_table || !seq_lens || !out)
    return set_error(KV_ERR_INVALID, "kvattn_probe_read_blocks: null pointer argument");
  if ((reinterpret_cast<uintptr_t>(kv_layer) & 15) != 0)
    return set_error(KV_ERR_INVALID, "kvattn_probe_read_blocks: layer not 16-byte aligned");
  hipLaunchKernelGGL(kvattn::read_blocks_kernel, dim3(waves), dim3(kvattn::kWave), 0,
                     static_cast<hipStream_t>(stream), static_cast<const uint8_t*>(kv_layer),
                     num_blocks, block_table, seq_lens, num_seqs, num_kv_heads, max_blocks,
                     max_seq_len, out);
  const hipError_t e = hipGetLastError();
  return e == hipSuccess ? KV_OK : kvattn::hip_fail(e, "kvattn_probe_read_blocks launch");
}
