// Chunked-prefill attention for gfx950 on bf16 MFMA (the paper, Section 5:
// prefill is compute bound and a chunk attends to all earlier context, so
// chunking splits the same work; Section 1: max_num_batched_tokens bounds
// the chunk).
//
// Work tile = (kv head g, 32 * 8 / G consecutive new rows of one sequence),
// G = 1, 2, 4 or 8 query heads per kv head.
// A workgroup of 8 wavefronts (two per SIMD) owns one tile: wave w serves
// query head g * G + w % G over 32 rows. K/V steps of 64 keys (4 blocks) are
// gathered through the block table straight into LDS (global_load_lds) once
// per workgroup and shared by the G query heads of the group; three LDS
// buffers each let K be gathered three steps and V one step ahead of their
// use, with one barrier per step.
//
// Per wave and step, with v_mfma_f32_32x32x16_bf16:
//   S^T[key][row] = K[key][:] . Q[row][:]   A = K rows read from the
//       chunk-major K tile, B = Q^T held in registers for the whole kernel.
//       The A rows of a 32-key tile are loaded in a permuted key order so
//       that the accumulator of each lane ends up holding 8 consecutive keys
//       of each of the two blocks for one query row;
//   softmax over keys in the log2 domain against a per-row reference (a
//       past row max): a row's 64 scores live in two lanes (l and l + 32)
//       and the row state is lane-local. The reference is only moved, and
//       O^T and the row sum rescaled, when the row's max grows past it by
//       more than 2^8, so every exponential stays below 256, which bf16 P
//       and fp32 accumulation hold. A lane's exponentials are at most its
//       partial row sum, so a step whose partial sums all stay within 2^8
//       (nearly every step after the first) needs no row max at all; the
//       others take the exact max (one exchange between the row's two
//       lanes) and recompute the step's exponentials;
//   O^T[d][row] += V^T[d][key] P^T[key][row]   A = 16-byte runs of the
//       dim-major V tile, B = the bf16 P values of 8 consecutive keys of one
//       block, already in the lane that produced them.
// Software pipeline: while a wave computes the softmax of step i on the
// vector ALU, its matrix work is p.v of step i - 1 and q.k of step i + 1, so
// both units stay busy; the second wave of the SIMD covers the LDS latency.
// V rows are stored in LDS with their two 16-byte halves swapped on every
// other group of 8 rows, so the A reads of 16 rows hit 16 distinct bank
// groups. The causal mask (bottom-right: row i at position L - n + i sees
// keys 0 .. L - n + i) is applied only on steps that reach the diagonal or
// the end of the sequence.

#include <type_traits>

#include "common.hpp"
#include "launch.hpp"

namespace kvattn {

namespace {

constexpr int kD = 128;
constexpr int kBS = 16;
constexpr int kKeys = 64;                  // keys per step
constexpr int kStepBlocks = 4;             // blocks per step
constexpr int kTileBytes = kBS * kD * 2;   // one (block, K/V, head) tile: 4 KiB
constexpr float kLazyRescale = 8.f;        // log2 headroom before the max moves
constexpr float kPsumBound = 256.f;         // 2^kLazyRescale
constexpr int kKBufs = 3;                  // LDS K steps (gathered three steps ahead)
constexpr int kVBufs = 3;                  // LDS V steps (gathered one step ahead)
constexpr int kWaves = 8;                  // wavefronts per workgroup
constexpr int kThreads = kWaves * kWave;

typedef float f32x16_t __attribute__((ext_vector_type(16)));

__device__ __forceinline__ f32x16_t mfma32(bf16x8_t a, bf16x8_t b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// max(a, b, c) in one instruction. The scores here are never NaN (masked
// keys are set to -inf by a select), so the IEEE NaN handling that fmaxf
// adds around every operand is not needed.
__device__ __forceinline__ float max3f(float a, float b, float c) {
  float r;
  asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}

constexpr uint32_t kBf16OnePair = 0x3f803f80u;   // (1.0, 1.0) in bf16

// Two loads of 16 bytes per lane from global memory straight into LDS
// (global_load_lds_dwordx4): load j has lane l read base_j + off_j and its
// bytes land at LDS byte address lds_j + 16 l (base_j and lds_j wave-uniform,
// in SGPRs). A wave-uniform base plus a 32-bit lane offset takes the address
// unit fewer cycles per instruction than 64 lanes of 64-bit addresses. M0
// carries each load's LDS address: the block saves the compiler's M0 first
// and restores it last, so no code outside the block sees M0 change. Issued
// as inline assembly so that the compiler does not treat the loads as LDS
// stores that every later LDS read must wait for: the callers wait for them
// themselves (s_waitcnt vmcnt) before the barrier that publishes the data.
__device__ __forceinline__ void dma16x2(const void* base0, uint32_t off0, uint32_t lds0,
                                        const void* base1, uint32_t off1, uint32_t lds1) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %3\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, %2\n\t"
      "s_mov_b32 m0, %6\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %4, %5\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(off0), "s"(base0), "s"(lds0), "v"(off1), "s"(base1), "s"(lds1)
      : "memory");
}

// Entry i of a block-table row, read by a scalar memory load: the row pointer
// is wave-uniform and the index is made so, and a load through the constant
// address space from a uniform address is a scalar load. It is therefore
// counted by lgkmcnt, never by the vmcnt that the gathers are waited with.
__device__ __forceinline__ int scalar_entry(const int* row, int i) {
  const __attribute__((address_space(4))) int* p =
      (const __attribute__((address_space(4))) int*)row;
  return p[(unsigned)__builtin_amdgcn_readfirstlane(i)];
}

typedef int i32x4_t __attribute__((ext_vector_type(4)));
typedef i32x4_t i32x4_a4_t __attribute__((aligned(4)));

// Entries i .. i + 3 of a block-table row in one 16-byte scalar load (scalar
// loads need only 4-byte alignment).
__device__ __forceinline__ i32x4_t scalar_entries4(const int* row, int i) {
  const __attribute__((address_space(4))) i32x4_a4_t* p =
      (const __attribute__((address_space(4))) i32x4_a4_t*)(
          row + (unsigned)__builtin_amdgcn_readfirstlane(i));
  return *p;
}

// LDS byte address of a pointer into a __shared__ array.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

// The lane's index in its wavefront, computed afresh at each call (volatile,
// so it is not merged with an earlier copy that would have to stay live).
__device__ __forceinline__ int lane_id_fresh() {
  int r;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(r));
  return r;
}

}  // namespace

// Rows [lo, hi) of sequence s's chunk, with the offsets clamped into
// [0, total_q] and hi >= lo, so that offsets that break the documented
// contract (decreasing, or past the end of q) can neither read nor write
// outside q and out.
__device__ __forceinline__ int2 chunk_rows(const int* __restrict__ cu, int s, int total_q) {
  const int lo = min(max(cu[s], 0), total_q);
  const int hi = min(max(cu[s + 1], lo), total_q);
  return make_int2(lo, hi);
}

// Lists the work tiles (sequence, first row) of a batch of chunks, the rows
// of a sequence's chunk in descending order so the longest rows start first.
__global__ __launch_bounds__(256) void prefill_tile_map_kernel(const int* __restrict__ cu,
                                                               int num_seqs, int total_q,
                                                               int rows_per_tile,
                                                               int2* __restrict__ tiles,
                                                               int* __restrict__ count,
                                                               int max_tiles) {
  __shared__ int scan[256];
  const int tid = threadIdx.x;
  const int per = (num_seqs + 255) / 256;
  const int s0 = min(num_seqs, tid * per);
  const int s1 = min(num_seqs, s0 + per);
  int mine = 0;
  for (int s = s0; s < s1; ++s) {
    const int2 r = chunk_rows(cu, s, total_q);
    mine += (r.y - r.x + rows_per_tile - 1) / rows_per_tile;
  }
  scan[tid] = mine;
  __syncthreads();
  for (int o = 1; o < 256; o <<= 1) {
    const int v = tid >= o ? scan[tid - o] : 0;
    __syncthreads();
    scan[tid] += v;
    __syncthreads();
  }
  int off = scan[tid] - mine;
  for (int s = s0; s < s1; ++s) {
    const int2 r = chunk_rows(cu, s, total_q);
    const int nt = (r.y - r.x + rows_per_tile - 1) / rows_per_tile;
    for (int k = 0; k < nt; ++k) {
      if (off < max_tiles) tiles[off] = make_int2(s, (nt - 1 - k) * rows_per_tile);
      ++off;
    }
  }
  if (tid == 255) *count = min(scan[255], max_tiles);
}

template <int G, bool kPow2Blocks>
__global__ __attribute__((amdgpu_flat_work_group_size(kThreads, kThreads),
                          amdgpu_waves_per_eu(2, 2)))
void prefill_kernel(const uint16_t* __restrict__ q, const uint8_t* __restrict__ kv,
                    int num_blocks, const int* __restrict__ block_table,
                    const int* __restrict__ seq_lens, const int* __restrict__ cu,
                    uint16_t* __restrict__ out, const int2* __restrict__ tiles,
                    const int* __restrict__ tile_count, int total_q, int num_q_heads,
                    int num_kv_heads,
                    int max_blocks, int max_seq_len, float scale_log2) {
  constexpr int kRows = 32 * kWaves / G;   // rows per work tile
  const int wid = blockIdx.x;
  const int g = wid % num_kv_heads;
  const int ti = wid / num_kv_heads;
  if (ti >= *tile_count) return;
  const int2 tl = tiles[ti];
  const int s = tl.x;
  const int q0 = tl.y;
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);  // uniform per wavefront
  const int lane = tid % kWave;
  const int h = g * G + wave % G;
  const int row0 = q0 + (wave / G) * 32;        // first row of this wave
  const int2 rows = chunk_rows(cu, s, total_q);
  const int cu0 = rows.x;
  const int n = rows.y - rows.x;
  int L = seq_lens[s];
  L = __builtin_amdgcn_readfirstlane(min(max(L, 0), min(max_seq_len, max_blocks * kBS)));
  const int c = L - n;                          // cached context before the chunk
  const int wg_rows = min(kRows, n - q0);
  const int last_pos = min(c + q0 + wg_rows - 1, L - 1);
  const int N = last_pos >= 0 ? last_pos / kKeys + 1 : 0;   // steps of the tile
  const bool idle = row0 >= n;                  // none of the wave's 32 rows is in the chunk

  __shared__ __attribute__((aligned(16))) uint8_t lds_k[kKBufs][kStepBlocks][kTileBytes];
  __shared__ __attribute__((aligned(16))) uint8_t lds_v[kVBufs][kStepBlocks][kTileBytes];

  const size_t block_bytes = 2 * (size_t)num_kv_heads * kTileBytes;
  // log2 of the block size when it is a power of two (a shift replaces the
  // 64-bit multiply in every gather's address)
  const int block_shift = kPow2Blocks ? __builtin_ctzll(block_bytes) : 0;
  const size_t k_off = (size_t)g * kTileBytes;
  const size_t v_off = (size_t)(num_kv_heads + g) * kTileBytes;
  const int* bt = block_table + (size_t)s * max_blocks;
  const int qstride = num_q_heads * kD;

  const int lm = lane % 32;     // MFMA row / column index of this lane
  const int lh = lane / 32;     // which 8-wide half of the 16-wide k slice
  // Key permutation of the S^T rows: A row m = 8a + 4b + e holds key
  // 16 (a / 2) + 8 b + 4 (a % 2) + e of the 32-key tile, so accumulator
  // element i of lane l is key 16 (i / 8) + 8 (l / 32) + i % 8.
  const int ka = lm / 8, kb4 = (lm / 4) % 2, ke = lm % 4;
  const int k_blk = ka / 2;                              // block within the key tile
  const int k_slot = 8 * kb4 + 4 * (ka % 2) + ke;        // slot within the block

  // ---- Q^T operand of the wave's 32 rows, loaded once into registers ----
  // Lane (lm, lh) of k-step ks holds dims ks * 16 + lh * 8 .. + 8 of row
  // row0 + lm; rows past the chunk read the chunk's last row (never written).
  bf16x8_t qr[8];
  if (!idle) {
    const int row = min(row0 + lm, n - 1);
    const uint16_t* qrow = q + (size_t)(cu0 + row) * qstride + (size_t)h * kD + lh * 8;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks)
      qr[ks] = *reinterpret_cast<const bf16x8_t*>(qrow + ks * 16);
  }

  f32x16_t oacc[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int i = 0; i < 16; ++i) oacc[dt][i] = 0.f;
  float m_ref = -INFINITY;   // reference max of the lane's row (log2 domain)
  float l_run = 0.f;         // lane-partial row sum

  // ---- gather of K or V of one 64-key step straight into LDS (global_load_lds) ----
  // The block ids of a step are read from the table first (step_ids), in
  // SGPRs: one 16-byte scalar load when all 4 blocks lie inside the sequence,
  // single entries otherwise; a block past L or with an id outside
  // [0, num_blocks) gets id -1. The bit mask of a step (bit kb: block kb is
  // real) lets the softmax mask its keys and patch_v zero its values.
  const int nblk = (L + kBS - 1) / kBS;   // table entries the sequence uses
  struct StepIds {
    int id[kStepBlocks];
  };
  auto step_ids = [&](int step) __attribute__((always_inline)) {
    StepIds r;
    const int b0 = step * kStepBlocks;
    if (b0 + kStepBlocks <= nblk) {
      const i32x4_t v = scalar_entries4(bt, b0);
#pragma unroll
      for (int kb = 0; kb < kStepBlocks; ++kb) r.id[kb] = v[kb];
    } else {
#pragma unroll
      for (int kb = 0; kb < kStepBlocks; ++kb)
        r.id[kb] = b0 + kb < nblk ? scalar_entry(bt, b0 + kb) : -1;
    }
    return r;
  };
  // Ids are checked against the layer only where they are used, so that
  // nothing waits for the loads where they are issued.
  auto real_id = [&](int id) __attribute__((always_inline)) {
    return (unsigned)id < (unsigned)num_blocks;
  };
  auto id_bits = [&](const StepIds& r) __attribute__((always_inline)) {
    int bits = 0;
#pragma unroll
    for (int kb = 0; kb < kStepBlocks; ++kb) bits |= real_id(r.id[kb]) ? (1 << kb) : 0;
    return bits;
  };
  // The gather itself: a half step is 4 tiles of 4 KiB (blocks 0..3); in
  // round j wavefront w fills quarter (w + 8 j) % 4 of tile (w + 8 j) / 4, a
  // contiguous 1 KiB with 16 bytes per lane. K is copied as stored; for V the
  // lane picks the global 16 bytes that belong at its swizzled LDS position
  // (row pos / 2, half pos % 2 holds global half (pos % 2) ^ ((row >> 3) & 1)).
  // A block that is not real is read from block 0 instead (the host
  // guarantees one exists) and masked afterwards.
  auto gather = [&](auto v_tag, int step, const StepIds& ids) __attribute__((always_inline)) {
    constexpr bool kV = decltype(v_tag)::value;
    // The lane id is recomputed here rather than kept live across the step.
    const int ln = lane_id_fresh();
    const uint8_t* base[2];
    uint32_t off[2], lds[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int kb = (wave + kWaves * j) / 4;     // wave-uniform
      const int quarter = (wave + kWaves * j) % 4;
      // kb is wave / 4 + 2 j: pick the id by a uniform select, not an index
      const int id = wave < 4 ? ids.id[2 * j] : ids.id[2 * j + 1];
      const size_t id0 = real_id(id) ? (size_t)(unsigned)id : 0;
      base[j] = kv + (kPow2Blocks ? id0 << block_shift : id0 * block_bytes) + (kV ? v_off : k_off);
      const unsigned pos = quarter * kWave + (unsigned)ln;   // 16-byte position in the tile
      if constexpr (kV) {
        const unsigned vrow = pos / 2;
        off[j] = vrow * 32 + (((pos % 2) ^ ((vrow >> 3) & 1)) * 16);
        lds[j] = __builtin_amdgcn_readfirstlane(
            lds_addr(&lds_v[step % kVBufs][kb][quarter * 1024]));
      } else {
        off[j] = pos * 16;
        lds[j] = __builtin_amdgcn_readfirstlane(
            lds_addr(&lds_k[step % kKBufs][kb][quarter * 1024]));
      }
    }
    dma16x2(base[0], off[0], lds[0], base[1], off[1], lds[1]);
  };
  auto load_half = [&](auto v_tag, int step) __attribute__((always_inline)) {
    const StepIds ids = step_ids(step);
    gather(v_tag, step, ids);
    return id_bits(ids);
  };
  // Zero the V slots of a landed step that must not contribute: blocks that
  // are not real, and slots at or past L (their bytes may be NaN, and a zero
  // weight times NaN is NaN). Every wavefront patches the whole step right
  // before its own p.v reads it: the writes of different wavefronts are
  // identical and idempotent, so no barrier is needed between them. Called
  // only when such slots exist.
  auto patch_v = [&](int step, int bits) __attribute__((always_inline)) {
    const int kbase = step * kKeys;
    // recomputed here, so no lane constant of this rare path stays live
    // across the pipelined loop
    const int ln = lane_id_fresh();
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const int cidx = ln + kWave * j;            // 16-byte chunk of the 4 V tiles
      const int kb = cidx / 256;
      const int pos = cidx % 256;
      const int vrow = pos / 2;
      const int half_g = (pos % 2) ^ ((vrow >> 3) & 1);
      uint4* v = reinterpret_cast<uint4*>(&lds_v[step % kVBufs][kb][pos * 16]);
      if (!((bits >> kb) & 1)) {
        *v = make_uint4(0, 0, 0, 0);
        continue;
      }
      const int key = kbase + kb * kBS + 8 * half_g;
      if (key + 8 <= L) continue;
      uint4 w4 = *v;
      uint32_t w[4] = {w4.x, w4.y, w4.z, w4.w};
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const uint32_t lo = (key + 2 * k < L) ? 0x0000ffffu : 0u;
        const uint32_t hi = (key + 2 * k + 1 < L) ? 0xffff0000u : 0u;
        w[k] &= (lo | hi);
      }
      *v = make_uint4(w[0], w[1], w[2], w[3]);
    }
  };
  auto step_clean = [&](int step, int bits) __attribute__((always_inline)) { return bits == 0xf && (step + 1) * kKeys <= L; };

  const int wave_pos0 = c + row0;   // position of the wave's first row
  const int v_read = lm * 32 + ((lh ^ ((lm >> 3) & 1)) * 16);

  // S^T for one step: 2 key tiles x 8 k-steps of 16 dims.
  auto qk = [&](int step, f32x16_t (&sa)[2]) {
    const int buf = step % kKBufs;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int i = 0; i < 16; ++i) sa[kt][i] = 0.f;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) {
      const bf16x8_t b = qr[ks];
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        const int chunk = 2 * ks + lh;
        const bf16x8_t a = *reinterpret_cast<const bf16x8_t*>(
            &lds_k[buf][2 * kt + k_blk][(chunk * kBS + k_slot) * 16]);
        sa[kt] = mfma32(a, b, sa[kt]);
      }
    }
  };
  // O^T += V^T P^T for one step: one k-step per block, 4 accumulator chains.
  // Used once per tile, after the pipelined loop; the fence after each block
  // keeps the compiler from hoisting all 16 operand reads at once, which
  // would need more registers than the kernel has left.
  auto pv = [&](int step, const bf16x8_t (&pr)[4]) {
    const int buf = step % kVBufs;
#pragma unroll
    for (int kb = 0; kb < kStepBlocks; ++kb) {
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) {
        const bf16x8_t a =
            *reinterpret_cast<const bf16x8_t*>(&lds_v[buf][kb][dt * 32 * 32 + v_read]);
        oacc[dt] = mfma32(a, pr[kb], oacc[dt]);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  // Causal / length / real-block mask of one step's scores, in place; run
  // only on the steps that need it.
  auto mask_scores = [&](int step, int bits, f32x16_t (&sr)[2]) {
    const int kbase = step * kKeys;
    const int ln = lane_id_fresh();   // as in patch_v
    const int qpos = wave_pos0 + ln % 32;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int kpos = kbase + kt * 32 + (i / 8) * 16 + (ln / 32) * 8 + (i % 8);
        const int blk_ok = (bits >> (2 * kt + i / 8)) & 1;
        const int keep = (kpos <= qpos) & (kpos < L) & blk_ok;
        sr[kt][i] = keep ? sr[kt][i] : -INFINITY;
      }
  };
  auto needs_mask = [&](int step, int bits) __attribute__((always_inline)) {
    return (step * kKeys + kKeys - 1 > wave_pos0) || !step_clean(step, bits);
  };
  // bitsm1, bits0 .. bits3: real-block masks of steps i - 1, i .. i + 3
  int bitsm1 = 0, bits0 = 0, bits1 = 0, bits2 = 0, bits3 = 0;
  // block ids of the gathers of the coming phase: K of step i + 3 and V of
  // step i + 1, read at the end of the phase before (ahead of its barrier)
  StepIds idsK, idsV;
  f32x16_t sA[2], sB[2];    // scores of even / odd steps
  bf16x8_t pA[4], pB[4];    // P of even / odd steps

  // One pipeline step i: the matrix work (p.v of step i - 1, q.k of step
  // i + 1) next to the softmax of step i, with the gathers of K of step i + 3
  // and V of step i + 1 in between. The step ends by waiting for the gathers
  // of the earlier steps only (those of this step get the whole next step to
  // land) and a barrier;
  // then O takes the rescale of step i's softmax, between the p.v of steps
  // i - 1 and i.
  //
  // The matrix and softmax work is laid out by hand in 32 issue slots: slot
  // k issues matrix instruction k (p.v for k < 16, q.k after), the LDS read
  // of the operand five slots ahead, and one exponential with its share of
  // the row sum and bf16 packing. A wavefront issues in order, so without
  // this the vector work would queue behind runs of matrix instructions
  // instead of running beside them. The gathers' branches split the slots
  // into three blocks, and the compiler gathers most exponentials of a block
  // into one run, so some slots issue their matrix instructions back to back.
  // Holding the exponentials in their slots measured slower, and so did
  // either strict order of the step's two halves (all matrix work first, or
  // all softmax first). The row max, when a step needs it, follows the slots.
  auto phase = [&](auto qk_tag, auto pv_tag, int i, f32x16_t (&s_cur)[2],
                   f32x16_t (&s_nxt)[2], const bf16x8_t (&p_prev)[4], bf16x8_t (&p_cur)[4]) __attribute__((always_inline)) {
    constexpr bool kQK = decltype(qk_tag)::value;
    constexpr bool kPV = decltype(pv_tag)::value;
    // The block ids were read before the barrier that ends the previous
    // phase: wait for them here, while no operand read of this phase is in
    // flight, so that the operand prefetch below is never drained for them
    // (scalar loads share the lgkm counter with LDS reads and return out of
    // order).
    __builtin_amdgcn_s_waitcnt(0xc07f);   // lgkmcnt(0)
    if (kPV && !step_clean(i - 1, bitsm1)) patch_v(i - 1, bitsm1);
    const bool do_k = i + 3 < N, do_v = i + 1 < N;
    if (needs_mask(i, bits0)) mask_scores(i, bits0, s_cur);

    const int vbuf = (i + kVBufs - 1) % kVBufs;   // V of step i - 1
    const int kbuf = (i + 1) % kKBufs;            // K of step i + 1
    auto has_mfma = [&](int k) __attribute__((always_inline)) { return k < 16 ? kPV : kQK; };
    auto a_frag = [&](int k) __attribute__((always_inline)) {
      if (k < 16)
        return *reinterpret_cast<const bf16x8_t*>(
            &lds_v[vbuf][k / 4][(k % 4) * 32 * 32 + v_read]);
      const int ks = (k - 16) / 2, kt = (k - 16) % 2;
      return *reinterpret_cast<const bf16x8_t*>(
          &lds_k[kbuf][2 * kt + k_blk][((2 * ks + lh) * kBS + k_slot) * 16]);
    };
    constexpr int kAhead = kQK ? 5 : 3;   // the last step keeps fewer reads in flight
    bf16x8_t fr[kAhead + 1];
#pragma unroll
    for (int k = 0; k < kAhead; ++k) {
      if (has_mfma(k)) fr[k % (kAhead + 1)] = a_frag(k);
    }
    float ref = (m_ref == -INFINITY) ? 0.f : m_ref, alpha = 1.f, psum = 0.f;
    bool rescale = false;
    float pe[32];
    uint32_t pw[16];
    f32x16_t zero;
#pragma unroll
    for (int e = 0; e < 16; ++e) zero[e] = 0.f;
    // Raised issue priority while this wavefront issues its matrix slots, so
    // that the arbiter prefers its MFMAs and operand reads over the vector
    // work of the other wavefront of the SIMD (0.5-0.9% faster, same-box A/B).
    __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int k = 0; k < 32; ++k) {
      // operand reads for slot k + kAhead
      const int kn = k + kAhead;
      if (kn < 32 && has_mfma(kn)) fr[kn % (kAhead + 1)] = a_frag(kn);
      // matrix instruction k
      if (k < 16) {
        if (kPV) oacc[k % 4] = mfma32(fr[k % (kAhead + 1)], p_prev[k / 4], oacc[k % 4]);
      } else if (kQK) {
        const int ks = (k - 16) / 2, kt = (k - 16) % 2;
        s_nxt[kt] = mfma32(fr[k % (kAhead + 1)], qr[ks], ks == 0 ? zero : s_nxt[kt]);
      }
      // softmax share of slot k: the exponential of score k against the
      // current reference
      {
        const int e = k;
        pe[e] = fast_exp2(fmaf(s_cur[e / 16][e % 16], scale_log2, -ref));
        if (e % 2 == 1) {
          // the row sum adds the bf16 values that p.v multiplies
          pw[e / 2] = pack_bf16x2(pe[e - 1], pe[e]);
          psum = dot2_bf16(pw[e / 2], kBf16OnePair, psum);
        }
      }
      // the step's gathers, issued inside the schedule (K in slot 10, V in
      // slot 26) so that their LDS writes do not land in one burst
      if (k == 10 && do_k) {
        gather(std::false_type{}, i + 3, idsK);
        bits3 = id_bits(idsK);
      }
      if (k == 26 && do_v) gather(std::true_type{}, i + 1, idsV);
      __builtin_amdgcn_sched_barrier(0);
    }
    __builtin_amdgcn_s_setprio(0);
    // A row without a reference yet, or a lane whose partial row sum (which
    // bounds each of its exponentials) left 2^8: take the exact row max, move
    // the reference of the rows that outgrew theirs by more than 2^8, and
    // redo the step's exponentials against it. Rows that did not outgrow
    // theirs get the same values again.
    if (__builtin_amdgcn_ballot_w64(m_ref == -INFINITY || !(psum <= kPsumBound)) != 0) {
      float mp0 = -INFINITY, mp1 = -INFINITY;
#pragma unroll
      for (int e = 0; e < 32; e += 4) {
        mp0 = max3f(mp0, s_cur[e / 16][e % 16], s_cur[e / 16][e % 16 + 1]);
        mp1 = max3f(mp1, s_cur[e / 16][e % 16 + 2], s_cur[e / 16][e % 16 + 3]);
      }
      float mx = max3f(mp0, mp1, mp1);
      mx = max3f(mx, __shfl_xor(mx, 32, kWave), mx);
      const float tmax = mx * scale_log2;
      const bool grow = tmax > m_ref + kLazyRescale;
      rescale = __builtin_amdgcn_ballot_w64(grow) != 0;
      const float nref = grow ? tmax : m_ref;
      alpha = (m_ref == -INFINITY) ? 0.f : fast_exp2(m_ref - nref);
      m_ref = nref;
      ref = (nref == -INFINITY) ? 0.f : nref;
      psum = 0.f;
#pragma unroll
      for (int e = 0; e < 32; e += 2) {
        pw[e / 2] = pack_bf16x2(fast_exp2(fmaf(s_cur[e / 16][e % 16], scale_log2, -ref)),
                                fast_exp2(fmaf(s_cur[e / 16][e % 16 + 1], scale_log2, -ref)));
        psum = dot2_bf16(pw[e / 2], kBf16OnePair, psum);
      }
    }
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
      p_cur[kb] = __builtin_bit_cast(
          bf16x8_t, make_uint4(pw[4 * kb], pw[4 * kb + 1], pw[4 * kb + 2], pw[4 * kb + 3]));
    l_run = l_run * alpha + psum;
    // keep the softmax in its slots (the compiler would otherwise sink it
    // next to its first use, away from the matrix work it should overlap)
#pragma unroll
    for (int k = 0; k < 4; ++k) asm volatile("" ::"v"(p_cur[k]));
    asm volatile("" ::"v"(l_run));
    // the block ids of the next phase's gathers
    if (i + 4 < N) idsK = step_ids(i + 4);
    if (i + 2 < N) idsV = step_ids(i + 2);
    // wait for the gathers of steps before this one (each thread issued two
    // for K when i + 3 < N and two for V when i + 1 < N in this step)
    if (i + 3 < N)
      asm volatile("s_waitcnt vmcnt(4)" ::: "memory");
    else if (i + 1 < N)
      asm volatile("s_waitcnt vmcnt(2)" ::: "memory");
    else
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (rescale) {
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) oacc[dt] *= alpha;
    }
    bitsm1 = bits0;
    bits0 = bits1;
    bits1 = bits2;
    bits2 = bits3;
  };

  // A wavefront none of whose rows lies in the chunk (a short chunk's last
  // tile, a one-row decode sequence in a unified batch) still takes its share
  // of every gather and meets every barrier, step for step like the others,
  // but does no matrix or softmax work and writes nothing.
  if (idle) {
    if (N > 0) {
      load_half(std::false_type{}, 0);
      if (N > 1) load_half(std::false_type{}, 1);
      if (N > 2) load_half(std::false_type{}, 2);
      load_half(std::true_type{}, 0);
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      __syncthreads();
      __syncthreads();   // the others' q.k of step 0
      for (int i = 0; i < N; ++i) {
        if (i + 3 < N) load_half(std::false_type{}, i + 3);
        if (i + 1 < N) load_half(std::true_type{}, i + 1);
        if (i + 3 < N)
          asm volatile("s_waitcnt vmcnt(4)" ::: "memory");
        else if (i + 1 < N)
          asm volatile("s_waitcnt vmcnt(2)" ::: "memory");
        else
          asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
      }
    }
    return;
  }

  if (N > 0) {
    bits0 = load_half(std::false_type{}, 0);
    if (N > 1) bits1 = load_half(std::false_type{}, 1);
    if (N > 2) bits2 = load_half(std::false_type{}, 2);
    load_half(std::true_type{}, 0);
    if (N > 3) idsK = step_ids(3);
    if (N > 1) idsV = step_ids(1);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    qk(0, sA);
    __syncthreads();   // K of step 0 is read; step 0 of the pipeline gathers step 3 into its buffer
    constexpr std::true_type T{};
    constexpr std::false_type F{};
    if (N > 1)
      phase(T, F, 0, sA, sB, pB, pA);
    else
      phase(F, F, 0, sA, sB, pB, pA);
    int i = 1;
    for (; i + 1 <= N - 2; i += 2) {
      phase(T, T, i, sB, sA, pA, pB);
      phase(T, T, i + 1, sA, sB, pB, pA);
    }
    if (i <= N - 2) {
      phase(T, T, i, sB, sA, pA, pB);
      ++i;
    }
    // p.v of the last step (its V landed by the last step's full wait)
    if (N > 1) {
      if (i & 1)
        phase(F, T, i, sB, sA, pA, pB);
      else
        phase(F, T, i, sA, sB, pB, pA);
    }
    if (!step_clean(N - 1, bitsm1)) patch_v(N - 1, bitsm1);
    pv(N - 1, ((N - 1) & 1) ? pB : pA);
  }

  // ---- normalise and write O (this lane: row lm) ----
  {
    const float lt = l_run + __shfl_xor(l_run, 32, kWave);
    const float inv = lt > 0.f ? 1.f / lt : 0.f;
    const int r = row0 + lm;
    if (r < n) {
      uint16_t* orow = out + (size_t)(cu0 + r) * qstride + (size_t)h * kD;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) {
#pragma unroll
        for (int a = 0; a < 4; ++a) {
          const f32x16_t& o = oacc[dt];
          const uint2 w = make_uint2(pack_bf16x2(o[4 * a + 0] * inv, o[4 * a + 1] * inv),
                                     pack_bf16x2(o[4 * a + 2] * inv, o[4 * a + 3] * inv));
          *reinterpret_cast<uint2*>(orow + dt * 32 + a * 8 + lh * 4) = w;
        }
      }
    }
  }
}

template <int G>
static hipError_t launch_prefill_t(const PrefillArgs& a) {
  constexpr int kRowsPerTile = 32 * kWaves / G;
  int* count = reinterpret_cast<int*>(a.workspace);
  int2* tiles = reinterpret_cast<int2*>(static_cast<uint8_t*>(a.workspace) + 16);
  const int max_tiles =
      static_cast<int>((a.workspace_bytes - 16) / sizeof(int2));
  const long long bound = (long long)a.total_q_tokens / kRowsPerTile + a.num_seqs;
  const int grid_tiles = (int)(bound < max_tiles ? bound : max_tiles);
  trace_before(a.stream, "prefill_tile_map");
  hipLaunchKernelGGL(prefill_tile_map_kernel, dim3(1), dim3(256), 0, a.stream, a.cu_seqlens_q,
                     a.num_seqs, a.total_q_tokens, kRowsPerTile, tiles, count, grid_tiles);
  trace_after(a.stream);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const long long blocks = (long long)grid_tiles * a.num_kv_heads;
  if (blocks <= 0) return hipSuccess;
  if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
  trace_before(a.stream, "prefill");
  const unsigned kvh = (unsigned)a.num_kv_heads;
  auto kernel = (kvh & (kvh - 1)) == 0 ? prefill_kernel<G, true> : prefill_kernel<G, false>;
  hipLaunchKernelGGL(kernel, dim3((unsigned)blocks), dim3(kThreads), 0, a.stream,
                     static_cast<const uint16_t*>(a.q), static_cast<const uint8_t*>(a.kv),
                     a.num_blocks, a.block_table, a.seq_lens, a.cu_seqlens_q,
                     static_cast<uint16_t*>(a.out), tiles, count, a.total_q_tokens,
                     a.num_q_heads, a.num_kv_heads, a.max_blocks, a.max_seq_len,
                     a.scale * kLog2e);
  trace_after(a.stream);
  return hipGetLastError();
}

hipError_t launch_prefill(const PrefillArgs& a) {
  if (a.head_dim != kD) return hipErrorNotSupported;
  switch (a.num_q_heads / a.num_kv_heads) {
    case 1: return launch_prefill_t<1>(a);
    case 2: return launch_prefill_t<2>(a);
    case 4: return launch_prefill_t<4>(a);
    case 8: return launch_prefill_t<8>(a);
    default: return hipErrorNotSupported;
  }
}

}  // namespace kvattn
