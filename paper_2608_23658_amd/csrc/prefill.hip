// Chunked-prefill attention for gfx950 on bf16 MFMA (the paper, Section 5:
// prefill is compute bound and a chunk attends to all earlier context, so
// chunking splits the same work; Section 1: max_num_batched_tokens bounds
// the chunk).
//
// Work tile = (kv head g, 64 * 4 / G consecutive new rows of one sequence).
// A workgroup of 4 wavefronts owns one tile: wave w serves query head
// g * G + w % G over 64 rows (two row tiles of 32). K/V steps of 64 keys (4
// blocks) are gathered through the block table into double-buffered LDS once
// per workgroup and shared by the G query heads of the group.
//
// Per wave and step, with v_mfma_f32_32x32x16_bf16 (four independent
// accumulator chains are enough to keep it busy, where the 16x16x32 form
// needs sixteen):
//   S^T[key][row] = K[key][:] . Q[row][:]   A = K rows read from the
//       chunk-major K tile, B = Q^T held in registers for the whole kernel.
//       The A rows of a 32-key tile are loaded in a permuted key order so
//       that the accumulator of each lane ends up holding 8 consecutive keys
//       of each of the two blocks for one query row;
//   softmax over keys in the log2 domain: a row's 64 scores live in two
//       lanes (l and l + 32), so the row max needs one exchange; the row
//       state is lane-local. The running max is only moved, and O^T and the
//       row sum rescaled, when a row's max grows by more than 2^8: the
//       exponentials stay below 256, which bf16 P and fp32 accumulation hold;
//   O^T[d][row] += V^T[d][key] P^T[key][row]   A = 16-byte runs of the
//       dim-major V tile, B = the bf16 P values of 8 consecutive keys of one
//       block, already in the lane that produced them.
// V rows are stored in LDS with their two 16-byte halves swapped on every
// other group of 8 rows, so the A reads of 16 rows hit 16 distinct bank
// groups. The causal mask (bottom-right: row i at position L - n + i sees
// keys 0 .. L - n + i) is applied only on steps that reach the diagonal or
// the end of the sequence.

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

typedef float f32x16_t __attribute__((ext_vector_type(16)));

__device__ __forceinline__ f32x16_t mfma32(bf16x8_t a, bf16x8_t b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

}  // namespace

// Lists the work tiles (sequence, first row) of a batch of chunks, the rows
// of a sequence's chunk in descending order so the longest rows start first.
__global__ __launch_bounds__(256) void prefill_tile_map_kernel(const int* __restrict__ cu,
                                                               int num_seqs, int rows_per_tile,
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
    const int n = max(0, cu[s + 1] - cu[s]);
    mine += (n + rows_per_tile - 1) / rows_per_tile;
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
    const int n = max(0, cu[s + 1] - cu[s]);
    const int nt = (n + rows_per_tile - 1) / rows_per_tile;
    for (int k = 0; k < nt; ++k) {
      if (off < max_tiles) tiles[off] = make_int2(s, (nt - 1 - k) * rows_per_tile);
      ++off;
    }
  }
  if (tid == 255) *count = min(scan[255], max_tiles);
}

template <int G>
__global__ __attribute__((amdgpu_flat_work_group_size(256, 256), amdgpu_waves_per_eu(1, 1)))
void prefill_kernel(const uint16_t* __restrict__ q, const uint8_t* __restrict__ kv,
                    int num_blocks, const int* __restrict__ block_table,
                    const int* __restrict__ seq_lens, const int* __restrict__ cu,
                    uint16_t* __restrict__ out, const int2* __restrict__ tiles,
                    const int* __restrict__ tile_count, int num_q_heads, int num_kv_heads,
                    int max_blocks, int max_seq_len, float scale_log2) {
  constexpr int kRows = 64 * 4 / G;      // rows per work tile
  const int wid = blockIdx.x;
  const int g = wid % num_kv_heads;
  const int ti = wid / num_kv_heads;
  if (ti >= *tile_count) return;
  const int2 tl = tiles[ti];
  const int s = tl.x;
  const int q0 = tl.y;
  const int tid = threadIdx.x;
  const int wave = tid / kWave;
  const int lane = tid % kWave;
  const int h = g * G + wave % G;
  const int row0 = q0 + (wave / G) * 64;        // first row of this wave
  const int cu0 = cu[s];
  const int n = cu[s + 1] - cu0;
  int L = seq_lens[s];
  L = min(max(L, 0), min(max_seq_len, max_blocks * kBS));
  const int c = L - n;                          // cached context before the chunk
  const int wg_rows = min(kRows, n - q0);
  const int last_pos = min(c + q0 + wg_rows - 1, L - 1);
  const int nsteps = last_pos >= 0 ? last_pos / kKeys + 1 : 0;

  __shared__ __attribute__((aligned(16))) uint8_t lds[2][2][kStepBlocks][kTileBytes];

  const size_t block_bytes = 2 * (size_t)num_kv_heads * kTileBytes;
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

  // ---- Q^T operands for the wave's 64 rows (2 row tiles of 32) ----
  bf16x8_t qb[2][8];
#pragma unroll
  for (int rt = 0; rt < 2; ++rt) {
    const int r = row0 + rt * 32 + lm;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) {
      uint4 v = make_uint4(0, 0, 0, 0);
      if (r < n)
        v = *reinterpret_cast<const uint4*>(q + (size_t)(cu0 + r) * qstride + (size_t)h * kD +
                                           ks * 16 + lh * 8);
      qb[rt][ks] = __builtin_bit_cast(bf16x8_t, v);
    }
  }

  f32x16_t oacc[4][2];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int rt = 0; rt < 2; ++rt)
#pragma unroll
      for (int i = 0; i < 16; ++i) oacc[dt][rt][i] = 0.f;
  float m_ref[2] = {-INFINITY, -INFINITY};   // reference max of each row (log2 domain)
  float l_run[2] = {0.f, 0.f};               // lane-partial row sums

  // ---- gather of one 64-key step into registers: 8 x 16 bytes per thread ----
  uint4 pre[2 * kStepBlocks];
  auto load_step = [&](int step) {
    const int kbase = step * kKeys;
#pragma unroll
    for (int kb = 0; kb < kStepBlocks; ++kb) {
      const int key0 = kbase + kb * kBS;
      int id = -1;
      if (key0 < L) {
        id = bt[key0 / kBS];
        if ((unsigned)id >= (unsigned)num_blocks) id = -1;
      }
      if (id >= 0) {
        const uint8_t* base = kv + (size_t)id * block_bytes + tid * 16;
        pre[kb * 2 + 0] = *reinterpret_cast<const uint4*>(base + k_off);
        pre[kb * 2 + 1] = *reinterpret_cast<const uint4*>(base + v_off);
      } else {
        pre[kb * 2 + 0] = make_uint4(0, 0, 0, 0);
        pre[kb * 2 + 1] = make_uint4(0, 0, 0, 0);
      }
    }
  };
  // V dim row tid / 2, half tid % 2 (slots 8 * (tid % 2) .. + 7); stored at
  // the swizzled half. Slots at or past L are zeroed (their bytes may be NaN).
  const int vrow = tid / 2, vhalf = tid % 2;
  const int v_lds = vrow * 32 + ((vhalf ^ ((vrow >> 3) & 1)) * 16);
  auto store_step = [&](int buf, int step) {
    const int kbase = step * kKeys;
    const bool tail = kbase + kKeys > L;
#pragma unroll
    for (int kb = 0; kb < kStepBlocks; ++kb) {
      uint4 v = pre[kb * 2 + 1];
      if (tail) {
        const int key = kbase + kb * kBS + 8 * vhalf;
        uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const uint32_t lo = (key + 2 * k < L) ? 0x0000ffffu : 0u;
          const uint32_t hi = (key + 2 * k + 1 < L) ? 0xffff0000u : 0u;
          w[k] &= (lo | hi);
        }
        v = make_uint4(w[0], w[1], w[2], w[3]);
      }
      *reinterpret_cast<uint4*>(&lds[buf][0][kb][tid * 16]) = pre[kb * 2 + 0];
      *reinterpret_cast<uint4*>(&lds[buf][1][kb][v_lds]) = v;
    }
  };

  if (nsteps > 0) {
    load_step(0);
    store_step(0, 0);
  }
  __syncthreads();

  const int wave_pos0 = c + row0;   // position of the wave's first row
  const int v_read = lm * 32 + ((lh ^ ((lm >> 3) & 1)) * 16);
  for (int step = 0; step < nsteps; ++step) {
    const int buf = step & 1;
    if (step + 1 < nsteps) load_step(step + 1);
    const int kbase = step * kKeys;

    // ---- S^T = K Q^T: 2 key tiles x 2 row tiles, 8 k-steps of 16 dims ----
    f32x16_t sacc[2][2];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int rt = 0; rt < 2; ++rt)
#pragma unroll
        for (int i = 0; i < 16; ++i) sacc[kt][rt][i] = 0.f;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) {
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        const int chunk = 2 * ks + lh;
        const bf16x8_t a = *reinterpret_cast<const bf16x8_t*>(
            &lds[buf][0][2 * kt + k_blk][(chunk * kBS + k_slot) * 16]);
#pragma unroll
        for (int rt = 0; rt < 2; ++rt) sacc[kt][rt] = mfma32(a, qb[rt][ks], sacc[kt][rt]);
      }
    }

    // ---- online softmax per row (lane holds row lm of each row tile) ----
    if ((kbase + kKeys - 1 > wave_pos0) || (kbase + kKeys > L)) {
      // causal / length mask, only on steps that reach the diagonal or the end
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int rt = 0; rt < 2; ++rt)
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            const int kpos = kbase + kt * 32 + (i / 8) * 16 + lh * 8 + (i % 8);
            const int qpos = wave_pos0 + rt * 32 + lm;
            if (kpos > qpos || kpos >= L) sacc[kt][rt][i] = -INFINITY;
          }
    }
    bf16x8_t pb[2][4];
    float alpha[2];
    float tmax[2];
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
      float mx = -INFINITY;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int i = 0; i < 16; ++i) mx = fmaxf(mx, sacc[kt][rt][i]);
      mx = fmaxf(mx, __shfl_xor(mx, 32, kWave));
      tmax[rt] = mx * scale_log2;
    }
    // Move a row's reference max only when its scores outgrow it by 2^8.
    const bool grow0 = tmax[0] > m_ref[0] + kLazyRescale;
    const bool grow1 = tmax[1] > m_ref[1] + kLazyRescale;
    const bool rescale = __builtin_amdgcn_ballot_w64(grow0 || grow1) != 0;
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
      const bool grow = rt == 0 ? grow0 : grow1;
      const float nref = grow ? tmax[rt] : m_ref[rt];
      alpha[rt] = (m_ref[rt] == -INFINITY) ? 0.f : fast_exp2(m_ref[rt] - nref);
      m_ref[rt] = nref;
      const float ref = (nref == -INFINITY) ? 0.f : nref;
      float psum = 0.f;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        float p[16];
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          p[i] = fast_exp2(fmaf(sacc[kt][rt][i], scale_log2, -ref));
          psum += p[i];
        }
#pragma unroll
        for (int half = 0; half < 2; ++half) {
          const uint4 w = make_uint4(pack_bf16x2(p[8 * half + 0], p[8 * half + 1]),
                                     pack_bf16x2(p[8 * half + 2], p[8 * half + 3]),
                                     pack_bf16x2(p[8 * half + 4], p[8 * half + 5]),
                                     pack_bf16x2(p[8 * half + 6], p[8 * half + 7]));
          pb[rt][2 * kt + half] = __builtin_bit_cast(bf16x8_t, w);
        }
      }
      l_run[rt] = l_run[rt] * alpha[rt] + psum;
    }

    // ---- O^T += V^T P^T: 4 dim tiles x 2 row tiles, one k-step per block ----
    // (the rescale of O^T, when a row max moved, is folded in one 16-value
    // accumulator at a time)
#pragma unroll
    for (int kb = 0; kb < kStepBlocks; ++kb) {
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) {
        const bf16x8_t a =
            *reinterpret_cast<const bf16x8_t*>(&lds[buf][1][kb][dt * 32 * 32 + v_read]);
#pragma unroll
        for (int rt = 0; rt < 2; ++rt) {
          if (kb == 0 && rescale) oacc[dt][rt] *= alpha[rt];
          oacc[dt][rt] = mfma32(a, pb[rt][kb], oacc[dt][rt]);
        }
      }
    }

    if (step + 1 < nsteps) store_step(buf ^ 1, step + 1);
    __syncthreads();
  }

  // ---- normalise and write O (this lane: row lm of each row tile) ----
#pragma unroll
  for (int rt = 0; rt < 2; ++rt) {
    float lt = l_run[rt] + __shfl_xor(l_run[rt], 32, kWave);
    const float inv = lt > 0.f ? 1.f / lt : 0.f;
    const int r = row0 + rt * 32 + lm;
    if (r < n) {
      uint16_t* orow = out + (size_t)(cu0 + r) * qstride + (size_t)h * kD;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) {
#pragma unroll
        for (int a = 0; a < 4; ++a) {
          const f32x16_t& o = oacc[dt][rt];
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
  constexpr int kRowsPerTile = 64 * 4 / G;
  int* count = reinterpret_cast<int*>(a.workspace);
  int2* tiles = reinterpret_cast<int2*>(static_cast<uint8_t*>(a.workspace) + 16);
  const int max_tiles =
      static_cast<int>((a.workspace_bytes - 16) / sizeof(int2));
  const long long bound = (long long)a.total_q_tokens / kRowsPerTile + a.num_seqs;
  const int grid_tiles = (int)(bound < max_tiles ? bound : max_tiles);
  trace_before(a.stream, "prefill_tile_map");
  hipLaunchKernelGGL(prefill_tile_map_kernel, dim3(1), dim3(256), 0, a.stream, a.cu_seqlens_q,
                     a.num_seqs, kRowsPerTile, tiles, count, grid_tiles);
  trace_after(a.stream);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const long long blocks = (long long)grid_tiles * a.num_kv_heads;
  if (blocks <= 0) return hipSuccess;
  if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
  trace_before(a.stream, "prefill");
  hipLaunchKernelGGL((prefill_kernel<G>), dim3((unsigned)blocks), dim3(256), 0, a.stream,
                     static_cast<const uint16_t*>(a.q), static_cast<const uint8_t*>(a.kv),
                     a.num_blocks, a.block_table, a.seq_lens, a.cu_seqlens_q,
                     static_cast<uint16_t*>(a.out), tiles, count, a.num_q_heads,
                     a.num_kv_heads, a.max_blocks, a.max_seq_len, a.scale * kLog2e);
  trace_after(a.stream);
  return hipGetLastError();
}

hipError_t launch_prefill(const PrefillArgs& a) {
  if (a.head_dim != kD) return hipErrorNotSupported;
  switch (a.num_q_heads / a.num_kv_heads) {
    case 1: return launch_prefill_t<1>(a);
    case 2: return launch_prefill_t<2>(a);
    case 4: return launch_prefill_t<4>(a);
    default: return hipErrorNotSupported;
  }
}

}  // namespace kvattn
