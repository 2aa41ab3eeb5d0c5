// Chunked-prefill attention for gfx950 on bf16 MFMA (the paper, Section 5:
// prefill is compute bound and a chunk attends to all earlier context, so
// chunking splits the same work; Section 1: max_num_batched_tokens bounds
// the chunk).
//
// Work tile = (kv head g, 64 * 4 / G consecutive new rows of one sequence).
// A workgroup of 4 wavefronts owns one tile: wave w serves query head
// g * G + w % G over 64 rows. K/V tiles of 64 keys (4 blocks) are gathered
// through the block table into LDS once per workgroup and shared by the G
// query heads of the group.
//
// Per wave and 64-key step, with v_mfma_f32_16x16x32_bf16:
//   S^T[key][row] = K[key][:] . Q[row][:]   A = K rows straight from the
//       chunk-major K tile (16-byte chunk c of slot r at (c * 16 + r) * 16),
//       B = Q^T held in registers for the whole kernel;
//   softmax over keys in the log2 domain: in the S^T accumulator layout every
//       lane holds 4 keys of one query row, so the row max needs 2 shuffles
//       and the rescale of O^T is lane-local;
//   O^T[d][row] += V^T[d][key] P^T[key][row]   A = 8-byte runs of the
//       dim-major V tile, B = the bf16 P values already in the lane that
//       produced them (keys 4j..4j+3 of two consecutive blocks).
// The causal mask (bottom-right: row i at position L - n + i sees keys
// 0 .. L - n + i) is applied only on steps that reach the diagonal.

#include "common.hpp"
#include "launch.hpp"

namespace kvattn {

namespace {

constexpr int kD = 128;
constexpr int kBS = 16;
constexpr int kKeys = 64;          // keys per step
constexpr int kStepBlocks = 4;     // blocks per step
constexpr int kTileBytes = kBS * kD * 2;   // one (block, K/V, head) tile: 4 KiB

typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f32x4_t mfma16(bf16x8_t a, bf16x8_t b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
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

  // ---- Q^T operands for the wave's 64 rows (4 groups of 16) ----
  const int lr = lane % 16;     // row within a group / key-or-dim index within a 16-tile
  const int lq = lane / 16;     // quarter: which 8-wide k slice / which 4 accumulator rows
  bf16x8_t qb[4][4];
#pragma unroll
  for (int rg = 0; rg < 4; ++rg) {
    const int r = row0 + rg * 16 + lr;
#pragma unroll
    for (int ds = 0; ds < 4; ++ds) {
      if (r < n) {
        const uint4 v = *reinterpret_cast<const uint4*>(
            q + (size_t)(cu0 + r) * qstride + (size_t)h * kD + ds * 32 + lq * 8);
        qb[rg][ds] = __builtin_bit_cast(bf16x8_t, v);
      } else {
        qb[rg][ds] = __builtin_bit_cast(bf16x8_t, make_uint4(0, 0, 0, 0));
      }
    }
  }

  f32x4_t oacc[8][4];
#pragma unroll
  for (int dt = 0; dt < 8; ++dt)
#pragma unroll
    for (int rg = 0; rg < 4; ++rg) oacc[dt][rg] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float m_run[4], l_run[4];
#pragma unroll
  for (int rg = 0; rg < 4; ++rg) {
    m_run[rg] = -INFINITY;
    l_run[rg] = 0.f;
  }

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
  auto store_step = [&](int buf, int step) {
    const int kbase = step * kKeys;
    const bool tail = kbase + kKeys > L;
#pragma unroll
    for (int kb = 0; kb < kStepBlocks; ++kb) {
      uint4 v = pre[kb * 2 + 1];
      if (tail) {
        // V dim row tid / 2, slots 8 * (tid % 2) .. + 7: zero slots at or past L
        const int key = kbase + kb * kBS + 8 * (tid % 2);
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
      *reinterpret_cast<uint4*>(&lds[buf][1][kb][tid * 16]) = v;
    }
  };

  if (nsteps > 0) {
    load_step(0);
    store_step(0, 0);
  }
  __syncthreads();

  const int wave_pos0 = c + row0;   // position of the wave's first row
  for (int step = 0; step < nsteps; ++step) {
    const int buf = step & 1;
    if (step + 1 < nsteps) load_step(step + 1);
    const int kbase = step * kKeys;

    // ---- S^T = K Q^T ----
    f32x4_t sacc[kStepBlocks][4];
#pragma unroll
    for (int kb = 0; kb < kStepBlocks; ++kb)
#pragma unroll
      for (int rg = 0; rg < 4; ++rg) sacc[kb][rg] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < kStepBlocks; ++kb) {
#pragma unroll
      for (int ds = 0; ds < 4; ++ds) {
        const bf16x8_t a = *reinterpret_cast<const bf16x8_t*>(&lds[buf][0][kb][(64 * ds + lane) * 16]);
#pragma unroll
        for (int rg = 0; rg < 4; ++rg) sacc[kb][rg] = mfma16(a, qb[rg][ds], sacc[kb][rg]);
      }
    }

    // ---- online softmax per row (lane holds row lr of each group) ----
    const bool mask = (kbase + kKeys - 1 > wave_pos0) || (kbase + kKeys > L);
    bf16x8_t pb[4][2];
#pragma unroll
    for (int rg = 0; rg < 4; ++rg) {
      const int qpos = wave_pos0 + rg * 16 + lr;
      float x[kStepBlocks][4];
      float tmax = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < kStepBlocks; ++kb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float v = sacc[kb][rg][i] * scale_log2;
          if (mask) {
            const int kpos = kbase + kb * kBS + lq * 4 + i;
            v = (kpos > qpos || kpos >= L) ? -INFINITY : v;
          }
          x[kb][i] = v;
          tmax = fmaxf(tmax, v);
        }
      tmax = fmaxf(tmax, __shfl_xor(tmax, 16, kWave));
      tmax = fmaxf(tmax, __shfl_xor(tmax, 32, kWave));
      const float mn = fmaxf(m_run[rg], tmax);
      const float ref = (mn == -INFINITY) ? 0.f : mn;
      const float alpha = fast_exp2(m_run[rg] - ref);
      m_run[rg] = mn;
      float psum = 0.f;
      float p[kStepBlocks][4];
#pragma unroll
      for (int kb = 0; kb < kStepBlocks; ++kb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          p[kb][i] = fast_exp2(x[kb][i] - ref);
          psum += p[kb][i];
        }
      l_run[rg] = l_run[rg] * alpha + psum;
#pragma unroll
      for (int bp = 0; bp < 2; ++bp) {
        const uint4 w = make_uint4(pack_bf16x2(p[2 * bp][0], p[2 * bp][1]),
                                   pack_bf16x2(p[2 * bp][2], p[2 * bp][3]),
                                   pack_bf16x2(p[2 * bp + 1][0], p[2 * bp + 1][1]),
                                   pack_bf16x2(p[2 * bp + 1][2], p[2 * bp + 1][3]));
        pb[rg][bp] = __builtin_bit_cast(bf16x8_t, w);
      }
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) oacc[dt][rg] *= alpha;
    }

    // ---- O^T += V^T P^T ----
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) {
#pragma unroll
      for (int bp = 0; bp < 2; ++bp) {
        const int off = (dt * 16 + lr) * 32 + lq * 8;
        const uint2 v0 = *reinterpret_cast<const uint2*>(&lds[buf][1][2 * bp][off]);
        const uint2 v1 = *reinterpret_cast<const uint2*>(&lds[buf][1][2 * bp + 1][off]);
        const bf16x8_t a = __builtin_bit_cast(bf16x8_t, make_uint4(v0.x, v0.y, v1.x, v1.y));
#pragma unroll
        for (int rg = 0; rg < 4; ++rg) oacc[dt][rg] = mfma16(a, pb[rg][bp], oacc[dt][rg]);
      }
    }

    if (step + 1 < nsteps) store_step(buf ^ 1, step + 1);
    __syncthreads();
  }

  // ---- normalise and write O (rows of this lane: lr of each group) ----
#pragma unroll
  for (int rg = 0; rg < 4; ++rg) {
    float lt = l_run[rg];
    lt += __shfl_xor(lt, 16, kWave);
    lt += __shfl_xor(lt, 32, kWave);
    const float inv = lt > 0.f ? 1.f / lt : 0.f;
    const int r = row0 + rg * 16 + lr;
    if (r < n) {
      uint16_t* orow = out + (size_t)(cu0 + r) * qstride + (size_t)h * kD;
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) {
        const f32x4_t o = oacc[dt][rg];
        const uint2 w = make_uint2(pack_bf16x2(o[0] * inv, o[1] * inv),
                                   pack_bf16x2(o[2] * inv, o[3] * inv));
        *reinterpret_cast<uint2*>(orow + dt * 16 + lq * 4) = w;
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
