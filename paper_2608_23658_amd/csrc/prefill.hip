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
constexpr int kBufs = 3;                   // LDS steps in the software pipeline

typedef float f32x16_t __attribute__((ext_vector_type(16)));

__device__ __forceinline__ f32x16_t mfma32(bf16x8_t a, bf16x8_t b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// acc *= a on an accumulator that lives in AGPRs. The running output stays in
// the accumulator registers the matrix instructions write; a plain vector
// multiply would make the compiler carry it in VGPRs and copy it across on
// every step, although the rescale itself is rare.
__device__ __forceinline__ void scale_acc(f32x16_t& acc, float a) {
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    float x = acc[i];
    float t;
    asm volatile(
        "v_accvgpr_read_b32 %1, %0\n\t"
        "v_mul_f32 %1, %1, %2\n\t"
        "v_accvgpr_write_b32 %0, %1"
        : "+a"(x), "=&v"(t)
        : "v"(a));
    acc[i] = x;
  }
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
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);  // uniform per wavefront
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

  __shared__ __attribute__((aligned(16))) uint8_t lds[kBufs][2][kStepBlocks][kTileBytes];

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

  // ---- Q^T operands of the wave's two streams of 32 rows ----
  bf16x8_t qb[2][8];
#pragma unroll
  for (int r = 0; r < 2; ++r) {
    const int row = row0 + r * 32 + lm;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) {
      uint4 v = make_uint4(0, 0, 0, 0);
      if (row < n)
        v = *reinterpret_cast<const uint4*>(q + (size_t)(cu0 + row) * qstride +
                                           (size_t)h * kD + ks * 16 + lh * 8);
      qb[r][ks] = __builtin_bit_cast(bf16x8_t, v);
    }
  }

  f32x16_t oacc[4][2];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int r = 0; r < 2; ++r)
#pragma unroll
      for (int i = 0; i < 16; ++i) oacc[dt][r][i] = 0.f;
  float m_ref[2] = {-INFINITY, -INFINITY};   // reference max of each row (log2 domain)
  float l_run[2] = {0.f, 0.f};               // lane-partial row sums

  // ---- gather of one 64-key step straight into LDS (global_load_lds, 16 B/lane) ----
  // Each wavefront fills a contiguous 1 KiB quarter of every 4 KiB tile. K is
  // copied as stored; for V the lane picks the global 16 bytes that belong at
  // its swizzled LDS position (row tid / 2, half tid % 2 holds global half
  // (tid % 2) ^ ((row >> 3) & 1)). A block past L or with an id outside
  // [0, num_blocks) is replaced by block 0 (the host guarantees one exists);
  // the returned bit mask (bit kb: block kb is real) lets the softmax mask its
  // keys and patch_step zero its values.
  const int vrow = tid / 2;
  const int v_src = vrow * 32 + (((tid % 2) ^ ((vrow >> 3) & 1)) * 16);
  auto load_step = [&](int step) {
    const int buf = step % kBufs;
    const int kbase = step * kKeys;
    int bits = 0;
#pragma unroll
    for (int kb = 0; kb < kStepBlocks; ++kb) {
      const int key0 = kbase + kb * kBS;
      int id = key0 < L ? bt[key0 / kBS] : -1;
      const bool ok = (unsigned)id < (unsigned)num_blocks;
      bits |= ok ? (1 << kb) : 0;
      const uint8_t* base = kv + (size_t)(ok ? id : 0) * block_bytes;
      __builtin_amdgcn_global_load_lds(base + k_off + tid * 16, &lds[buf][0][kb][wave * 1024], 16,
                                       0, 0);
      __builtin_amdgcn_global_load_lds(base + v_off + v_src, &lds[buf][1][kb][wave * 1024], 16,
                                       0, 0);
    }
    return bits;
  };
  // Zero the V slots of a landed step that must not contribute: blocks that
  // are not real, and slots at or past L (their bytes may be NaN, and a zero
  // weight times NaN is NaN). Called only when such slots exist.
  auto patch_step = [&](int step, int bits) {
    const int buf = step % kBufs;
    const int kbase = step * kKeys;
    const int half_g = (tid % 2) ^ ((vrow >> 3) & 1);
#pragma unroll
    for (int kb = 0; kb < kStepBlocks; ++kb) {
      uint4* v = reinterpret_cast<uint4*>(&lds[buf][1][kb][tid * 16]);
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
  auto step_clean = [&](int step, int bits) { return bits == 0xf && (step + 1) * kKeys <= L; };
  // All of this wave's direct-to-LDS loads have landed.
  auto wait_loads = [&]() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); };

  const int wave_pos0 = c + row0;   // position of the wave's first row
  const int v_read = lm * 32 + ((lh ^ ((lm >> 3) & 1)) * 16);

  // S^T of stream r for one step: 2 key tiles x 8 k-steps of 16 dims.
  auto qk = [&](int r, int step, f32x16_t (&sa)[2]) {
    const int buf = step % kBufs;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int i = 0; i < 16; ++i) sa[kt][i] = 0.f;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) {
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        const int chunk = 2 * ks + lh;
        const bf16x8_t a = *reinterpret_cast<const bf16x8_t*>(
            &lds[buf][0][2 * kt + k_blk][(chunk * kBS + k_slot) * 16]);
        sa[kt] = mfma32(a, qb[r][ks], sa[kt]);
      }
    }
  };
  // O^T_r += V^T P^T_r for one step: one k-step per block, 4 accumulator chains.
  auto pv = [&](int r, int step, const bf16x8_t (&pr)[4]) {
    const int buf = step % kBufs;
#pragma unroll
    for (int kb = 0; kb < kStepBlocks; ++kb) {
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) {
        const bf16x8_t a =
            *reinterpret_cast<const bf16x8_t*>(&lds[buf][1][kb][dt * 32 * 32 + v_read]);
        oacc[dt][r] = mfma32(a, pr[kb], oacc[dt][r]);
      }
    }
  };
  // Softmax of stream r at one step: P (bf16, 8 consecutive keys of each
  // block), the row-sum update, and the rescale factor for O if the row's
  // reference max moved.
  // Causal / length / real-block mask of stream r's scores at one step, in
  // place; run only on the steps that need it.
  auto mask_scores = [&](int r, int step, int bits, f32x16_t (&sr)[2]) {
    const int kbase = step * kKeys;
    const int qpos = wave_pos0 + r * 32 + lm;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int kpos = kbase + kt * 32 + (i / 8) * 16 + lh * 8 + (i % 8);
        const int blk_ok = (bits >> (2 * kt + i / 8)) & 1;
        const int keep = (kpos <= qpos) & (kpos < L) & blk_ok;
        sr[kt][i] = keep ? sr[kt][i] : -INFINITY;
      }
  };
  auto sm = [&](int r, const f32x16_t (&x)[2], bf16x8_t (&pr)[4], float& alpha, bool& rescale) {
    float mx = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int i = 0; i < 16; ++i) mx = fmaxf(mx, x[kt][i]);
    mx = fmaxf(mx, __shfl_xor(mx, 32, kWave));
    const float tmax = mx * scale_log2;
    // Move the row's reference max only when its scores outgrow it by 2^8.
    const bool grow = tmax > m_ref[r] + kLazyRescale;
    rescale = __builtin_amdgcn_ballot_w64(grow) != 0;
    const float nref = grow ? tmax : m_ref[r];
    alpha = (m_ref[r] == -INFINITY) ? 0.f : fast_exp2(m_ref[r] - nref);
    m_ref[r] = nref;
    const float ref = (nref == -INFINITY) ? 0.f : nref;
    float psum = 0.f;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      float p[16];
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        p[i] = fast_exp2(fmaf(x[kt][i], scale_log2, -ref));
        psum += p[i];
      }
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        const uint4 w = make_uint4(pack_bf16x2(p[8 * half + 0], p[8 * half + 1]),
                                   pack_bf16x2(p[8 * half + 2], p[8 * half + 3]),
                                   pack_bf16x2(p[8 * half + 4], p[8 * half + 5]),
                                   pack_bf16x2(p[8 * half + 6], p[8 * half + 7]));
        pr[2 * kt + half] = __builtin_bit_cast(bf16x8_t, w);
      }
    }
    l_run[r] = l_run[r] * alpha + psum;
  };
  // The step needs the mask if a key can lie past a row of the stream or the
  // end, or a block of the step was not loaded.
  auto needs_mask = [&](int r, int step, int bits) {
    return (step * kKeys + kKeys - 1 > wave_pos0 + r * 32) || !step_clean(step, bits);
  };

  f32x16_t sc[2][2];      // sc[r]: scores of stream r waiting for its softmax
  bf16x8_t pp[2][4];      // pp[r]: P of stream r waiting for its p.v
  float al[2] = {1.f, 1.f};
  bool rs[2] = {false, false};

  // One phase: the MFMA work of stream `mr` (p.v of step i, then q.k of step
  // i + 1 when there is one) interleaved with the softmax of stream `vr` at
  // step `vs`. The two are independent, so the matrix cores and the vector
  // ALU run side by side. O of stream mr is rescaled first if its last
  // softmax moved the reference max; the scores of stream vr are masked first
  // on the steps that need it.
  auto run_phase = [&](auto next_tag, int mr, int i, int vr, int vs, int vbits) {
    constexpr bool kNext = decltype(next_tag)::value;
    if (rs[mr]) {
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) scale_acc(oacc[dt][mr], al[mr]);
      rs[mr] = false;
    }
    if (needs_mask(vr, vs, vbits)) mask_scores(vr, vs, vbits, sc[vr]);
    pv(mr, i, pp[mr]);
    if constexpr (kNext) qk(mr, i + 1, sc[mr]);
    sm(vr, sc[vr], pp[vr], al[vr], rs[vr]);
    // keep the softmax in this phase (the compiler would otherwise sink it
    // next to its first use, away from the matrix work it should overlap)
#pragma unroll
    for (int k = 0; k < 4; ++k) asm volatile("" ::"v"(pp[vr][k]));
  };

  // bits0, bits1, bits2: real-block masks of steps i, i + 1, i + 2
  int bits0 = 0, bits1 = 0, bits2 = 0;
  if (nsteps > 0) bits0 = load_step(0);
  if (nsteps > 1) bits1 = load_step(1);
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  if (nsteps > 0 && !step_clean(0, bits0)) patch_step(0, bits0);
  if (nsteps > 1 && !step_clean(1, bits1)) patch_step(1, bits1);
  __syncthreads();
  if (nsteps > 0) {
    qk(0, 0, sc[0]);
    qk(1, 0, sc[1]);
    if (needs_mask(0, 0, bits0)) mask_scores(0, 0, bits0, sc[0]);
    sm(0, sc[0], pp[0], al[0], rs[0]);
  }
  for (int i = 0; i + 1 < nsteps; ++i) {
    // step i + 1 landed before the last barrier; its V is patched here and
    // first read after the next barrier
    if (i >= 1 && !step_clean(i + 1, bits1)) patch_step(i + 1, bits1);
    if (i + 2 < nsteps) bits2 = load_step(i + 2);
    run_phase(std::true_type{}, 0, i, 1, i, bits0);
    run_phase(std::true_type{}, 1, i, 0, i + 1, bits1);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    bits0 = bits1;
    bits1 = bits2;
  }
  if (nsteps > 0) {
    // last step: p.v of both streams, the softmax of stream 1 in between
    const int i = nsteps - 1;
    run_phase(std::false_type{}, 0, i, 1, i, bits0);
    if (rs[1]) {
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) scale_acc(oacc[dt][1], al[1]);
    }
    pv(1, i, pp[1]);
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
