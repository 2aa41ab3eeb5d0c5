// Split-K paged decode for gfx950: one new query token per sequence attends
// to its whole context, read through the block table (the paper, Section 3
// "The contiguity constraint"; Section 5, decode is one token per sequence).
//
// One workgroup = one wavefront = one (kv head, sequence, split of the
// context). The grid is one-dimensional with the kv head varying fastest and
// the split slowest, so consecutive workgroups, which the dispatcher deals
// round-robin to the 8 XCDs, carry equal work: putting the split first would
// send split k of every sequence to XCD k and starve the XCDs that hold the
// late splits only long sequences have. The G query heads sharing the kv
// head are served by every K/V byte read (grouped-query sharing). The
// wavefront walks its split in steps of 64 tokens (4 blocks of 16):
//   * loads: each block's K tile and V tile are read as they lie in memory,
//     1 KiB per 16-byte load (K and V are read once, so the loads are
//     non-temporal), and the K and V loads of a block are issued together.
//     Reading K lane-per-token instead (four 256-byte pieces from four blocks
//     per load), or all K loads before all V loads, measured 4-6% slower:
//     the memory system serves a block's two tiles best when they are asked
//     for at once.
//   * K: with the chunk-major K tile, load i of a block gives lane l chunk
//     4 i + l / 16 of token slot l % 16, a quarter of that token's row. Each
//     lane dots its quarters of the rows of the four tokens in its slot (one
//     per block) with the same dims of q (read from LDS), and the four lanes
//     of a slot add their quarters with two row swaps. Lane t then takes the
//     score of token t of the step (block t / 16, slot t % 16).
//   * softmax: wavefront max per head (DPP and lane-row swaps), exp2 in the
//     log2 domain, lane-local partial sums, one rescale of the accumulators
//     per step.
//   * V: in the dim-major V tile lane l owns dim rows l / R (R = 16-byte
//     chunks per row) and a run of consecutive tokens, so for bf16 p.v is a
//     bf16 dot2 over token pairs. p reaches those lanes through LDS.
// Only the last step of a split can hold slots past the sequence's length,
// whose contents are arbitrary (possibly NaN); that step masks them. Partials
// (m, l, o) of every split go to the workspace; a second kernel merges them
// (log-sum-exp) in split order, so the result depends only on the sequence's
// own length.

#include "common.hpp"
#include "launch.hpp"

namespace kvattn {

template <int D, int G, bool BF16>
struct DecodeShape {
  static constexpr int kEsz = BF16 ? 2 : 4;
  static constexpr int kVec = 16 / kEsz;          // elements per 16-byte chunk
  static constexpr int kBS = 16;                  // tokens per block
  static constexpr int kTile = 64;                // tokens per wavefront step
  static constexpr int kTB = kTile / kBS;         // blocks per step
  static constexpr int kKCh = D / kVec;           // 16-byte chunks per K row
  static constexpr int kR = kBS * kEsz / 16;      // 16-byte chunks per V dim row
  static constexpr int kDPI = kWave / kR;         // V dim rows per load
  static constexpr int kVI = D / kDPI;            // V loads per block
  static constexpr int kTileElems = kBS * D;      // one (block, K/V, head) tile
  static constexpr int kPWords = BF16 ? (kTile / 2) * G : kTile * G;
  static_assert(kVI * 1024 == kTileElems * kEsz, "V tile is kVI loads of 1 KiB");
  static_assert(kKCh == 4 * kVI, "a K load of 1 KiB holds a quarter of each of 16 rows");
};

// kTwo: the layer is split over two tensors (the design the paper rejects in
// Section 3, "The contiguity constraint"): ids below num_base address kv, the
// others kv2 at id - num_base. Otherwise kv2 and num_base are unused.
template <int D, int G, bool BF16, bool kTwo = false>
__global__ __launch_bounds__(64) void decode_split_kernel(
    const uint8_t* __restrict__ q, const uint8_t* __restrict__ kv,
    const uint8_t* __restrict__ kv2, int num_base, int num_blocks,
    const int* __restrict__ block_table, const int* __restrict__ seq_lens,
    uint8_t* __restrict__ out, float* __restrict__ ws_o, float2* __restrict__ ws_ml,
    int num_seqs, int num_q_heads, int num_kv_heads, int max_blocks, int max_seq_len,
    int split_tokens, int max_splits, float scale_log2) {
  using S = DecodeShape<D, G, BF16>;
  const int wid = blockIdx.x;
  const int g = wid % num_kv_heads;
  const int s = (wid / num_kv_heads) % num_seqs;
  const int split = wid / (num_kv_heads * num_seqs);
  const int lane = threadIdx.x;
  const int h0 = g * G;
  const size_t row_bytes = (size_t)D * S::kEsz;

  int L = seq_lens[s];
  L = min(max(L, 0), min(max_seq_len, max_blocks * S::kBS));
  const int nsplit = (L + split_tokens - 1) / split_tokens;

  if (L == 0) {
    if (split == 0) {
      uint4* o = reinterpret_cast<uint4*>(out + ((size_t)s * num_q_heads + h0) * row_bytes);
      for (int c = lane; c < G * D * S::kEsz / 16; c += kWave) o[c] = make_uint4(0, 0, 0, 0);
    }
    return;
  }
  if (split >= nsplit) return;
  const int t0 = split * split_tokens;
  const int t1 = min(L, t0 + split_tokens);

  __shared__ uint32_t p_lds[S::kPWords];
  __shared__ uint4 q_lds[G * S::kKCh];
  {
    const uint4* qsrc = reinterpret_cast<const uint4*>(q + ((size_t)s * num_q_heads + h0) * row_bytes);
    for (int i = lane; i < G * S::kKCh; i += kWave) q_lds[i] = qsrc[i];
  }
  __syncthreads();

  const int* bt = block_table + (size_t)s * max_blocks;
  const size_t tile_bytes = (size_t)S::kTileElems * S::kEsz;
  const size_t head_off = (size_t)g * tile_bytes;
  const size_t block_bytes = 2 * (size_t)num_kv_heads * tile_bytes;
  const size_t v_off = (size_t)num_kv_heads * tile_bytes + head_off;
  auto block_ptr = [&](int id) -> const uint8_t* {
    if constexpr (kTwo)
      return id < num_base ? kv + (size_t)id * block_bytes
                           : kv2 + (size_t)(id - num_base) * block_bytes;
    else
      return kv + (size_t)id * block_bytes;
  };

  float m_run[G], l_run[G], acc[S::kVI][G];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    m_run[h] = -INFINITY;
    l_run[h] = 0.f;
#pragma unroll
    for (int i = 0; i < S::kVI; ++i) acc[i][h] = 0.f;
  }

  // block of this lane's token within the step, and which quarter of the K
  // rows of its slot the lane holds
  const int kj = lane / S::kBS;
  const int vrc = lane % S::kR;   // this lane's chunk of a V dim row

  // Steps of 64 tokens; in the last one (kTail) the step may end inside a
  // block, so tokens at or past t1 are masked.
  for (int tb = t0; tb < t1; tb += S::kTile) {
    const bool kTail = tb + S::kTile > t1;
    const int blk0 = tb / S::kBS;
    int bid[S::kTB];
#pragma unroll
    for (int j = 0; j < S::kTB; ++j) {
      int id = -1;
      if (!kTail || tb + j * S::kBS < t1) {
        id = bt[blk0 + j];
        if ((unsigned)id >= (unsigned)num_blocks) id = -1;
      }
      bid[j] = id;
    }
    int my_b = bid[0];
#pragma unroll
    for (int j = 1; j < S::kTB; ++j) my_b = (kj == j) ? bid[j] : my_b;
    const bool kvalid = (!kTail || tb + lane < t1) && (my_b >= 0);

    // ---- loads: each block's K tile and V tile as they lie in memory, 1 KiB
    // per load, the two tiles of a block issued together ----
    // K piece i of a block gives lane l the 16-byte chunk 4 i + l / 16 of the
    // block's token slot l % 16: a quarter of that token's row.
    uint4 kreg[S::kTB][S::kVI];
    uint4 vreg[S::kTB][S::kVI];
#pragma unroll
    for (int j = 0; j < S::kTB; ++j) {
      if (bid[j] >= 0) {
        const uint8_t* bp = block_ptr(bid[j]);
        const uint4* kp = reinterpret_cast<const uint4*>(bp + head_off) + lane;
        const uint4* vp = reinterpret_cast<const uint4*>(bp + v_off) + lane;
#pragma unroll
        for (int i = 0; i < S::kVI; ++i) {
          kreg[j][i] = load_nt(kp + i * kWave);
          vreg[j][i] = load_nt(vp + i * kWave);
        }
      } else {
#pragma unroll
        for (int i = 0; i < S::kVI; ++i) {
          kreg[j][i] = make_uint4(0, 0, 0, 0);
          vreg[j][i] = make_uint4(0, 0, 0, 0);
        }
      }
    }

    // ---- scores: each lane dots its quarter of the rows of the four tokens
    // in its slot (one per block) with the same dims of q, then the four
    // lanes of a slot (l, l ^ 16, l ^ 32, l ^ 48) add their quarters ----
    float part[S::kTB][G];
#pragma unroll
    for (int j = 0; j < S::kTB; ++j)
#pragma unroll
      for (int h = 0; h < G; ++h) part[j][h] = 0.f;
#pragma unroll
    for (int i = 0; i < S::kVI; ++i) {
#pragma unroll
      for (int h = 0; h < G; ++h) {
        const uint4 qc = q_lds[h * S::kKCh + 4 * i + kj];
#pragma unroll
        for (int j = 0; j < S::kTB; ++j) {
          const uint4 k = kreg[j][i];
          float a = part[j][h];
          if constexpr (BF16) {
            a = dot2_bf16(k.x, qc.x, a);
            a = dot2_bf16(k.y, qc.y, a);
            a = dot2_bf16(k.z, qc.z, a);
            a = dot2_bf16(k.w, qc.w, a);
          } else {
            a = fmaf(__uint_as_float(k.x), __uint_as_float(qc.x), a);
            a = fmaf(__uint_as_float(k.y), __uint_as_float(qc.y), a);
            a = fmaf(__uint_as_float(k.z), __uint_as_float(qc.z), a);
            a = fmaf(__uint_as_float(k.w), __uint_as_float(qc.w), a);
          }
          part[j][h] = a;
        }
      }
    }
    // this lane's token is slot lane % 16 of block kj
    float sc[G];
#pragma unroll
    for (int h = 0; h < G; ++h) {
#pragma unroll
      for (int j = 0; j < S::kTB; ++j) part[j][h] = cross_row_sum(part[j][h]);
      sc[h] = part[0][h];
#pragma unroll
      for (int j = 1; j < S::kTB; ++j) sc[h] = (kj == j) ? part[j][h] : sc[h];
    }

    // ---- online softmax over the step (log2 domain) ----
    float alpha[G];
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const float x = kvalid ? sc[h] * scale_log2 : -INFINITY;
      const float mn = fmaxf(m_run[h], wave_max(x));
      const float ref = (mn == -INFINITY) ? 0.f : mn;
      alpha[h] = fast_exp2(m_run[h] - ref);
      float p = fast_exp2(x - ref);
      if constexpr (BF16) {
        const uint16_t pb = to_bf16(p);
        p = __uint_as_float((uint32_t)pb << 16);
        reinterpret_cast<uint16_t*>(p_lds)[((lane >> 1) * G + h) * 2 + (lane & 1)] = pb;
      } else {
        reinterpret_cast<float*>(p_lds)[lane * G + h] = p;
      }
      l_run[h] = l_run[h] * alpha[h] + p;
      m_run[h] = mn;
    }
#pragma unroll
    for (int i = 0; i < S::kVI; ++i)
#pragma unroll
      for (int h = 0; h < G; ++h) acc[i][h] *= alpha[h];
    __syncthreads();

    // ---- p . v ----
#pragma unroll
    for (int j = 0; j < S::kTB; ++j) {
      if (bid[j] < 0) continue;
      const int tok0 = tb + j * S::kBS + vrc * S::kVec;   // first token of this lane's chunk
      if constexpr (BF16) {
        // 4 token pairs x G heads of bf16 pairs
        uint32_t pw[4][G];
        const uint4* pp = reinterpret_cast<const uint4*>(p_lds) + ((j * 8 + vrc * 4) * G) / 4;
#pragma unroll
        for (int x = 0; x < G; ++x) {
          const uint4 w = pp[x];
          const uint32_t ws4[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
          for (int y = 0; y < 4; ++y) {
            const int idx = x * 4 + y;      // = pair * G + head
            pw[idx / G][idx % G] = ws4[y];
          }
        }
#pragma unroll
        for (int i = 0; i < S::kVI; ++i) {
          uint4 v = vreg[j][i];
          if (kTail) {
            uint32_t vv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
            for (int k = 0; k < 4; ++k) {
              const uint32_t lo = (tok0 + 2 * k < t1) ? 0x0000ffffu : 0u;
              const uint32_t hi = (tok0 + 2 * k + 1 < t1) ? 0xffff0000u : 0u;
              vv[k] &= (lo | hi);
            }
            v = make_uint4(vv[0], vv[1], vv[2], vv[3]);
          }
#pragma unroll
          for (int h = 0; h < G; ++h) {
            float a = acc[i][h];
            a = dot2_bf16(v.x, pw[0][h], a);
            a = dot2_bf16(v.y, pw[1][h], a);
            a = dot2_bf16(v.z, pw[2][h], a);
            a = dot2_bf16(v.w, pw[3][h], a);
            acc[i][h] = a;
          }
        }
      } else {
        float pf[4][G];
        const float* pp = reinterpret_cast<const float*>(p_lds) + (j * S::kBS + vrc * 4) * G;
#pragma unroll
        for (int k = 0; k < 4; ++k)
#pragma unroll
          for (int h = 0; h < G; ++h) pf[k][h] = pp[k * G + h];
#pragma unroll
        for (int i = 0; i < S::kVI; ++i) {
          const uint4 v = vreg[j][i];
          float vf[4] = {__uint_as_float(v.x), __uint_as_float(v.y), __uint_as_float(v.z),
                         __uint_as_float(v.w)};
          if (kTail) {
#pragma unroll
            for (int k = 0; k < 4; ++k) vf[k] = (tok0 + k < t1) ? vf[k] : 0.f;
          }
#pragma unroll
          for (int h = 0; h < G; ++h) {
            float a = acc[i][h];
#pragma unroll
            for (int k = 0; k < 4; ++k) a = fmaf(pf[k][h], vf[k], a);
            acc[i][h] = a;
          }
        }
      }
    }
    __syncthreads();
  }

  // ---- finish: lane sums, merge the chunks of a dim row ----
  float l_tot[G];
#pragma unroll
  for (int h = 0; h < G; ++h) l_tot[h] = wave_sum(l_run[h]);
#pragma unroll
  for (int i = 0; i < S::kVI; ++i)
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
      for (int o = 1; o < S::kR; o <<= 1) acc[i][h] += __shfl_xor(acc[i][h], o, kWave);

  if (nsplit == 1) {
    if (vrc == 0) {
#pragma unroll
      for (int h = 0; h < G; ++h) {
        const float inv = l_tot[h] > 0.f ? 1.f / l_tot[h] : 0.f;
        uint8_t* orow = out + ((size_t)s * num_q_heads + h0 + h) * row_bytes;
#pragma unroll
        for (int i = 0; i < S::kVI; ++i) {
          const int d = i * S::kDPI + lane / S::kR;
          if constexpr (BF16)
            reinterpret_cast<uint16_t*>(orow)[d] = to_bf16(acc[i][h] * inv);
          else
            reinterpret_cast<float*>(orow)[d] = acc[i][h] * inv;
        }
      }
    }
  } else {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const size_t idx = ((size_t)s * num_q_heads + h0 + h) * max_splits + split;
      if (vrc == 0) {
#pragma unroll
        for (int i = 0; i < S::kVI; ++i) ws_o[idx * D + i * S::kDPI + lane / S::kR] = acc[i][h];
      }
      if (lane == 0) ws_ml[idx] = make_float2(m_run[h], l_tot[h]);
    }
  }
}

// Merge the split partials of one (sequence, query head) per wavefront.
template <int D, bool BF16>
__global__ __launch_bounds__(256) void decode_combine_kernel(
    const float* __restrict__ ws_o, const float2* __restrict__ ws_ml,
    const int* __restrict__ seq_lens, uint8_t* __restrict__ out, int num_seqs,
    int num_q_heads, int max_blocks, int max_seq_len, int split_tokens, int max_splits) {
  const int w = blockIdx.x * 4 + threadIdx.x / kWave;
  const int lane = threadIdx.x % kWave;
  if (w >= num_seqs * num_q_heads) return;
  const int s = w / num_q_heads;
  int L = seq_lens[s];
  L = min(max(L, 0), min(max_seq_len, max_blocks * 16));
  const int ns = (L + split_tokens - 1) / split_tokens;
  if (ns <= 1) return;
  const size_t base = (size_t)w * max_splits;
  float m = -INFINITY;
  for (int j = 0; j < ns; ++j) m = fmaxf(m, ws_ml[base + j].x);
  constexpr int kPer = D / kWave;
  float o[kPer];
#pragma unroll
  for (int k = 0; k < kPer; ++k) o[k] = 0.f;
  float l = 0.f;
  if (m != -INFINITY) {
    for (int j = 0; j < ns; ++j) {
      const float2 ml = ws_ml[base + j];
      const float wgt = fast_exp2(ml.x - m);
      l += wgt * ml.y;
      const float* oj = ws_o + (base + j) * D;
#pragma unroll
      for (int k = 0; k < kPer; ++k) o[k] = fmaf(wgt, oj[lane + k * kWave], o[k]);
    }
  }
  const float inv = l > 0.f ? 1.f / l : 0.f;
  const size_t row = (size_t)w * D;
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    if constexpr (BF16)
      reinterpret_cast<uint16_t*>(out)[row + lane + k * kWave] = to_bf16(o[k] * inv);
    else
      reinterpret_cast<float*>(out)[row + lane + k * kWave] = o[k] * inv;
  }
}

template <int D, int G, bool BF16, bool kTwo = false>
static hipError_t launch_decode_t(const DecodeArgs& a) {
  const int max_splits = (a.max_seq_len + a.split_tokens - 1) / a.split_tokens;
  const int splits = max_splits > 0 ? max_splits : 1;
  const long long blocks = (long long)splits * a.num_kv_heads * a.num_seqs;
  if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
  float* ws_o = reinterpret_cast<float*>(a.workspace);
  float2* ws_ml = reinterpret_cast<float2*>(static_cast<uint8_t*>(a.workspace) + a.ws_ml_offset);
  trace_before(a.stream, kTwo ? "decode_split_two_tensor" : "decode_split");
  hipLaunchKernelGGL((decode_split_kernel<D, G, BF16, kTwo>), dim3((unsigned)blocks), dim3(64), 0,
                     a.stream, static_cast<const uint8_t*>(a.q),
                     static_cast<const uint8_t*>(a.kv), static_cast<const uint8_t*>(a.kv2),
                     a.num_base, a.num_blocks, a.block_table, a.seq_lens,
                     static_cast<uint8_t*>(a.out), ws_o, ws_ml, a.num_seqs, a.num_q_heads,
                     a.num_kv_heads, a.max_blocks, a.max_seq_len, a.split_tokens, splits,
                     a.scale * kLog2e);
  trace_after(a.stream);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || max_splits <= 1) return e;
  const int pairs = a.num_seqs * a.num_q_heads;
  trace_before(a.stream, "decode_combine");
  hipLaunchKernelGGL((decode_combine_kernel<D, BF16>), dim3((pairs + 3) / 4), dim3(256), 0,
                     a.stream, ws_o, ws_ml, a.seq_lens, static_cast<uint8_t*>(a.out),
                     a.num_seqs, a.num_q_heads, a.max_blocks, a.max_seq_len, a.split_tokens,
                     splits);
  trace_after(a.stream);
  return hipGetLastError();
}

template <int D, bool BF16>
static hipError_t dispatch_g(const DecodeArgs& a, int G) {
  switch (G) {
    case 1: return launch_decode_t<D, 1, BF16>(a);
    case 2: return launch_decode_t<D, 2, BF16>(a);
    case 4: return launch_decode_t<D, 4, BF16>(a);
    case 8: return launch_decode_t<D, 8, BF16>(a);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_decode(const DecodeArgs& a) {
  const int G = a.num_q_heads / a.num_kv_heads;
  if (a.kv2) {   // two-tensor layer: built for bf16, head_dim 128
    if (!a.bf16 || a.head_dim != 128) return hipErrorNotSupported;
    switch (G) {
      case 1: return launch_decode_t<128, 1, true, true>(a);
      case 2: return launch_decode_t<128, 2, true, true>(a);
      case 4: return launch_decode_t<128, 4, true, true>(a);
      case 8: return launch_decode_t<128, 8, true, true>(a);
      default: return hipErrorInvalidValue;
    }
  }
  if (a.bf16) {
    if (a.head_dim == 128) return dispatch_g<128, true>(a, G);
    if (a.head_dim == 64) return dispatch_g<64, true>(a, G);
  } else {
    if (a.head_dim == 64) return dispatch_g<64, false>(a, G);
  }
  return hipErrorInvalidValue;
}

}  // namespace kvattn
