// Writing a step's new K/V rows into their paged slots: the step before
// attention reads them (Section 3, "The contiguity constraint": the kernel
// indexes one tensor per layer by block id; Section 2: the cache is handed out
// in fixed-size blocks).
//
// Four wavefronts per (run of 16 consecutive tokens, kv head). When the run's
// slots are one whole block in order (what a prefill chunk produces), the K
// tile is written as contiguous 256-byte rows of 16 slots (the tile is
// chunk-major: chunk c of slot r at (c * 16 + r) * 16 bytes) and the V rows are
// staged in LDS and written as whole 16-byte pieces of the dim-major V tile;
// wavefront q of the four takes a quarter of each row's chunks. Any other run
// (decode steps, partial blocks, padding) takes the general path, wavefront q
// taking 4 of the run's tokens: each 16-byte chunk of a row is read once,
// lands as one 16-byte run in the K tile, and its elements land 16 slots apart
// in the V tile.

#include "common.hpp"
#include "launch.hpp"

namespace kvattn {

namespace {
constexpr int kAppendBS = 16;        // slots per block, tokens per run
constexpr int kAppendWaves = 4;
constexpr int kMaxChunks = 32;       // 16-byte chunks per row (head_dim * esz <= 512)
}  // namespace

template <int ESZ>
__global__ __launch_bounds__(kAppendWaves * kWave) void kv_append_kernel(
    const uint4* __restrict__ k_new, const uint4* __restrict__ v_new,
    const int* __restrict__ slot_mapping, uint8_t* __restrict__ kv, int num_tokens,
    int num_kv_heads, int chunks_per_row, int capacity, long long num_items) {
  constexpr int kVec = 16 / ESZ;     // elements per 16-byte chunk
  constexpr int kParts = kAppendWaves;
  // V rows of this wavefront's chunks of the run, padded by 16 bytes per row
  // against bank conflicts.
  __shared__ __attribute__((aligned(16)))
      uint4 stage[kAppendWaves][kAppendBS][kMaxChunks / kParts + 1];
  const int q = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const long long item = blockIdx.x;              // (run, head)
  if (item >= num_items) return;
  const int g = (int)(item % num_kv_heads);
  const int t0 = (int)(item / num_kv_heads) * kAppendBS;
  const int n = min(kAppendBS, num_tokens - t0);
  const int CH = chunks_per_row;
  const size_t tile_bytes = (size_t)kAppendBS * CH * 16;
  auto row_index = [&](int t) { return ((size_t)t * num_kv_heads + g) * CH; };

  // Is the run one whole block, in slot order?
  const int my_slot = lane < n ? slot_mapping[t0 + lane] : -1;
  const int s0 = __shfl(my_slot, 0, kWave);
  const bool in_order = lane >= kAppendBS || my_slot == s0 + lane;
  const bool fast = n == kAppendBS && s0 >= 0 && s0 % kAppendBS == 0 &&
                    s0 + kAppendBS <= capacity && __all(in_order);
  if (fast) {
    const int b = s0 / kAppendBS;
    uint8_t* kt = kv + ((size_t)b * 2 * num_kv_heads + g) * tile_bytes;
    uint8_t* vt = kt + (size_t)num_kv_heads * tile_bytes;
    const int cq = CH / kParts;                    // chunks of this wavefront
    const int c0 = q * cq;
    // K: lane -> (chunk c, slot r), slots fastest: 16 lanes write 256 bytes
    for (int idx = lane; idx < kAppendBS * cq; idx += kWave) {
      const int c = c0 + idx / kAppendBS, r = idx % kAppendBS;
      *reinterpret_cast<uint4*>(kt + ((size_t)c * kAppendBS + r) * 16) =
          k_new[row_index(t0 + r) + c];
    }
    // V: stage the run's chunks c0 .. c0 + cq of the 16 rows, then write dim rows
    for (int idx = lane; idx < kAppendBS * cq; idx += kWave) {
      const int r = idx / cq, c = idx % cq;
      stage[q][r][c] = v_new[row_index(t0 + r) + c0 + c];
    }
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
    // dim row j holds 16 slots = kAppendBS / kVec pieces of 16 bytes
    constexpr int kPieces = kAppendBS / kVec;
    const int dims = cq * kVec;                    // dims of this wavefront
    for (int idx = lane; idx < dims * kPieces; idx += kWave) {
      const int jl = idx / kPieces, p = idx % kPieces;
      const int c = jl / kVec, e = jl % kVec;
      uint32_t w[4];
      if constexpr (ESZ == 2) {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const uint16_t* lo = reinterpret_cast<const uint16_t*>(&stage[q][p * 8 + 2 * k][c]);
          const uint16_t* hi = reinterpret_cast<const uint16_t*>(&stage[q][p * 8 + 2 * k + 1][c]);
          w[k] = (uint32_t)lo[e] | ((uint32_t)hi[e] << 16);
        }
      } else {
#pragma unroll
        for (int k = 0; k < 4; ++k)
          w[k] = reinterpret_cast<const uint32_t*>(&stage[q][p * 4 + k][c])[e];
      }
      const int j = c0 * kVec + jl;
      *reinterpret_cast<uint4*>(vt + ((size_t)j * kAppendBS + p * kVec) * ESZ) =
          make_uint4(w[0], w[1], w[2], w[3]);
    }
    return;
  }
  // General path: wavefront q takes tokens 4q .. 4q + 3 of the run,
  // lane -> (token, chunk)
  constexpr int kTok = kAppendBS / kParts;
  for (int idx = lane; idx < kTok * CH; idx += kWave) {
    const int i = q * kTok + idx / CH, c = idx % CH;
    if (i >= n) break;
    const int slot = slot_mapping[t0 + i];
    if (slot < 0 || slot >= capacity) continue;        // padding / outside the layer
    const int b = slot / kAppendBS, r = slot % kAppendBS;
    uint8_t* kt = kv + ((size_t)b * 2 * num_kv_heads + g) * tile_bytes;
    uint8_t* vt = kt + (size_t)num_kv_heads * tile_bytes;
    *reinterpret_cast<uint4*>(kt + ((size_t)c * kAppendBS + r) * 16) = k_new[row_index(t0 + i) + c];
    const uint4 vc = v_new[row_index(t0 + i) + c];
    const uint32_t w[4] = {vc.x, vc.y, vc.z, vc.w};
    const int j0 = c * kVec;
    if constexpr (ESZ == 2) {
      uint16_t* v16 = reinterpret_cast<uint16_t*>(vt);
#pragma unroll
      for (int e = 0; e < kVec; ++e)
        v16[(size_t)(j0 + e) * kAppendBS + r] = (uint16_t)(w[e / 2] >> (16 * (e % 2)));
    } else {
      uint32_t* v32 = reinterpret_cast<uint32_t*>(vt);
#pragma unroll
      for (int e = 0; e < kVec; ++e) v32[(size_t)(j0 + e) * kAppendBS + r] = w[e];
    }
  }
}

hipError_t launch_append(const AppendArgs& a) {
  const int chunks_per_row = a.head_dim * a.esz / 16;
  if (chunks_per_row > kMaxChunks || chunks_per_row % kAppendWaves) return hipErrorNotSupported;
  const long long runs = (a.num_tokens + kAppendBS - 1) / kAppendBS;
  const long long items = runs * a.num_kv_heads;   // one workgroup per (run, head)
  if (items == 0) return hipSuccess;
  const long long blocks = items;
  if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
  const int capacity = a.num_blocks * kAppendBS;
  trace_before(a.stream, "kv_append");
  if (a.esz == 2)
    hipLaunchKernelGGL(kv_append_kernel<2>, dim3((unsigned)blocks), dim3(kAppendWaves * kWave),
                       0, a.stream, static_cast<const uint4*>(a.k_new),
                       static_cast<const uint4*>(a.v_new), a.slot_mapping,
                       static_cast<uint8_t*>(a.kv), a.num_tokens, a.num_kv_heads,
                       chunks_per_row, capacity, items);
  else
    hipLaunchKernelGGL(kv_append_kernel<4>, dim3((unsigned)blocks), dim3(kAppendWaves * kWave),
                       0, a.stream, static_cast<const uint4*>(a.k_new),
                       static_cast<const uint4*>(a.v_new), a.slot_mapping,
                       static_cast<uint8_t*>(a.kv), a.num_tokens, a.num_kv_heads,
                       chunks_per_row, capacity, items);
  trace_after(a.stream);
  return hipGetLastError();
}

}  // namespace kvattn
