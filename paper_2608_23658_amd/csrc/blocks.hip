// Copying whole KV blocks from one block id to another in every layer: how a
// caller drains the elastic block-id range before decommitting it (the
// paper, Section 3 "Controller": decommitting first drains the elastic blocks,
// syncs, then unmaps). One workgroup per (pair, layer); 16-byte loads and
// stores, coalesced over the block.

#include "common.hpp"
#include "launch.hpp"

namespace kvattn {

__global__ __launch_bounds__(256) void copy_blocks_kernel(CopyLayers layers,
                                                          const int* __restrict__ src,
                                                          const int* __restrict__ dst,
                                                          int num_blocks, size_t block_bytes) {
  const int pair = blockIdx.x;
  const int s = src[pair], d = dst[pair];
  if (s < 0 || s >= num_blocks || d < 0 || d >= num_blocks || s == d) return;
  uint8_t* base = static_cast<uint8_t*>(layers.p[blockIdx.y]);
  const uint4* from = reinterpret_cast<const uint4*>(base + (size_t)s * block_bytes);
  uint4* to = reinterpret_cast<uint4*>(base + (size_t)d * block_bytes);
  const size_t n16 = block_bytes / 16;
  for (size_t i = threadIdx.x; i < n16; i += 256) to[i] = from[i];
}

hipError_t launch_copy_blocks(const CopyArgs& a) {
  if (a.n == 0 || a.num_layers == 0) return hipSuccess;
  for (int l0 = 0; l0 < a.num_layers; l0 += kMaxCopyLayers) {
    CopyLayers layers = {};
    const int nl = a.num_layers - l0 < kMaxCopyLayers ? a.num_layers - l0 : kMaxCopyLayers;
    for (int l = 0; l < nl; ++l) layers.p[l] = a.layers[l0 + l];
    trace_before(a.stream, "copy_blocks");
    hipLaunchKernelGGL(copy_blocks_kernel, dim3(a.n, nl), dim3(256), 0, a.stream, layers,
                       a.src, a.dst, a.num_blocks, a.block_bytes);
    trace_after(a.stream);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace kvattn
