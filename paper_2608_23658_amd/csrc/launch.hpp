// Host-side launch descriptors shared by the C ABI and the kernel files.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace kvattn {

struct DecodeArgs {
  const void* q;
  const void* kv;
  const void* kv2 = nullptr;   // second tensor of a two-tensor layer (ids >= num_base)
  int num_base = 0;
  int num_blocks;
  const int32_t* block_table;
  const int32_t* seq_lens;
  void* out;
  int num_seqs, num_q_heads, num_kv_heads, head_dim;
  int max_blocks, max_seq_len, split_tokens;
  float scale;
  bool bf16;
  void* workspace;
  size_t ws_ml_offset;   // byte offset of the (m, l) partials in the workspace
  hipStream_t stream;
};

struct PrefillArgs {
  const void* q;
  const void* kv;
  int num_blocks;
  const int32_t* block_table;
  const int32_t* seq_lens;
  const int32_t* cu_seqlens_q;
  void* out;
  int num_seqs, total_q_tokens, num_q_heads, num_kv_heads, head_dim;
  int max_blocks, max_seq_len;
  float scale;
  void* workspace;
  size_t workspace_bytes;
  hipStream_t stream;
};

struct AppendArgs {
  const void* k_new;
  const void* v_new;
  const int32_t* slot_mapping;
  void* kv;
  int num_blocks, num_tokens, num_kv_heads, head_dim;
  int esz;   // bytes per element: 2 (bf16) or 4 (fp32)
  hipStream_t stream;
};

// Layer base pointers passed by value to the block-copy kernel.
constexpr int kMaxCopyLayers = 128;
struct CopyLayers {
  void* p[kMaxCopyLayers];
};

struct CopyArgs {
  void* const* layers;   // host array of num_layers device pointers
  int num_layers, num_blocks, n;
  size_t block_bytes;
  const int32_t* src;
  const int32_t* dst;
  hipStream_t stream;
};

// Tracing hooks around each kernel launch (no-ops unless a trace is installed).
void trace_before(hipStream_t stream, const char* kernel);
void trace_after(hipStream_t stream);

hipError_t launch_decode(const DecodeArgs& a);
hipError_t launch_prefill(const PrefillArgs& a);
hipError_t launch_append(const AppendArgs& a);
hipError_t launch_copy_blocks(const CopyArgs& a);

// Fewest query rows per prefill work tile (per query head): 32 at group
// size 8; the workspace's tile list is sized for it.
constexpr int kPrefillRows = 32;

}  // namespace kvattn
