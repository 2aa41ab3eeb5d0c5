// C-ABI entry points for paged-KV attention: argument checks, workspace
// sizing and kernel launches. No allocation happens here.

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <mutex>
#include <string>
#include <vector>

#include "abi_internal.hpp"
#include "kvattn.h"
#include "launch.hpp"

namespace kvattn {

namespace {
thread_local std::string g_error;
}

int set_error(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_error = buf;
  return code;
}

void clear_error() { g_error.clear(); }

namespace {
struct Trace {
  void* const* events = nullptr;
  int capacity = 0;
  int used = 0;
  std::vector<std::string> names;
};
thread_local Trace g_trace;
thread_local std::vector<std::string> g_last_names;
}  // namespace

void trace_before(hipStream_t stream, const char* kernel) {
  Trace& t = g_trace;
  if (!t.events || t.used + 2 > t.capacity) return;
  (void)hipEventRecord(static_cast<hipEvent_t>(t.events[t.used]), stream);
  t.names.emplace_back(kernel);
}

void trace_after(hipStream_t stream) {
  Trace& t = g_trace;
  if (!t.events || t.used + 2 > t.capacity) return;
  (void)hipEventRecord(static_cast<hipEvent_t>(t.events[t.used + 1]), stream);
  t.used += 2;
}

}  // namespace kvattn

using kvattn::clear_error;
using kvattn::set_error;

namespace {

constexpr int kAbiVersion = 1;
constexpr int kDecodeSplitTokens = 1024;

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

struct DecodeWs {
  size_t ml_offset;
  size_t total;
};

bool decode_ws(int num_seqs, int num_q_heads, int head_dim, int max_seq_len, DecodeWs* w) {
  if (num_seqs < 0 || num_q_heads <= 0 || head_dim <= 0 || max_seq_len < 0) return false;
  const int split = kvattn_decode_split_tokens(max_seq_len);
  const size_t splits = max_seq_len > 0 ? (size_t)(max_seq_len + split - 1) / split : 1;
  const size_t n = (size_t)num_seqs * num_q_heads * splits;
  w->ml_offset = align256(n * head_dim * sizeof(float));
  w->total = w->ml_offset + align256(n * 2 * sizeof(float));
  if (w->total == 0) w->total = 256;
  return true;
}

bool group_ok(int hq, int hkv, int max_group) {
  if (hq <= 0 || hkv <= 0 || hq % hkv) return false;
  const int g = hq / hkv;
  return g == 1 || g == 2 || g == 4 || (g == 8 && max_group >= 8);
}

int hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return KV_OK;
  (void)hipGetLastError();   // the runtime keeps the error sticky: clear it for the caller
  return set_error(KV_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

}  // namespace

extern "C" const char* kv_last_error(void) { return kvattn::g_error.c_str(); }

extern "C" int kvattn_abi_version(void) { return kAbiVersion; }

extern "C" int kvattn_trace_begin(void* const* events, int capacity) {
  clear_error();
  if (!events || capacity < 2)
    return set_error(KV_ERR_INVALID, "kvattn_trace_begin: need at least 2 events");
  kvattn::g_trace = kvattn::Trace{};
  kvattn::g_trace.events = events;
  kvattn::g_trace.capacity = capacity;
  return KV_OK;
}

extern "C" int kvattn_trace_end(int* events_used) {
  clear_error();
  if (events_used) *events_used = kvattn::g_trace.used;
  kvattn::g_last_names = kvattn::g_trace.names;
  kvattn::g_trace = kvattn::Trace{};
  return KV_OK;
}

extern "C" const char* kvattn_trace_kernel_name(int i) {
  if (i < 0 || i >= (int)kvattn::g_last_names.size()) return "";
  return kvattn::g_last_names[i].c_str();
}

extern "C" int kvattn_decode_split_tokens(int max_seq_len) {
  (void)max_seq_len;
  return kDecodeSplitTokens;
}

extern "C" size_t kvattn_decode_workspace_bytes(int num_seqs, int num_q_heads, int head_dim,
                                                int max_seq_len) {
  DecodeWs w;
  return decode_ws(num_seqs, num_q_heads, head_dim, max_seq_len, &w) ? w.total : 0;
}

namespace {

// Checks a decode call and fills the launch descriptor; the workspace is
// checked only when check_workspace is set.
int decode_check(const char* fn, const void* q, const void* kv_layer, const void* kv2,
                 int num_base, int num_blocks, const int32_t* block_table,
                 const int32_t* seq_lens, void* out, int num_seqs, int num_q_heads,
                 int num_kv_heads, int head_dim, int block_size, int max_blocks_per_seq,
                 int max_seq_len, float scale, kv_dtype dtype, void* workspace,
                 size_t workspace_bytes, bool check_workspace, void* stream,
                 kvattn::DecodeArgs* a);

int decode_launch(const char* fn, const kvattn::DecodeArgs& a);

int decode_common(const char* fn, const void* q, const void* kv_layer, const void* kv2,
                  int num_base, int num_blocks, const int32_t* block_table,
                  const int32_t* seq_lens, void* out, int num_seqs, int num_q_heads,
                  int num_kv_heads, int head_dim, int block_size, int max_blocks_per_seq,
                  int max_seq_len, float scale, kv_dtype dtype, void* workspace,
                  size_t workspace_bytes, void* stream) {
  kvattn::DecodeArgs a;
  const int rc = decode_check(fn, q, kv_layer, kv2, num_base, num_blocks, block_table, seq_lens,
                              out, num_seqs, num_q_heads, num_kv_heads, head_dim, block_size,
                              max_blocks_per_seq, max_seq_len, scale, dtype, workspace,
                              workspace_bytes, true, stream, &a);
  if (rc != KV_OK || num_seqs == 0) return rc;
  return decode_launch(fn, a);
}

}  // namespace

extern "C" int kvattn_decode(const void* q, const void* kv_layer, int num_blocks,
                             const int32_t* block_table, const int32_t* seq_lens, void* out,
                             int num_seqs, int num_q_heads, int num_kv_heads, int head_dim,
                             int block_size, int max_blocks_per_seq, int max_seq_len,
                             float scale, kv_dtype dtype, void* workspace,
                             size_t workspace_bytes, void* stream) {
  clear_error();
  return decode_common("kvattn_decode", q, kv_layer, nullptr, 0, num_blocks, block_table,
                       seq_lens, out, num_seqs, num_q_heads, num_kv_heads, head_dim,
                       block_size, max_blocks_per_seq, max_seq_len, scale, dtype, workspace,
                       workspace_bytes, stream);
}

extern "C" int kvattn_decode_two_tensor(const void* q, const void* kv_base, int num_base_blocks,
                                        const void* kv_elastic, int num_elastic_blocks,
                                        const int32_t* block_table, const int32_t* seq_lens,
                                        void* out, int num_seqs, int num_q_heads,
                                        int num_kv_heads, int head_dim, int block_size,
                                        int max_blocks_per_seq, int max_seq_len, float scale,
                                        kv_dtype dtype, void* workspace, size_t workspace_bytes,
                                        void* stream) {
  clear_error();
  if (num_base_blocks <= 0 || num_elastic_blocks <= 0 ||
      (long long)num_base_blocks + num_elastic_blocks > 0x7fffffffLL)
    return set_error(KV_ERR_INVALID, "kvattn_decode_two_tensor: %d base + %d elastic blocks",
                     num_base_blocks, num_elastic_blocks);
  if (dtype != KV_BF16 || head_dim != 128)
    return set_error(KV_ERR_UNSUPPORTED,
                     "kvattn_decode_two_tensor: built for bf16 with head_dim 128 only");
  if (num_seqs > 0 && (!kv_elastic || !aligned16(kv_elastic)))
    return set_error(KV_ERR_INVALID,
                     "kvattn_decode_two_tensor: kv_elastic null or not 16-byte aligned");
  return decode_common("kvattn_decode_two_tensor", q, kv_base, kv_elastic, num_base_blocks,
                       num_base_blocks + num_elastic_blocks, block_table, seq_lens, out,
                       num_seqs, num_q_heads, num_kv_heads, head_dim, block_size,
                       max_blocks_per_seq, max_seq_len, scale, dtype, workspace,
                       workspace_bytes, stream);
}

namespace {

int decode_check(const char* fn, const void* q, const void* kv_layer, const void* kv2,
                 int num_base, int num_blocks, const int32_t* block_table,
                 const int32_t* seq_lens, void* out, int num_seqs, int num_q_heads,
                 int num_kv_heads, int head_dim, int block_size, int max_blocks_per_seq,
                 int max_seq_len, float scale, kv_dtype dtype, void* workspace,
                 size_t workspace_bytes, bool check_workspace, void* stream,
                 kvattn::DecodeArgs* out_args) {
  if (num_seqs < 0) return set_error(KV_ERR_INVALID, "%s: num_seqs %d < 0", fn, num_seqs);
  if (dtype != KV_F32 && dtype != KV_BF16)
    return set_error(KV_ERR_INVALID, "%s: unknown dtype %d", fn, (int)dtype);
  if (num_q_heads <= 0 || num_kv_heads <= 0 || num_q_heads % num_kv_heads)
    return set_error(KV_ERR_INVALID, "%s: %d query heads over %d kv heads", fn,
                     num_q_heads, num_kv_heads);
  if (!group_ok(num_q_heads, num_kv_heads, 8))
    return set_error(KV_ERR_UNSUPPORTED, "%s: group size %d not built", fn,
                     num_q_heads / num_kv_heads);
  if (head_dim != 64 && !(head_dim == 128 && dtype == KV_BF16))
    return set_error(KV_ERR_UNSUPPORTED, "%s: head_dim %d not built for %s", fn,
                     head_dim, dtype == KV_BF16 ? "bf16" : "fp32");
  if (block_size != 16)
    return set_error(KV_ERR_UNSUPPORTED, "%s: block_size %d not built", fn, block_size);
  if (max_blocks_per_seq <= 0 || max_seq_len < 0 ||
      (long long)max_seq_len > (long long)max_blocks_per_seq * block_size)
    return set_error(KV_ERR_INVALID,
                     "%s: max_seq_len %d does not fit %d blocks of %d tokens", fn,
                     max_seq_len, max_blocks_per_seq, block_size);
  if (num_blocks <= 0) return set_error(KV_ERR_INVALID, "%s: num_blocks %d", fn, num_blocks);
  if (!std::isfinite(scale)) return set_error(KV_ERR_INVALID, "%s: scale not finite", fn);
  if (num_kv_heads > 65535 || num_seqs > 65535)
    return set_error(KV_ERR_UNSUPPORTED, "%s: grid too large", fn);
  if (num_seqs == 0) return KV_OK;
  if (!q || !kv_layer || !block_table || !seq_lens || !out)
    return set_error(KV_ERR_INVALID, "%s: null pointer argument", fn);
  if (!aligned16(q) || !aligned16(kv_layer) || !aligned16(out))
    return set_error(KV_ERR_INVALID, "%s: q, kv_layer and out must be 16-byte aligned", fn);
  DecodeWs w;
  decode_ws(num_seqs, num_q_heads, head_dim, max_seq_len, &w);
  if (check_workspace) {
    if (!workspace) return set_error(KV_ERR_INVALID, "%s: null workspace", fn);
    if (!aligned16(workspace))
      return set_error(KV_ERR_INVALID, "%s: workspace must be 16-byte aligned", fn);
    if (workspace_bytes < w.total)
      return set_error(KV_ERR_INVALID, "%s: workspace %zu bytes < %zu needed", fn,
                       workspace_bytes, w.total);
  }
  kvattn::DecodeArgs& a = *out_args;
  a.q = q;
  a.kv = kv_layer;
  a.num_blocks = num_blocks;
  a.block_table = block_table;
  a.seq_lens = seq_lens;
  a.out = out;
  a.num_seqs = num_seqs;
  a.num_q_heads = num_q_heads;
  a.num_kv_heads = num_kv_heads;
  a.head_dim = head_dim;
  a.max_blocks = max_blocks_per_seq;
  a.max_seq_len = max_seq_len;
  a.split_tokens = kvattn_decode_split_tokens(max_seq_len);
  a.scale = scale;
  a.bf16 = dtype == KV_BF16;
  a.workspace = workspace;
  a.ws_ml_offset = w.ml_offset;
  a.stream = static_cast<hipStream_t>(stream);
  a.kv2 = kv2;
  a.num_base = num_base;
  return KV_OK;
}

int decode_launch(const char* fn, const kvattn::DecodeArgs& a) {
  const hipError_t e = kvattn::launch_decode(a);
  if (e == hipErrorNotSupported) return set_error(KV_ERR_UNSUPPORTED, "%s: not built", fn);
  return hip_status(e, fn);
}

}  // namespace

extern "C" size_t kvattn_prefill_workspace_bytes(int num_seqs, int total_q_tokens,
                                                 int num_q_heads, int head_dim) {
  if (num_seqs < 0 || total_q_tokens < 0 || num_q_heads <= 0 || head_dim <= 0) return 0;
  // Work-tile list: one int2 per tile of kPrefillRows query rows of a sequence.
  const size_t tiles = (size_t)total_q_tokens / kvattn::kPrefillRows + num_seqs + 1;
  return align256(tiles * 2 * sizeof(int32_t) + 16);
}

extern "C" int kvattn_prefill_chunk(const void* q, const void* kv_layer, int num_blocks,
                                    const int32_t* block_table, const int32_t* seq_lens,
                                    const int32_t* cu_seqlens_q, void* out, int num_seqs,
                                    int total_q_tokens, int max_num_batched_tokens,
                                    int num_q_heads, int num_kv_heads, int head_dim,
                                    int block_size, int max_blocks_per_seq, int max_seq_len,
                                    float scale, kv_dtype dtype, void* workspace,
                                    size_t workspace_bytes, void* stream) {
  clear_error();
  if (dtype == KV_F32)
    return set_error(KV_ERR_UNSUPPORTED, "kvattn_prefill_chunk: fp32 prefill is not built");
  if (dtype != KV_BF16)
    return set_error(KV_ERR_INVALID, "kvattn_prefill_chunk: unknown dtype %d", (int)dtype);
  if (num_seqs < 0 || total_q_tokens < 0)
    return set_error(KV_ERR_INVALID, "kvattn_prefill_chunk: negative sizes");
  if (total_q_tokens > max_num_batched_tokens)
    return set_error(KV_ERR_INVALID,
                     "kvattn_prefill_chunk: %d new tokens exceed max_num_batched_tokens %d",
                     total_q_tokens, max_num_batched_tokens);
  if (num_q_heads <= 0 || num_kv_heads <= 0 || num_q_heads % num_kv_heads)
    return set_error(KV_ERR_INVALID, "kvattn_prefill_chunk: %d query heads over %d kv heads",
                     num_q_heads, num_kv_heads);
  if (!group_ok(num_q_heads, num_kv_heads, 8))
    return set_error(KV_ERR_UNSUPPORTED, "kvattn_prefill_chunk: group size %d not built",
                     num_q_heads / num_kv_heads);
  if (head_dim != 128)
    return set_error(KV_ERR_UNSUPPORTED, "kvattn_prefill_chunk: head_dim %d not built",
                     head_dim);
  if (block_size != 16)
    return set_error(KV_ERR_UNSUPPORTED, "kvattn_prefill_chunk: block_size %d not built",
                     block_size);
  if (max_blocks_per_seq <= 0 || max_seq_len < 0 ||
      (long long)max_seq_len > (long long)max_blocks_per_seq * block_size)
    return set_error(KV_ERR_INVALID,
                     "kvattn_prefill_chunk: max_seq_len %d does not fit %d blocks of %d tokens",
                     max_seq_len, max_blocks_per_seq, block_size);
  if (num_blocks <= 0)
    return set_error(KV_ERR_INVALID, "kvattn_prefill_chunk: num_blocks %d", num_blocks);
  if (!std::isfinite(scale))
    return set_error(KV_ERR_INVALID, "kvattn_prefill_chunk: scale not finite");
  if (num_kv_heads > 65535) return set_error(KV_ERR_UNSUPPORTED, "kvattn_prefill_chunk: grid");
  if (num_seqs == 0 || total_q_tokens == 0) return KV_OK;
  if (!q || !kv_layer || !block_table || !seq_lens || !cu_seqlens_q || !out || !workspace)
    return set_error(KV_ERR_INVALID, "kvattn_prefill_chunk: null pointer argument");
  if (!aligned16(q) || !aligned16(kv_layer) || !aligned16(out) || !aligned16(workspace))
    return set_error(KV_ERR_INVALID, "kvattn_prefill_chunk: q, kv_layer, out and workspace "
                                     "must be 16-byte aligned");
  const size_t need = kvattn_prefill_workspace_bytes(num_seqs, total_q_tokens, num_q_heads,
                                                     head_dim);
  if (workspace_bytes < need)
    return set_error(KV_ERR_INVALID, "kvattn_prefill_chunk: workspace %zu bytes < %zu needed",
                     workspace_bytes, need);
  kvattn::PrefillArgs a;
  a.q = q;
  a.kv = kv_layer;
  a.num_blocks = num_blocks;
  a.block_table = block_table;
  a.seq_lens = seq_lens;
  a.cu_seqlens_q = cu_seqlens_q;
  a.out = out;
  a.num_seqs = num_seqs;
  a.total_q_tokens = total_q_tokens;
  a.num_q_heads = num_q_heads;
  a.num_kv_heads = num_kv_heads;
  a.head_dim = head_dim;
  a.max_blocks = max_blocks_per_seq;
  a.max_seq_len = max_seq_len;
  a.scale = scale;
  a.workspace = workspace;
  a.workspace_bytes = workspace_bytes;
  a.stream = static_cast<hipStream_t>(stream);
  const hipError_t e = kvattn::launch_prefill(a);
  if (e == hipErrorNotSupported)
    return set_error(KV_ERR_UNSUPPORTED, "kvattn_prefill_chunk: kernel not built");
  return hip_status(e, "kvattn_prefill_chunk launch");
}

extern "C" int kvattn_kv_append(const void* k_new, const void* v_new,
                                const int32_t* slot_mapping, void* kv_layer, int num_blocks,
                                int num_tokens, int num_kv_heads, int head_dim, int block_size,
                                kv_dtype dtype, void* stream) {
  clear_error();
  if (dtype != KV_F32 && dtype != KV_BF16)
    return set_error(KV_ERR_INVALID, "kvattn_kv_append: unknown dtype %d", (int)dtype);
  const int esz = dtype == KV_BF16 ? 2 : 4;
  if (num_tokens < 0) return set_error(KV_ERR_INVALID, "kvattn_kv_append: num_tokens < 0");
  if (num_kv_heads <= 0 || head_dim <= 0 || (head_dim * esz) % 16)
    return set_error(KV_ERR_INVALID,
                     "kvattn_kv_append: %d kv heads of dim %d (a row must be whole 16-byte "
                     "chunks)", num_kv_heads, head_dim);
  if (head_dim * esz % 64 || head_dim * esz > 512)
    return set_error(KV_ERR_UNSUPPORTED,
                     "kvattn_kv_append: rows must be 64 to 512 bytes in steps of 64, not %d",
                     head_dim * esz);
  if (block_size != 16)
    return set_error(KV_ERR_UNSUPPORTED, "kvattn_kv_append: block_size %d not built",
                     block_size);
  if (num_blocks <= 0 || (long long)num_blocks * block_size > 0x7fffffffLL)
    return set_error(KV_ERR_INVALID, "kvattn_kv_append: num_blocks %d", num_blocks);
  if (num_tokens == 0) return KV_OK;
  if (!k_new || !v_new || !slot_mapping || !kv_layer)
    return set_error(KV_ERR_INVALID, "kvattn_kv_append: null pointer argument");
  if (!aligned16(k_new) || !aligned16(v_new) || !aligned16(kv_layer))
    return set_error(KV_ERR_INVALID,
                     "kvattn_kv_append: k_new, v_new and kv_layer must be 16-byte aligned");
  kvattn::AppendArgs a;
  a.k_new = k_new;
  a.v_new = v_new;
  a.slot_mapping = slot_mapping;
  a.kv = kv_layer;
  a.num_blocks = num_blocks;
  a.num_tokens = num_tokens;
  a.num_kv_heads = num_kv_heads;
  a.head_dim = head_dim;
  a.esz = esz;
  a.stream = static_cast<hipStream_t>(stream);
  const hipError_t e = kvattn::launch_append(a);
  if (e == hipErrorNotSupported)
    return set_error(KV_ERR_UNSUPPORTED,
                     "kvattn_kv_append: rows must be 64 to 512 bytes in steps of 64");
  return hip_status(e, "kvattn_kv_append launch");
}

extern "C" int kvattn_copy_blocks(void* const* layers, int num_layers, int num_blocks,
                                  size_t block_bytes, const int32_t* src_ids,
                                  const int32_t* dst_ids, int n, void* stream) {
  clear_error();
  if (num_layers < 0 || n < 0 || num_blocks <= 0)
    return set_error(KV_ERR_INVALID, "kvattn_copy_blocks: %d layers, %d pairs, %d blocks",
                     num_layers, n, num_blocks);
  if (block_bytes == 0 || block_bytes % 16)
    return set_error(KV_ERR_INVALID, "kvattn_copy_blocks: block_bytes %zu not a multiple of 16",
                     block_bytes);
  if (n > 0x7fffffff / 2)
    return set_error(KV_ERR_UNSUPPORTED, "kvattn_copy_blocks: too many pairs");
  if (n == 0 || num_layers == 0) return KV_OK;
  if (!layers || !src_ids || !dst_ids)
    return set_error(KV_ERR_INVALID, "kvattn_copy_blocks: null pointer argument");
  for (int l = 0; l < num_layers; ++l)
    if (!layers[l] || !aligned16(layers[l]))
      return set_error(KV_ERR_INVALID, "kvattn_copy_blocks: layer %d pointer null or not "
                                       "16-byte aligned", l);
  kvattn::CopyArgs a;
  a.layers = layers;
  a.num_layers = num_layers;
  a.num_blocks = num_blocks;
  a.n = n;
  a.block_bytes = block_bytes;
  a.src = src_ids;
  a.dst = dst_ids;
  a.stream = static_cast<hipStream_t>(stream);
  return hip_status(kvattn::launch_copy_blocks(a), "kvattn_copy_blocks launch");
}

// ---------------------------------------------------------------------------
// Decode without a caller workspace, for callers that cannot allocate device
// memory (code under HIP graph capture, tight serving loops). The split-K
// partials live in a file-scope device array of fixed size instead. Each GPU
// the library runs on holds its own copy of the array, at its own address,
// until the process ends. In host code the array's name is only a host-side
// stand-in, so the device address is looked up once per device with
// hipGetSymbolAddress and only that address is passed to the kernels.

namespace {

constexpr size_t kNoAllocScratchBytes = size_t(32) << 20;
constexpr int kMaxDevices = 64;

__device__ __align__(256) uint8_t scratch[kNoAllocScratchBytes];

std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of the current device's copy of `scratch`, looked up with
// that device current on the first call on it and kept for later calls.
int scratch_on_current_device(const char* fn, void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_status(e, fn);
  if (dev < 0 || dev >= kMaxDevices)
    return set_error(KV_ERR_UNSUPPORTED, "%s: device %d beyond the %d the library tracks", fn,
                     dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_status(e, fn);
    if (!ptr) return set_error(KV_ERR_HIP, "%s: hipGetSymbolAddress gave no address", fn);
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return KV_OK;
}

}  // namespace

extern "C" size_t kvattn_decode_noalloc_max_scratch_bytes(void) { return kNoAllocScratchBytes; }

extern "C" int kvattn_decode_noalloc(const void* q, const void* kv_layer, int num_blocks,
                                     const int32_t* block_table, const int32_t* seq_lens,
                                     void* out, int num_seqs, int num_q_heads, int num_kv_heads,
                                     int head_dim, int block_size, int max_blocks_per_seq,
                                     int max_seq_len, float scale, kv_dtype dtype,
                                     void* stream) {
  clear_error();
  const char* fn = "kvattn_decode_noalloc";
  DecodeWs w;
  if (!decode_ws(num_seqs, num_q_heads, head_dim, max_seq_len, &w))
    return set_error(KV_ERR_INVALID, "%s: %d sequences, %d query heads, head_dim %d, "
                                     "max_seq_len %d", fn, num_seqs, num_q_heads, head_dim,
                     max_seq_len);
  if (w.total > kNoAllocScratchBytes)
    return set_error(KV_ERR_INVALID,
                     "%s: the batch needs %zu bytes of split partials, more than the %zu-byte "
                     "static scratch; use kvattn_decode with a workspace", fn, w.total,
                     kNoAllocScratchBytes);
  kvattn::DecodeArgs a;
  int rc = decode_check(fn, q, kv_layer, nullptr, 0, num_blocks, block_table, seq_lens, out,
                        num_seqs, num_q_heads, num_kv_heads, head_dim, block_size,
                        max_blocks_per_seq, max_seq_len, scale, dtype, nullptr, 0, false,
                        stream, &a);
  if (rc != KV_OK || num_seqs == 0) return rc;
  rc = scratch_on_current_device(fn, &a.workspace);
  if (rc != KV_OK) return rc;
  return decode_launch(fn, a);
}
