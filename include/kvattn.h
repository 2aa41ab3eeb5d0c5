/*
 * kvattn: attention over a block-indexed paged KV cache on one MI355X
 * (gfx950), and the elastic per-layer VMM pool the cache lives in.
 *
 * C ABI: plain pointers and sizes only. Every entry point returns a
 * kv_status; a failure leaves a message readable via kv_last_error()
 * (thread-local). Nothing crosses the boundary as an exception or abort.
 *
 * ---------------------------------------------------------------------------
 * Paged KV layout of one layer (the paper, Section 3 "The contiguity
 * constraint": one contiguous tensor per layer, indexed by block id through a
 * single base pointer). Block-major, so that the top block ids are the top of
 * the address range, which is where the elastic sub-range maps (Section 3,
 * "Two handles, one virtual range"):
 *
 *   layer[num_blocks][2 (K=0, V=1)][num_kv_heads][block_size * head_dim]
 *
 * One (block, K/V, kv head) tile of block_size * head_dim elements:
 *   K tile, chunk-major: token slot r, dim j at
 *       ((j / VEC) * block_size + r) * VEC + (j % VEC),  VEC = 16 / element size
 *   V tile, dim-major (transposed): token slot r, dim j at  j * block_size + r
 * Element type is the call's kv_dtype (fp32 or bf16). Token t of sequence s
 * is slot t % block_size of block block_table[s * max_blocks_per_seq + t /
 * block_size].
 *
 * Attention computed (Section 5, "Why the penalty is small": a chunk attends
 * to all prior context, decode is one token per sequence): for sequence s
 * with L_s context tokens of which the last n_s are new, new row i (absolute
 * position p = L_s - n_s + i), query head h, kv head g = h / (Hq / Hkv):
 *   out = sum_{t <= p} softmax_t(scale * q . K_s[t]) V_s[t]
 * Softmax accumulates in fp32; bf16 outputs are rounded to nearest even.
 * ---------------------------------------------------------------------------
 */
#ifndef KVATTN_H
#define KVATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  KV_OK = 0,
  KV_ERR_INVALID = -1,      /* bad argument: shape, alignment, size, null pointer */
  KV_ERR_UNSUPPORTED = -2,  /* valid but not built: head_dim, group size, dtype */
  KV_ERR_HIP = -3,          /* a HIP runtime call failed */
  KV_ERR_OOM = -4,          /* physical memory could not be created */
  KV_ERR_STATE = -5         /* call not allowed in the pool's current state */
} kv_status;

typedef enum { KV_F32 = 0, KV_BF16 = 1 } kv_dtype;

/* Message of the calling thread's last failure ("" if none). Owned by the
 * library; valid until the thread's next call into it. */
const char* kv_last_error(void);

/* ABI version, bumped on any signature or layout change. */
int kvattn_abi_version(void);

/* ------------------------------------------------------------------------- */
/* Decode: one new query token per sequence (Section 5). Split-K over the
 * context: each (sequence, kv head, split of the context) is one workgroup,
 * whose partial softmax state is merged by a second kernel.
 *
 * Workspace: device memory of at least kvattn_decode_workspace_bytes(...)
 * bytes, owned by the caller, 256-byte aligned, no initial contents needed,
 * must not be used by another call in flight. Returns 0 if the sizes are
 * invalid. */
size_t kvattn_decode_workspace_bytes(int num_seqs, int num_q_heads, int head_dim,
                                     int max_seq_len);

/* Context tokens per split used by kvattn_decode for a batch whose longest
 * sequence is max_seq_len (a multiple of 64; depends on nothing else, so a
 * sequence's arithmetic depends only on its own length). */
int kvattn_decode_split_tokens(int max_seq_len);

/*
 * q            device, [num_seqs][num_q_heads][head_dim] of dtype, 16-B aligned
 * kv_layer     device, base of one layer in the layout above, 16-B aligned
 * num_blocks   blocks in the layer; block ids outside [0, num_blocks) are
 *              skipped (they contribute nothing) rather than read
 * block_table  device int32 [num_seqs][max_blocks_per_seq]; entries past
 *              ceil(seq_len / block_size) are never read (pad with -1)
 * seq_lens     device int32 [num_seqs], 0 <= seq_len <= max_seq_len and
 *              <= max_blocks_per_seq * block_size; the query token is the
 *              last of its sequence. A sequence of length 0 gets zeros.
 * out          device, [num_seqs][num_q_heads][head_dim] of dtype, 16-B aligned
 * scale        softmax scale (1/sqrt(head_dim) for standard attention)
 * stream       hipStream_t to enqueue on (NULL: the null stream)
 *
 * Supported: block_size 16; num_q_heads / num_kv_heads in {1, 2, 4, 8}; bf16
 * with head_dim 64 or 128, fp32 with head_dim 64. Asynchronous: returns after enqueueing. The
 * library allocates nothing.
 */
int kvattn_decode(const void* q, const void* kv_layer, int num_blocks,
                  const int32_t* block_table, const int32_t* seq_lens, void* out,
                  int num_seqs, int num_q_heads, int num_kv_heads, int head_dim,
                  int block_size, int max_blocks_per_seq, int max_seq_len, float scale,
                  kv_dtype dtype, void* workspace, size_t workspace_bytes, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * decode as kvattn_decode, same arguments minus the workspace, and the same
 * kernels and results. The split-K partials go to a fixed device array inside
 * the library instead of a caller workspace:
 *   - its size is kvattn_decode_noalloc_max_scratch_bytes() (32 MiB); a batch
 *     whose partials need more (kvattn_decode_workspace_bytes(...) above that)
 *     is refused with KV_ERR_INVALID before anything is launched (256
 *     sequences of 32 query heads, head_dim 128, up to 4096 tokens, fit);
 *   - each GPU the library runs on holds its own copy from its first call on
 *     that GPU until the process ends; the array's device address is looked
 *     up (hipGetSymbolAddress) on that first call, with the current device
 *     being the one the stream belongs to;
 *   - it allocates nothing and needs no initial contents, but every call on a
 *     GPU shares that GPU's array: calls that overlap in time on one GPU
 *     (different streams, or host threads) race and give undefined results.
 *     Calls on one stream are ordered and safe.
 * Errors as for kvattn_decode; KV_ERR_HIP if the array's address cannot be
 * found. Asynchronous. */
size_t kvattn_decode_noalloc_max_scratch_bytes(void);
int kvattn_decode_noalloc(const void* q, const void* kv_layer, int num_blocks,
                          const int32_t* block_table, const int32_t* seq_lens, void* out,
                          int num_seqs, int num_q_heads, int num_kv_heads, int head_dim,
                          int block_size, int max_blocks_per_seq, int max_seq_len, float scale,
                          kv_dtype dtype, void* stream);

/* The rejected alternative (Section 3, "The contiguity constraint": split the
 * KV into two tensors and make the kernel read both). Same as kvattn_decode
 * but block ids below num_base_blocks address kv_base and ids from
 * num_base_blocks to num_base_blocks + num_elastic_blocks - 1 address
 * kv_elastic at id - num_base_blocks; both tensors use the per-block layout
 * above. Built for bf16 with head_dim 128 (KV_ERR_UNSUPPORTED otherwise); it
 * exists to measure the cost of the second pointer against the one-range
 * layer the elastic pool gives. */
int kvattn_decode_two_tensor(const void* q, const void* kv_base, int num_base_blocks,
                             const void* kv_elastic, int num_elastic_blocks,
                             const int32_t* block_table, const int32_t* seq_lens, void* out,
                             int num_seqs, int num_q_heads, int num_kv_heads, int head_dim,
                             int block_size, int max_blocks_per_seq, int max_seq_len,
                             float scale, kv_dtype dtype, void* workspace,
                             size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------- */
/* Kernel tracing. While a trace buffer is installed on the calling thread,
 * every kernel the library launches from that thread is bracketed by
 * hipEventRecord of the next two events of the buffer (hipEvent_t handles
 * owned by the caller) on the launch stream, so per-kernel durations can be
 * read with hipEventElapsedTime. Launches beyond the buffer are not traced.
 * kvattn_trace_end uninstalls the buffer and reports the events used. */
int kvattn_trace_begin(void* const* events, int capacity);
int kvattn_trace_end(int* events_used);
/* Name of the kernel traced by events 2i and 2i+1 of the last trace ("" if none). */
const char* kvattn_trace_kernel_name(int i);

/* ------------------------------------------------------------------------- */
/* Chunked prefill (Section 5 and Section 1: max_num_batched_tokens bounds the
 * new tokens of one step; a chunk attends causally to itself and to all of
 * its sequence's earlier tokens, which are already in the cache).
 *
 * q             device, [total_q_tokens][num_q_heads][head_dim] bf16, 16-B aligned
 * kv_layer      as for decode; the chunk's own K/V must already be written
 * block_table   as for decode
 * seq_lens      device int32 [num_seqs]: context length INCLUDING the chunk
 * cu_seqlens_q  device int32 [num_seqs + 1], nondecreasing from 0: the chunk of
 *               sequence s is rows [cu[s], cu[s+1]) of q and out, with
 *               cu[s+1] - cu[s] <= seq_lens[s]; cu[num_seqs] == total_q_tokens
 * out           device, [total_q_tokens][num_q_heads][head_dim] bf16
 * max_num_batched_tokens  the step's token budget: total_q_tokens must not
 *               exceed it (KV_ERR_INVALID otherwise); it sizes no buffer and
 *               never changes the arithmetic
 * workspace     device scratch of kvattn_prefill_workspace_bytes(...) bytes
 *
 * Causal alignment is bottom-right: row i of sequence s sees keys
 * 0 .. seq_lens[s] - n_s + i. Supported: bf16, block_size 16, head_dim 128,
 * num_q_heads / num_kv_heads in {1, 2, 4, 8}; KV_F32 returns KV_ERR_UNSUPPORTED.
 * Asynchronous; allocates nothing.
 */
size_t kvattn_prefill_workspace_bytes(int num_seqs, int total_q_tokens, int num_q_heads,
                                      int head_dim);

int kvattn_prefill_chunk(const void* q, const void* kv_layer, int num_blocks,
                         const int32_t* block_table, const int32_t* seq_lens,
                         const int32_t* cu_seqlens_q, void* out, int num_seqs,
                         int total_q_tokens, int max_num_batched_tokens, int num_q_heads,
                         int num_kv_heads, int head_dim, int block_size,
                         int max_blocks_per_seq, int max_seq_len, float scale,
                         kv_dtype dtype, void* workspace, size_t workspace_bytes,
                         void* stream);

/* ------------------------------------------------------------------------- */
/* Write the new K and V rows of a step into their paged slots, the step that
 * precedes attention on every decode and prefill step (Section 3, "The
 * contiguity constraint": attention reads one tensor per layer indexed by
 * block id; Section 2: the cache is handed out to sequences in fixed-size
 * blocks).
 *
 * k_new, v_new  device, [num_tokens][num_kv_heads][head_dim] of dtype, 16-B
 *               aligned; head_dim * element size must be a multiple of 16
 * slot_mapping  device int32 [num_tokens]: token t goes to slot
 *               block_id * block_size + slot_in_block of kv_layer; negative
 *               slots (padding) and slots >= num_blocks * block_size are
 *               skipped. Slots must be distinct (a repeated slot is written
 *               by an unspecified one of its tokens).
 * kv_layer      device, one layer in the layout above, 16-B aligned; the K row
 *               lands in the chunk-major K tile, the V row in the dim-major V
 *               tile of the block, for every kv head
 * Supported: bf16 and fp32, block_size 16, rows (head_dim x element size) of
 * 64 to 512 bytes in steps of 64 (KV_ERR_UNSUPPORTED otherwise). Asynchronous on
 * stream; allocates nothing; num_tokens == 0 is a no-op.
 */
int kvattn_kv_append(const void* k_new, const void* v_new, const int32_t* slot_mapping,
                     void* kv_layer, int num_blocks, int num_tokens, int num_kv_heads,
                     int head_dim, int block_size, kv_dtype dtype, void* stream);

/* ------------------------------------------------------------------------- */
/* Elastic per-layer KV pool (Section 3, "Two handles, one virtual range").
 * Each layer owns one reserved virtual range of base + elastic bytes plus one
 * unmapped guard granule. A base physical handle backs [0, base) for the
 * pool's life; an elastic handle backs [base, base + elastic) only while
 * committed. Layer pointers never move, so kernels and captured graphs keep
 * working across toggles. Sizes must be multiples of kvpool_granularity(). */
typedef struct kvpool kvpool;

/* Minimum VMM granularity of the device, in bytes. */
int kvpool_granularity(int device, size_t* bytes);

/* Reserve and map every layer's base sub-range; the elastic sub-ranges start
 * decommitted. On failure nothing stays allocated and *out is NULL.
 * KV_ERR_OOM if the base handles cannot be created. */
int kvpool_create(int device, int num_layers, size_t base_bytes_per_layer,
                  size_t elastic_bytes_per_layer, kvpool** out);

/* Base address of a layer's range; stable for the pool's lifetime. */
int kvpool_layer_ptr(const kvpool* pool, int layer, void** ptr);

/* 1 if the elastic sub-ranges are mapped, 0 if not, <0 on a bad pool. */
int kvpool_is_committed(const kvpool* pool);

/* Commit: for every layer create an elastic physical handle, map it at the
 * top of the layer's range and grant the device read/write access. Synchronous:
 * the memory is usable from any stream on return. Committing a committed pool
 * is a successful no-op. If any layer's handle cannot be created, every handle
 * made so far is released, the pool stays decommitted with its base contents
 * intact, and KV_ERR_OOM is returned. Contents of freshly committed memory are
 * undefined. elapsed_ms (nullable) receives the host wall time of the call. */
int kvpool_commit_elastic(kvpool* pool, double* elapsed_ms);

/* Decommit: wait for all work on the device to finish, then unmap and release
 * every layer's elastic handle, returning the memory to the device (Section 3,
 * "Controller": drain, sync, unmap). The caller must first stop handing out
 * elastic block ids. Decommitting a decommitted pool is a successful no-op.
 * elapsed_ms (nullable) receives the host wall time of the call. */
int kvpool_decommit_elastic(kvpool* pool, double* elapsed_ms);

/* Sizes as created. */
int kvpool_sizes(const kvpool* pool, int* num_layers, size_t* base_bytes_per_layer,
                 size_t* elastic_bytes_per_layer);

/* Host wall-time breakdown of the last commit (create, map, set access) and
 * of the last decommit (device sync, unmap + release), in milliseconds.
 * Any output pointer may be NULL. kvpool_last_toggle_steps below has every
 * step on its own. */
int kvpool_last_toggle_breakdown(const kvpool* pool, double* create_ms, double* map_ms,
                                 double* access_ms, double* sync_ms, double* unmap_ms);

/* Host wall time of each step of the pool's last commit and last decommit,
 * in milliseconds (steps a path does not take read 0). */
typedef struct {
  double commit_create_ms;     /* physical handles created */
  double commit_copy_ms;       /* base contents copied into new handles (whole-handle) */
  double commit_map_ms;        /* handles mapped into the layer ranges (whole-handle:
                                  with the base handles unmapped first) */
  double commit_access_ms;     /* read/write access granted */
  double commit_release_ms;    /* base handles released (whole-handle) */
  double decommit_sync_ms;     /* device synchronised */
  double decommit_create_ms;   /* base handles created (whole-handle) */
  double decommit_copy_ms;     /* base contents copied out (whole-handle) */
  double decommit_unmap_ms;    /* elastic (whole-handle: whole) mappings removed */
  double decommit_map_ms;      /* base handles mapped back (whole-handle) */
  double decommit_access_ms;   /* access granted on the base (whole-handle) */
  double decommit_release_ms;  /* elastic (whole-handle: whole) handles released */
} kvpool_steps;

int kvpool_last_toggle_steps(const kvpool* pool, kvpool_steps* out);

/* The naive toggle the paper measures against (Section 3, "Toggle cost": a
 * commit that creates and maps a whole handle, where the physical allocation
 * dominates). For every layer: create one physical handle of base + elastic
 * bytes, copy the layer's base contents into it (through a staging mapping),
 * unmap the base handle from the layer's range, map the whole handle over
 * [0, base + elastic), grant access, release the base handle. The layer
 * pointers do not move and base contents are preserved bit for bit.
 * Requires a decommitted pool (KV_ERR_STATE if it was committed with
 * kvpool_commit_elastic; a successful no-op if committed by this call). On any
 * failure every layer is left on its base handle and the new handles are
 * released (KV_ERR_OOM if they could not be created). kvpool_decommit_elastic
 * on a pool committed this way does the whole-handle decommit: new base
 * handles, the base contents copied back, the whole handles unmapped and
 * released. Synchronous. elapsed_ms (nullable) receives the host wall time. */
int kvpool_commit_whole(kvpool* pool, double* elapsed_ms);

/* Decommit if needed, unmap the base handles, free the ranges. NULL is a no-op. */
void kvpool_destroy(kvpool* pool);

/* Cost of the naive toggle (Section 3, "Toggle cost": a whole-handle commit of
 * the entire reserve, where physical allocation dominates). On ROCm a handle
 * maps only at offset 0, so one handle cannot back the per-layer elastic
 * slices at all; this times what such a commit would pay for the allocation
 * and mapping: reserve a fresh range, create one handle of `bytes` (a multiple
 * of the granularity), map it, grant access, then unmap and release it and free
 * the range. Host wall times in ms; any output pointer may be NULL. Returns
 * KV_ERR_OOM if the handle cannot be created. */
int kvpool_time_single_handle(int device, size_t bytes, double* create_ms, double* map_ms,
                              double* access_ms, double* release_ms);

/* ------------------------------------------------------------------------- */
/* Block-id pool with the elastic gate (Section 3, "Two handles, one virtual
 * range": the top elastic block-id range is handed out only while the elastic
 * slice is committed). Ids [0, num_base) are base blocks, ids
 * [num_base, num_base + num_elastic) the elastic blocks at the top of every
 * layer's range. Host memory only; not thread-safe (one scheduler drives it).
 * Base blocks are handed out before elastic ones, lowest id first, so that as
 * few sequences as possible hold elastic blocks when a prefill comes. */
typedef struct kvblocks kvblocks;

int kvblocks_create(int num_base_blocks, int num_elastic_blocks, kvblocks** out);
void kvblocks_destroy(kvblocks* blocks);
/* Admit (admit != 0) or stop handing out (admit == 0) the elastic ids. Live
 * elastic blocks stay allocated until freed; the controller below admits and
 * withdraws the range together with the commit and decommit. */
int kvblocks_set_elastic(kvblocks* blocks, int admit);
int kvblocks_is_admitted(const kvblocks* blocks);
/* Allocate n ids into the host array ids; KV_ERR_OOM (and nothing allocated)
 * if fewer than n admitted ids are free. */
int kvblocks_alloc(kvblocks* blocks, int n, int32_t* ids);
/* Free n ids; KV_ERR_INVALID (and nothing freed) if any id is not allocated
 * or appears twice. */
int kvblocks_free(kvblocks* blocks, int n, const int32_t* ids);
/* Free admitted ids; ids usable now (num_gpu_blocks): num_base, plus
 * num_elastic while admitted; allocated ids in the elastic range. */
int kvblocks_num_free(const kvblocks* blocks);
int kvblocks_num_admitted(const kvblocks* blocks);
int kvblocks_live_elastic(const kvblocks* blocks);
/* Plan a drain of the elastic range by migration: for every live elastic id
 * (ascending) allocate a free base id; writes *n pairs from[i] -> to[i] into
 * host arrays of room for `capacity` pairs. The caller copies each block in
 * every layer (kvattn_copy_blocks), rewrites its block tables, and frees the
 * `from` ids. KV_ERR_OOM (nothing allocated) if the base range has too few free
 * ids; KV_ERR_INVALID if capacity is too small. */
int kvblocks_plan_drain(kvblocks* blocks, int capacity, int32_t* from, int32_t* to, int* n);

/* Copy whole blocks src_ids[i] -> dst_ids[i] (device int32 arrays of n) in each
 * of num_layers layers (layers: host array of 16-B aligned device pointers, each
 * the base of a layer of num_blocks blocks of block_bytes bytes, a multiple of
 * 16). Pairs with an id outside [0, num_blocks), or src == dst, are skipped;
 * destinations must be distinct and must not be sources of other pairs.
 * Asynchronous on stream; allocates nothing. Used to drain the elastic range
 * before a decommit (Section 3, "Controller"). */
int kvattn_copy_blocks(void* const* layers, int num_layers, int num_blocks,
                       size_t block_bytes, const int32_t* src_ids, const int32_t* dst_ids,
                       int n, void* stream);

/* ------------------------------------------------------------------------- */
/* One-step-ahead toggle controller (Section 3, "Controller"). The scheduler
 * knows its next batch before running it and calls kvctl_before_step with
 * whether that batch contains a prefill:
 *   - prefill next: if committed, stop admitting elastic ids and decommit
 *     (device sync, unmap). If elastic blocks are still live it returns
 *     KV_ERR_STATE and changes nothing: drain them (free or migrate) and call
 *     again. Prefill runs with the reserve returned to the device. If the
 *     decommit itself fails, the error is returned and the controller takes
 *     the pool's state: still committed after a failed device sync,
 *     decommitted (elastic ids no longer admitted) after a failed unmap or
 *     release.
 *   - decode-only next: count the run of decode-only steps; after
 *     hysteresis_steps of them, commit and admit the elastic ids. A failed
 *     commit (KV_ERR_OOM) leaves the pool decommitted and restarts the count.
 * *action (nullable) receives KVCTL_NONE, KVCTL_COMMIT or KVCTL_DECOMMIT and
 * *ms (nullable) the toggle's host wall time. With pool == NULL the controller
 * runs the same state machine without a device (the gate only). Callers that
 * use a caching allocator should return its cached memory to the device before
 * a step for which kvctl_would_commit() is 1 (Section 4: a recommit after a
 * large prefill otherwise fails while the allocator holds the freed memory). */
typedef struct kvctl kvctl;
enum { KVCTL_NONE = 0, KVCTL_COMMIT = 1, KVCTL_DECOMMIT = 2 };

int kvctl_create(kvpool* pool, kvblocks* blocks, int hysteresis_steps, kvctl** out);
void kvctl_destroy(kvctl* ctl);
int kvctl_before_step(kvctl* ctl, int next_has_prefill, int* action, double* ms);
int kvctl_would_commit(const kvctl* ctl, int next_has_prefill);
int kvctl_is_committed(const kvctl* ctl);
int kvctl_counts(const kvctl* ctl, int* commits, int* decommits);

#ifdef __cplusplus
}
#endif

#endif /* KVATTN_H */
