"""Plain, slow fp64 CPU oracle for attention over a block-indexed paged KV cache.

TEST INFRASTRUCTURE ONLY. Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or call anything in this
package. The HIP library and its Python binding never import it, and it
imports nothing from them: the two share no code. Only the seeded input
generator (``workloads``) feeds both.

What is computed
----------------
The paper keeps each layer's KV cache as one tensor that the attention kernel
indexes by block id through a single base pointer (Section 3, "The contiguity
constraint"; Section 1). Decode gives each running sequence one new query
token per step, and a prefill chunk attends to all of the prompt before it, so
cutting a prompt into chunks splits the same work across steps (Section 5,
"Why the penalty is small"). The elastic pool changes where the bytes live,
never the arithmetic (Section 3, "Two handles, one virtual range").

For sequence ``s`` with ``L_s`` context tokens of which the last ``n_s`` are
new (``c_s = L_s - n_s`` cached), new row ``i`` sits at absolute position
``p = c_s + i``. For query head ``h`` with KV head ``g = h // (Hq // Hkv)``::

    K_s[t] = K part of block bt[s][t // bs], kv head g, slot t % bs
    V_s[t] = V part of the same block, head and slot
    out[cu[s] + i, h] = sum_{t <= p} softmax_t(scale * q[cu[s] + i, h] . K_s[t]) V_s[t]

Readings where the paper is silent: the causal mask is aligned bottom-right
(row ``i`` sees keys up to ``c_s + i``), the only alignment under which a chunk
does the same work as the unchunked pass; query heads map to KV heads in
consecutive groups; a sequence with no context produces zeros.

Steps, in order
---------------
1. Upcast the stored bytes exactly to fp64 (bf16 bit patterns are widened by a
   16-bit shift).
2. Gather ``K_s`` and ``V_s`` by walking the block table one block at a time,
   never past ``L_s``; padding entries are never read.
3. For each run of new rows inside one tile of 256 absolute positions aligned
   to a multiple of 256: ``S = scale * Q K^T`` over keys ``[0, tile_end)``, keys
   after a row's own position set to ``-inf``, ``m`` = row max,
   ``W = exp(S - m)``, ``Z`` = row sum of ``W``, ``out = (W V) / Z``. The softmax
   is the exact two-pass form, with no running rescale.

Because the tiles are fixed in absolute position, a row's arithmetic is the
same whether its prompt arrived in one chunk or in several chunks whose
boundaries are multiples of 256.

Paged layout read here (one layer)::

    layer[num_blocks][2 (K, V)][num_kv_heads][block_size * head_dim]

K tile: slot ``r``, dim ``j`` at ``((j // VEC) * block_size + r) * VEC + j % VEC``
with ``VEC = 16 / element_size``; V tile: at ``j * block_size + r``.
"""
from __future__ import annotations

import numpy as np

ROW_TILE = 256


def storage_to_f64(raw: np.ndarray, dtype: str) -> np.ndarray:
    """Exact widening of stored values: bf16 bit patterns (uint16) or fp32."""
    if dtype == "bf16":
        u = np.asarray(raw, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
        return u.view(np.float32).astype(np.float64)
    if dtype == "f32":
        return np.asarray(raw, dtype=np.float32).astype(np.float64)
    raise ValueError(f"unknown dtype {dtype!r}")


def _element_size(dtype: str) -> int:
    return {"bf16": 2, "f32": 4}[dtype]


def gather_kv(kv_raw: np.ndarray, dtype: str, block_ids: np.ndarray, seq_len: int,
              num_kv_heads: int, block_size: int, head_dim: int):
    """Step 2: K_s, V_s as fp64 ``[seq_len, Hkv, d]`` read through the block table.

    Reads the first ``ceil(seq_len / block_size)`` table entries only, one
    block at a time, and keeps the first ``seq_len`` slots.
    """
    tile = block_size * head_dim
    num_blocks = kv_raw.size // (2 * num_kv_heads * tile)
    layer = kv_raw.reshape(num_blocks, 2, num_kv_heads, tile)
    vec = 16 // _element_size(dtype)
    nblk = -(-seq_len // block_size)
    K = np.empty((nblk * block_size, num_kv_heads, head_dim), dtype=np.float64)
    V = np.empty_like(K)
    for j in range(nblk):
        b = int(block_ids[j])
        if not 0 <= b < num_blocks:
            raise IndexError(f"block id {b} outside the pool of {num_blocks} blocks")
        kt = storage_to_f64(layer[b, 0], dtype)   # [Hkv, tile]
        vt = storage_to_f64(layer[b, 1], dtype)
        # K tile [Hkv][d/VEC][bs][VEC] -> [bs][Hkv][d]
        k = kt.reshape(num_kv_heads, head_dim // vec, block_size, vec)
        k = k.transpose(2, 0, 1, 3).reshape(block_size, num_kv_heads, head_dim)
        # V tile [Hkv][d][bs] -> [bs][Hkv][d]
        v = vt.reshape(num_kv_heads, head_dim, block_size).transpose(2, 0, 1)
        K[j * block_size:(j + 1) * block_size] = k
        V[j * block_size:(j + 1) * block_size] = v
    return K[:seq_len], V[:seq_len]


def attend(qf: np.ndarray, K: np.ndarray, V: np.ndarray, context: int, scale: float) -> np.ndarray:
    """Step 3 for one sequence: ``qf`` holds the new rows ``[n, Hq, d]`` (fp64),
    which sit at absolute positions ``context .. context + n - 1``."""
    n, num_q_heads, head_dim = qf.shape
    L, num_kv_heads, _ = K.shape
    assert context + n == L, "rows must end at the sequence's last position"
    group = num_q_heads // num_kv_heads
    out = np.zeros((n, num_q_heads, head_dim), dtype=np.float64)
    if n == 0:
        return out
    Kg = [np.ascontiguousarray(K[:, g, :]) for g in range(num_kv_heads)]
    Vg = [np.ascontiguousarray(V[:, g, :]) for g in range(num_kv_heads)]
    first = (context // ROW_TILE) * ROW_TILE
    for a in range(first, L, ROW_TILE):
        lo, hi = max(a, context), min(a + ROW_TILE, L)
        tile_end = min(a + ROW_TILE, L)
        pos = np.arange(lo, hi)
        keys = np.arange(tile_end)
        future = keys[None, :] > pos[:, None]
        for h in range(num_q_heads):
            g = h // group
            Q = np.ascontiguousarray(qf[lo - context:hi - context, h, :])
            S = scale * (Q @ Kg[g][:tile_end].T)
            S[future] = -np.inf
            m = S.max(axis=1, keepdims=True)
            W = np.exp(S - m)
            Z = W.sum(axis=1, keepdims=True)
            out[lo - context:hi - context, h, :] = (W @ Vg[g][:tile_end]) / Z
    return out


def paged_attention(q_raw: np.ndarray, kv_raw: np.ndarray, block_table: np.ndarray,
                    seq_lens: np.ndarray, cu_seqlens_q: np.ndarray, *, dtype: str,
                    num_q_heads: int, num_kv_heads: int, head_dim: int,
                    block_size: int, scale: float, seqs=None) -> np.ndarray:
    """Attention for every new token of a batch of chunks: fp64 ``[T, Hq, d]``.

    ``seq_lens`` counts the context including the chunk; the chunk of
    sequence ``s`` is query rows ``[cu[s], cu[s+1])``. ``seqs`` restricts the
    work to some sequences (other rows stay zero).
    """
    T = int(cu_seqlens_q[-1])
    q = storage_to_f64(np.asarray(q_raw).reshape(T, num_q_heads, head_dim), dtype)
    out = np.zeros((T, num_q_heads, head_dim), dtype=np.float64)
    for s in (range(len(seq_lens)) if seqs is None else seqs):
        L = int(seq_lens[s])
        r0, r1 = int(cu_seqlens_q[s]), int(cu_seqlens_q[s + 1])
        n = r1 - r0
        if n == 0:
            continue
        if n > L:
            raise ValueError(f"sequence {s}: {n} new tokens but context {L}")
        K, V = gather_kv(kv_raw, dtype, block_table[s], L, num_kv_heads, block_size, head_dim)
        out[r0:r1] = attend(q[r0:r1], K, V, L - n, scale)
    return out


def paged_decode(q_raw: np.ndarray, kv_raw: np.ndarray, block_table: np.ndarray,
                 seq_lens: np.ndarray, *, dtype: str, num_q_heads: int, num_kv_heads: int,
                 head_dim: int, block_size: int, scale: float, seqs=None) -> np.ndarray:
    """Decode: one new query token per sequence, ``q`` is ``[B, Hq, d]``.

    The token is the last of its sequence's ``L_s`` tokens; a sequence with
    ``L_s == 0`` has nothing to attend to and yields zeros.
    """
    B = len(seq_lens)
    q = storage_to_f64(np.asarray(q_raw).reshape(B, num_q_heads, head_dim), dtype)
    out = np.zeros((B, num_q_heads, head_dim), dtype=np.float64)
    for s in (range(B) if seqs is None else seqs):
        L = int(seq_lens[s])
        if L == 0:
            continue
        K, V = gather_kv(kv_raw, dtype, block_table[s], L, num_kv_heads, block_size, head_dim)
        out[s:s + 1] = attend(q[s:s + 1], K, V, L - 1, scale)
    return out


def paged_attention_rows(q_raw: np.ndarray, kv_raw: np.ndarray, block_table: np.ndarray,
                         seq_lens: np.ndarray, cu_seqlens_q: np.ndarray, rows, *, dtype: str,
                         num_q_heads: int, num_kv_heads: int, head_dim: int,
                         block_size: int, scale: float) -> np.ndarray:
    """The same definition for a sample of query rows (global token indices):
    fp64 ``[len(rows), Hq, d]``. Each row is computed on its own over keys
    ``[0, p]``, for checks at sizes where the full output is too costly."""
    T = int(cu_seqlens_q[-1])
    qv = np.asarray(q_raw).reshape(T, num_q_heads, head_dim)
    group = num_q_heads // num_kv_heads
    rows = [int(r) for r in rows]
    out = np.zeros((len(rows), num_q_heads, head_dim), dtype=np.float64)
    cache = {}
    for k, r in enumerate(rows):
        s = int(np.searchsorted(cu_seqlens_q, r, side="right") - 1)
        L = int(seq_lens[s])
        n = int(cu_seqlens_q[s + 1] - cu_seqlens_q[s])
        p = L - n + (r - int(cu_seqlens_q[s]))
        if s not in cache:
            cache.clear()
            cache[s] = gather_kv(kv_raw, dtype, block_table[s], L, num_kv_heads,
                                 block_size, head_dim)
        K, V = cache[s]
        q = storage_to_f64(qv[r], dtype)
        for h in range(num_q_heads):
            g = h // group
            S = scale * (K[:p + 1, g, :] @ q[h])
            W = np.exp(S - S.max())
            out[k, h] = (W @ V[:p + 1, g, :]) / W.sum()
    return out
