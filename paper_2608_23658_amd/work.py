"""Algorithmic work of the hot path: what the method must move or compute.

Counts exclude padding, masked work and re-reads: decode moves every context
token's K and V once (token granularity, not whole blocks), plus q, out and
the block-table entries; chunked prefill performs 2 * d multiply-adds for
q.k and 2 * d for p.v per unmasked (query, key) pair and head.
"""
from __future__ import annotations

import numpy as np


def prefill_pairs(seq_lens, q_lens) -> int:
    """Unmasked (query, key) pairs: row i of a chunk of n new tokens over c
    cached ones sees c + i + 1 keys (bottom-right causal)."""
    L = np.asarray(seq_lens, dtype=np.int64)
    n = np.asarray(q_lens, dtype=np.int64)
    c = L - n
    return int(np.sum(n * c + n * (n + 1) // 2))


def prefill_flops(seq_lens, q_lens, num_q_heads: int, head_dim: int) -> int:
    return 4 * head_dim * num_q_heads * prefill_pairs(seq_lens, q_lens)


def decode_kv_bytes(seq_lens, num_kv_heads: int, head_dim: int, esz: int) -> int:
    L = np.asarray(seq_lens, dtype=np.int64)
    return int(L.sum()) * num_kv_heads * head_dim * 2 * esz


def decode_bytes(seq_lens, num_q_heads: int, num_kv_heads: int, head_dim: int, esz: int,
                 block_size: int = 16) -> int:
    """KV bytes + q and out + block-table entries + seq_lens."""
    L = np.asarray(seq_lens, dtype=np.int64)
    B = L.size
    kv = decode_kv_bytes(L, num_kv_heads, head_dim, esz)
    qo = 2 * B * num_q_heads * head_dim * esz
    bt = int(np.sum((L + block_size - 1) // block_size)) * 4
    return kv + qo + bt + 4 * B


def decode_flops(seq_lens, num_q_heads: int, head_dim: int) -> int:
    return 4 * head_dim * num_q_heads * int(np.asarray(seq_lens, dtype=np.int64).sum())


def append_bytes(num_tokens: int, num_kv_heads: int, head_dim: int, esz: int) -> int:
    """Writing T new rows: K and V read once and written once, plus the slots."""
    row = num_kv_heads * head_dim * esz
    return 4 * num_tokens * row + 4 * num_tokens
