"""Seeded inputs for writing new K/V rows into a paged layer.

Recipe: new K and V rows are N(0, 1) drawn with ``torch.randn`` on a CPU
generator seeded ``seed`` (K first, then V), cast to the storage dtype; slots
are distinct, drawn as the first ``num_tokens`` entries of a seeded
permutation of all ``num_blocks * block_size`` slots, and a seeded fraction of
the tokens is turned into padding (slot -1). No attention arithmetic lives here.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np
import torch

_TDT = {"bf16": torch.bfloat16, "f32": torch.float32}


@dataclass
class AppendBatch:
    k_new: torch.Tensor          # [T, Hkv, d] storage dtype (CPU)
    v_new: torch.Tensor
    slot_mapping: np.ndarray     # int32 [T], -1 = padding

    def k_raw(self) -> np.ndarray:
        return _raw(self.k_new)

    def v_raw(self) -> np.ndarray:
        return _raw(self.v_new)


def _raw(t: torch.Tensor) -> np.ndarray:
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def make_append(num_tokens: int, *, num_kv_heads: int, head_dim: int, dtype: str,
                num_blocks: int, block_size: int, seed: int,
                pad_fraction: float = 0.0) -> AppendBatch:
    g = torch.Generator().manual_seed(seed)
    k = torch.randn(num_tokens, num_kv_heads, head_dim, generator=g).to(_TDT[dtype])
    v = torch.randn(num_tokens, num_kv_heads, head_dim, generator=g).to(_TDT[dtype])
    cap = num_blocks * block_size
    assert num_tokens <= cap
    slots = torch.randperm(cap, generator=g)[:num_tokens].numpy().astype(np.int32)
    if pad_fraction > 0:
        pad = torch.rand(num_tokens, generator=g).numpy() < pad_fraction
        slots[pad] = -1
    return AppendBatch(k_new=k, v_new=v, slot_mapping=slots)


def next_slots(block_table: np.ndarray, seq_lens: np.ndarray, block_size: int) -> np.ndarray:
    """Slot of position seq_len of each sequence (the slot a decode step writes);
    -1 where that position needs a block the table does not hold."""
    out = np.full(len(seq_lens), -1, dtype=np.int32)
    for s, L in enumerate(seq_lens):
        j = int(L) // block_size
        if j < block_table.shape[1] and block_table[s, j] >= 0:
            out[s] = int(block_table[s, j]) * block_size + int(L) % block_size
    return out
