"""Plain CPU oracle for writing new K/V rows into the paged layer.

TEST INFRASTRUCTURE ONLY (see ``oracle.paged_kv``): only ``tests/``,
``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py`` may
use it; the HIP library never does.

What is computed
----------------
Before attention reads a step's keys and values, the rows of the step's new
tokens must sit in the layer tensor that the kernel indexes by block id
(Section 3, "The contiguity constraint"; Section 2, "KV allocation in vLLM":
the KV cache is fixed-size blocks handed out to sequences). Token ``t`` goes to
slot ``slot_mapping[t] = block * block_size + r``; its K row lands in the K
tile and its V row in the V tile of that block, for every KV head::

    K tile of (block, head): dim j of slot r at ((j // VEC) * block_size + r) * VEC + j % VEC
    V tile of (block, head): dim j of slot r at j * block_size + r

with ``VEC = 16 / element_size`` and the layer laid out as
``layer[num_blocks][2 (K, V)][num_kv_heads][block_size * head_dim]``.
A negative slot (padding) or one past the layer is skipped. Tokens are
written in order, so with repeated slots the later token wins (callers of the
GPU path must not repeat slots).

This is a copy: no arithmetic, so the result is exact.
"""
from __future__ import annotations

import numpy as np


def kv_append(kv_raw: np.ndarray, k_new: np.ndarray, v_new: np.ndarray,
              slot_mapping: np.ndarray, *, dtype: str, num_kv_heads: int, head_dim: int,
              block_size: int) -> np.ndarray:
    """Return a copy of the layer (storage elements, any shape) with the new rows written.

    ``k_new``/``v_new``: storage elements ``[num_tokens, num_kv_heads, head_dim]``
    (uint16 bf16 bit patterns or float32).
    """
    esz = {"bf16": 2, "f32": 4}[dtype]
    vec = 16 // esz
    out = np.array(kv_raw, copy=True)
    flat = out.reshape(-1)
    tile = block_size * head_dim
    num_blocks = flat.size // (2 * num_kv_heads * tile)
    layer = flat.reshape(num_blocks, 2, num_kv_heads, tile)
    j = np.arange(head_dim)
    for t in range(len(slot_mapping)):
        slot = int(slot_mapping[t])
        if slot < 0 or slot >= num_blocks * block_size:
            continue
        b, r = divmod(slot, block_size)
        k_pos = ((j // vec) * block_size + r) * vec + j % vec
        v_pos = j * block_size + r
        for g in range(num_kv_heads):
            layer[b, 0, g, k_pos] = k_new[t, g]
            layer[b, 1, g, v_pos] = v_new[t, g]
    return out


def copy_blocks(kv_raw: np.ndarray, src, dst, *, num_blocks: int) -> np.ndarray:
    """Copy of the layer with block ``dst[i]`` replaced by block ``src[i]`` (as it
    was before any copy); pairs with an id outside ``[0, num_blocks)`` or with
    ``src == dst`` are skipped. This is how the elastic range is drained by
    migration before a decommit (Section 3, "Controller")."""
    out = np.array(kv_raw, copy=True)
    before = np.asarray(kv_raw).reshape(num_blocks, -1)
    after = out.reshape(num_blocks, -1)
    for s, d in zip(np.asarray(src).tolist(), np.asarray(dst).tolist()):
        if 0 <= s < num_blocks and 0 <= d < num_blocks and s != d:
            after[d] = before[s]
    return out
