"""Seeded generator: sequence lengths, block tables, Q and paged K/V bytes.

Paged layout of one layer (the layout every consumer reads)
-----------------------------------------------------------
One layer is one contiguous array of ``num_blocks`` blocks, block-major, so
block ids grow with the address and the top block ids sit at the top of the
range. One block holds, for each of K and V and each KV head, ``block_size``
tokens of ``head_dim`` elements::

    layer[num_blocks][2 (K, V)][num_kv_heads][block_size * head_dim]

Within the ``block_size * head_dim`` tile of one (block, K/V, head):

* K is chunk-major: element (slot r, dim j) sits at
  ``((j // VEC) * block_size + r) * VEC + j % VEC`` with ``VEC = 16 / esz``
  (8 for bf16, 4 for fp32), i.e. 16-byte chunks of one token's row, with the
  chunks of all slots of the block laid side by side.
* V is dim-major (transposed): element (slot r, dim j) sits at
  ``j * block_size + r``.

Everything not covered by a sequence's tokens (blocks no table references,
and slots past a sequence's length in its last block) is filled with NaN, so
a stray read shows in the output.

Recipe
------
With ``g = torch.Generator().manual_seed(spec.seed)``, in this order:

1. random sequence lengths ``torch.randint(lo, hi + 1, (count,), generator=g)``;
2. a permutation ``torch.randperm(num_blocks, generator=g)``; its first
   ``sum(ceil(L_s / block_size))`` entries become the block tables, sequence
   0's logical blocks first;
3. ``q = torch.randn(total_q_tokens, Hq, d, generator=g)`` in fp32, cast to
   the storage dtype;
4. per sequence in order: ``K_s = randn(L_s, Hkv, d)``, ``V_s = randn(L_s,
   Hkv, d)`` in fp32, cast, scattered into the pool.

Values are N(0, 1). bf16 casts round to nearest even (torch's cast).
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import List, Optional, Sequence

import numpy as np
import torch

from .configs import BatchSpec, pool_blocks_rule

_TORCH_DTYPES = {"f32": torch.float32, "bf16": torch.bfloat16}
_ESZ = {"f32": 4, "bf16": 2}


def storage_torch_dtype(dtype: str) -> torch.dtype:
    return _TORCH_DTYPES[dtype]


def nan_bits(dtype: str) -> int:
    """Bit pattern of the quiet NaN used as poison."""
    return 0x7FC0 if dtype == "bf16" else 0x7FC00000


def layout_offsets(which: int, block, head, slot, dim, num_kv_heads: int,
                   block_size: int, head_dim: int, esz: int):
    """Flat element index of (block, K=0/V=1, kv head, slot, dim) in a layer."""
    vec = 16 // esz
    tile = block_size * head_dim
    base = ((np.asarray(block, dtype=np.int64) * 2 + which) * num_kv_heads + head) * tile
    if which == 0:
        inner = ((np.asarray(dim) // vec) * block_size + slot) * vec + np.asarray(dim) % vec
    else:
        inner = np.asarray(dim) * block_size + slot
    return base + inner


@dataclass
class PagedBatch:
    """Host-side bytes of one attention call (torch CPU tensors)."""

    dtype: str
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    block_size: int
    num_blocks: int
    scale: float
    seq_lens: np.ndarray        # int32 [B], context length including the new tokens
    q_lens: np.ndarray          # int32 [B], new tokens per sequence
    cu_seqlens_q: np.ndarray    # int32 [B + 1]
    block_table: np.ndarray     # int32 [B, max_blocks], -1 padded
    q: torch.Tensor             # [T, Hq, d] storage dtype
    kv_layer: torch.Tensor      # flat [num_blocks * 2 * Hkv * bs * d] storage dtype
    k_contig: Optional[List[torch.Tensor]] = None   # per sequence [L, Hkv, d]
    v_contig: Optional[List[torch.Tensor]] = None

    @property
    def num_seqs(self) -> int:
        return int(self.seq_lens.shape[0])

    @property
    def total_q_tokens(self) -> int:
        return int(self.cu_seqlens_q[-1])

    @property
    def max_blocks_per_seq(self) -> int:
        return int(self.block_table.shape[1])

    @property
    def max_seq_len(self) -> int:
        return int(self.seq_lens.max()) if self.seq_lens.size else 0

    @property
    def esz(self) -> int:
        return _ESZ[self.dtype]

    def q_raw(self) -> np.ndarray:
        """Q as stored: uint16 bit patterns for bf16, float32 otherwise."""
        return _raw(self.q)

    def kv_raw(self) -> np.ndarray:
        return _raw(self.kv_layer)


def _raw(t: torch.Tensor) -> np.ndarray:
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def _scatter_sequence(pool4: torch.Tensor, k: torch.Tensor, v: torch.Tensor,
                      blocks: np.ndarray, num_kv_heads: int, block_size: int,
                      head_dim: int, vec: int) -> None:
    L = k.shape[0]
    if L == 0:
        return
    t = torch.arange(L)
    b_idx = torch.as_tensor(blocks, dtype=torch.int64)[t // block_size]
    r_idx = t % block_size
    nb = pool4.shape[0]
    kview = pool4[:, 0].view(nb, num_kv_heads, head_dim // vec, block_size, vec)
    vview = pool4[:, 1].view(nb, num_kv_heads, head_dim, block_size)
    kview[b_idx, :, :, r_idx, :] = k.reshape(L, num_kv_heads, head_dim // vec, vec)
    vview[b_idx, :, :, r_idx] = v


def make_batch_from_lens(seq_lens: Sequence[int], q_lens: Sequence[int], *, dtype: str,
                         num_q_heads: int, num_kv_heads: int, head_dim: int,
                         block_size: int, seed: int, num_blocks: Optional[int] = None,
                         keep_contig: bool = False,
                         generator: Optional[torch.Generator] = None,
                         block_perm: Optional[np.ndarray] = None) -> PagedBatch:
    """Build a batch for given lengths; steps 2-4 of the recipe.

    ``block_perm`` replaces the drawn permutation (used to lay the same
    logical K/V out under a different block table); the generator still
    draws its permutation so that Q and K/V values do not change.
    """
    g = generator if generator is not None else torch.Generator().manual_seed(seed)
    seq_lens = np.asarray(seq_lens, dtype=np.int32)
    q_lens = np.asarray(q_lens, dtype=np.int32)
    assert seq_lens.shape == q_lens.shape
    assert np.all(q_lens <= seq_lens) and np.all(q_lens >= 0)
    nblk = [-(-int(L) // block_size) for L in seq_lens]
    total_blocks = int(sum(nblk))
    if num_blocks is None:
        num_blocks = pool_blocks_rule(total_blocks)
    assert num_blocks >= total_blocks, "pool smaller than the batch"
    perm = torch.randperm(num_blocks, generator=g).numpy().astype(np.int32)
    if block_perm is not None:
        perm = np.asarray(block_perm, dtype=np.int32)
        assert perm.shape == (num_blocks,)
    max_blocks = max(nblk) if nblk else 0
    max_blocks = max(max_blocks, 1)
    bt = np.full((len(seq_lens), max_blocks), -1, dtype=np.int32)
    pos = 0
    for s, n in enumerate(nblk):
        bt[s, :n] = perm[pos:pos + n]
        pos += n
    cu = np.zeros(len(seq_lens) + 1, dtype=np.int32)
    cu[1:] = np.cumsum(q_lens)
    T = int(cu[-1])
    tdt = _TORCH_DTYPES[dtype]
    q = torch.randn(T, num_q_heads, head_dim, generator=g).to(tdt)
    esz = _ESZ[dtype]
    vec = 16 // esz
    tile = block_size * head_dim
    pool = torch.full((num_blocks * 2 * num_kv_heads * tile,), float("nan"), dtype=tdt)
    pool4 = pool.view(num_blocks, 2, num_kv_heads, tile)
    kc, vc = ([], []) if keep_contig else (None, None)
    for s, L in enumerate(seq_lens):
        L = int(L)
        k = torch.randn(L, num_kv_heads, head_dim, generator=g).to(tdt)
        v = torch.randn(L, num_kv_heads, head_dim, generator=g).to(tdt)
        _scatter_sequence(pool4, k, v, bt[s, :nblk[s]], num_kv_heads, block_size, head_dim, vec)
        if keep_contig:
            kc.append(k)
            vc.append(v)
    return PagedBatch(dtype=dtype, num_q_heads=num_q_heads, num_kv_heads=num_kv_heads,
                      head_dim=head_dim, block_size=block_size, num_blocks=num_blocks,
                      scale=1.0 / math.sqrt(head_dim), seq_lens=seq_lens, q_lens=q_lens,
                      cu_seqlens_q=cu, block_table=bt, q=q, kv_layer=pool,
                      k_contig=kc, v_contig=vc)


def spec_lengths(spec: BatchSpec, g: torch.Generator):
    """Step 1 of the recipe: the (seq_len, q_len) list of a spec."""
    seq_lens: List[int] = []
    q_lens: List[int] = []
    for L, n in spec.fixed_prefix:
        seq_lens.append(int(L))
        q_lens.append(int(n))
    if spec.fixed_seq_lens is not None:
        for L in spec.fixed_seq_lens:
            seq_lens.append(int(L))
            q_lens.append(spec.q_len_rand)
    if spec.rand_count:
        r = torch.randint(spec.rand_lo, spec.rand_hi + 1, (spec.rand_count,), generator=g)
        for L in r.tolist():
            seq_lens.append(int(L))
            q_lens.append(spec.q_len_rand)
    return seq_lens, q_lens


def make_batch(spec: BatchSpec, keep_contig: bool = False,
               block_perm: Optional[np.ndarray] = None) -> PagedBatch:
    g = torch.Generator().manual_seed(spec.seed)
    seq_lens, q_lens = spec_lengths(spec, g)
    return make_batch_from_lens(seq_lens, q_lens, dtype=spec.dtype,
                                num_q_heads=spec.num_q_heads,
                                num_kv_heads=spec.num_kv_heads,
                                head_dim=spec.head_dim, block_size=spec.block_size,
                                seed=spec.seed, num_blocks=spec.num_blocks,
                                keep_contig=keep_contig, generator=g,
                                block_perm=block_perm)
