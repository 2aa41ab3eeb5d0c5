"""Inputs of the elastic-pool decode workload (32 layers, shared block table).

Recipe:

* ``numpy.random.default_rng(seed)`` draws, in order: the 512 sequence
  lengths (uniform integers in [8192, 32768]); the positions of the elastic
  references, ``ceil(0.15 * R)`` of the ``R = sum(ceil(L / 16))`` table
  entries without replacement; the elastic ids, uniform over the top
  ``elastic_blocks`` ids with replacement; the base ids, uniform over
  ``[0, base_blocks)`` with replacement. One table serves every layer, as
  block ids are global in the pool.
* Queries: ``torch.randn`` on the CPU generator seeded with ``seed``, cast to bf16.
* Layer contents: every byte of layer ``l`` is N(0, 1) bf16 drawn on the device
  by ``normal_`` from a CUDA generator seeded ``seed * 1000 + 2 * l`` for the
  base part and ``seed * 1000 + 2 * l + 1`` for the elastic part, so either
  part can be refilled on its own.

No attention arithmetic lives here.
"""
from __future__ import annotations

import math

import numpy as np
import torch

from .configs import ELASTIC, ElasticSpec


def elastic_tables(spec: ElasticSpec = ELASTIC):
    """(seq_lens int32 [B], block_table int32 [B, max_blocks], is_elastic bool [B, max_blocks])."""
    rng = np.random.default_rng(spec.seed)
    lens = rng.integers(spec.len_lo, spec.len_hi + 1, size=spec.batch).astype(np.int32)
    nblk = (lens + spec.block_size - 1) // spec.block_size
    R = int(nblk.sum())
    n_el = int(math.ceil(spec.elastic_fraction * R))
    el_pos = rng.choice(R, size=n_el, replace=False)
    flat = np.empty(R, dtype=np.int32)
    is_el = np.zeros(R, dtype=bool)
    is_el[el_pos] = True
    flat[is_el] = spec.base_blocks + rng.integers(0, spec.elastic_blocks, size=n_el)
    flat[~is_el] = rng.integers(0, spec.base_blocks, size=R - n_el)
    maxb = (spec.len_hi + spec.block_size - 1) // spec.block_size
    bt = np.full((spec.batch, maxb), -1, dtype=np.int32)
    el = np.zeros((spec.batch, maxb), dtype=bool)
    pos = 0
    for s, n in enumerate(nblk):
        bt[s, :n] = flat[pos:pos + n]
        el[s, :n] = is_el[pos:pos + n]
        pos += n
    return lens, bt, el


def elastic_queries(spec: ElasticSpec = ELASTIC) -> torch.Tensor:
    g = torch.Generator().manual_seed(spec.seed)
    return torch.randn(spec.batch, spec.num_q_heads, spec.head_dim, generator=g).to(torch.bfloat16)


def fill_layer(view: torch.Tensor, layer: int, base_elems: int, part: str = "all",
               spec: ElasticSpec = ELASTIC) -> None:
    """Fill a bf16 device view of one layer (base + elastic elements)."""
    dev = view.device
    if part in ("all", "base"):
        g = torch.Generator(device=dev).manual_seed(spec.seed * 1000 + 2 * layer)
        view[:base_elems].normal_(generator=g)
    if part in ("all", "elastic"):
        g = torch.Generator(device=dev).manual_seed(spec.seed * 1000 + 2 * layer + 1)
        view[base_elems:].normal_(generator=g)


def remap_elastic_to_base(bt: np.ndarray, spec: ElasticSpec = ELASTIC) -> np.ndarray:
    """The same reuse structure on base ids only: elastic id e -> e - base_blocks."""
    out = bt.copy()
    m = out >= spec.base_blocks
    out[m] -= spec.base_blocks
    return out
