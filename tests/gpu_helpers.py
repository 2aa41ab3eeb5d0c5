"""Shared pieces of the GPU parity tests: moving a generated batch to the
device, calling the HIP path through the binding, and the oracle side."""
import sys

import numpy as np
import torch

import oracle
import paper_2608_23658_amd.kvattn as K
from tests.tolerance import compare


def say(*a):
    """Name the case before a GPU step, flushed, so a failure names it."""
    print("[gpu]", *a, flush=True)
    sys.stdout.flush()


def require_gpu():
    assert torch.cuda.is_available(), "GPU test run without a GPU"
    K.lib()   # raises if the HIP library is missing


class Dev:
    """Device copies of a PagedBatch."""

    def __init__(self, b, kv=None):
        self.b = b
        self.q = b.q.cuda()
        self.kv = b.kv_layer.cuda() if kv is None else kv
        self.bt = torch.from_numpy(b.block_table).cuda()
        self.sl = torch.from_numpy(b.seq_lens).cuda()
        self.cu = torch.from_numpy(b.cu_seqlens_q).cuda()

    def decode(self, **kw):
        b = self.b
        return K.decode(self.q, self.kv, b.num_blocks, self.bt, self.sl,
                        num_kv_heads=b.num_kv_heads, max_seq_len=b.max_seq_len,
                        block_size=b.block_size, scale=b.scale, **kw)

    def prefill(self, **kw):
        b = self.b
        return K.prefill_chunk(self.q, self.kv, b.num_blocks, self.bt, self.sl, self.cu,
                               num_kv_heads=b.num_kv_heads, max_seq_len=b.max_seq_len,
                               block_size=b.block_size, scale=b.scale, **kw)


def oracle_decode(b, seqs=None):
    return oracle.paged_decode(b.q_raw(), b.kv_raw(), b.block_table, b.seq_lens, dtype=b.dtype,
                               num_q_heads=b.num_q_heads, num_kv_heads=b.num_kv_heads,
                               head_dim=b.head_dim, block_size=b.block_size, scale=b.scale,
                               seqs=seqs)


def oracle_prefill(b, seqs=None):
    return oracle.paged_attention(b.q_raw(), b.kv_raw(), b.block_table, b.seq_lens,
                                  b.cu_seqlens_q, dtype=b.dtype, num_q_heads=b.num_q_heads,
                                  num_kv_heads=b.num_kv_heads, head_dim=b.head_dim,
                                  block_size=b.block_size, scale=b.scale, seqs=seqs)


def oracle_rows(b, rows):
    return oracle.paged_attention_rows(b.q_raw(), b.kv_raw(), b.block_table, b.seq_lens,
                                       b.cu_seqlens_q, rows, dtype=b.dtype,
                                       num_q_heads=b.num_q_heads, num_kv_heads=b.num_kv_heads,
                                       head_dim=b.head_dim, block_size=b.block_size,
                                       scale=b.scale)


def f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().double().numpy()


def assert_parity(got, ref, dtype, what="", bounds=None):
    """The tolerance gate over the whole output; with ``bounds`` (row offsets
    of the sequences: ``cu_seqlens_q`` for prefill, ``0..B`` for decode) also
    over each sequence's rows on their own, so that the large outputs of short
    sequences cannot hide an error in the small outputs of long ones."""
    got = f64(got) if isinstance(got, torch.Tensor) else got
    r = compare(got, ref, dtype)
    say(what, f"max_abs={r['max_abs']:.3e} rel_l2={r['rel_l2']:.3e}")
    assert r["pass"], (what, r)
    if bounds is not None:
        worst = 0.0
        for s in range(len(bounds) - 1):
            lo, hi = int(bounds[s]), int(bounds[s + 1])
            if hi == lo:
                continue
            rs = compare(got[lo:hi], ref[lo:hi], dtype)
            assert rs["pass"], (what, "sequence", s, rs)
            worst = max(worst, rs["rel_l2"])
        say(what, f"worst sequence rel_l2={worst:.3e}")
    return r


def seq_bounds(b, decode=False):
    """Row offsets of each sequence's outputs in a batch's result."""
    return np.arange(len(b.seq_lens) + 1) if decode else b.cu_seqlens_q
