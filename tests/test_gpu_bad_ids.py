"""Block ids outside [0, num_blocks) are skipped: their 16 keys contribute
nothing, for decode and for prefill. The expectation is computed by brute
force with a library routine (torch's scaled_dot_product_attention in fp64 on
the contiguous K/V), with an explicit mask that removes the skipped block's
positions as well as the causal future."""
import numpy as np
import pytest
import torch

from workloads import make_batch_from_lens
from tests.gpu_helpers import Dev, assert_parity, require_gpu, say, seq_bounds

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _expected(b, skipped):
    """fp64 attention with the positions of skipped blocks removed."""
    T = b.total_q_tokens
    out = np.zeros((T, b.num_q_heads, b.head_dim))
    qf = b.q.to(torch.float64)
    for s in range(b.num_seqs):
        L = int(b.seq_lens[s])
        r0, r1 = int(b.cu_seqlens_q[s]), int(b.cu_seqlens_q[s + 1])
        n = r1 - r0
        k = b.k_contig[s].to(torch.float64).permute(1, 0, 2)[None]
        v = b.v_contig[s].to(torch.float64).permute(1, 0, 2)[None]
        q = qf[r0:r1].permute(1, 0, 2)[None]
        pos = torch.arange(L - n, L)[:, None]
        t = torch.arange(L)[None, :]
        allowed = t <= pos
        for j in skipped.get(s, []):
            allowed &= ~((t >= 16 * j) & (t < 16 * j + 16))
        o = torch.nn.functional.scaled_dot_product_attention(
            q, k, v, attn_mask=allowed, scale=b.scale, enable_gqa=True)
        o = o[0].permute(1, 0, 2).numpy()
        # a row that sees no key at all gets zeros, as a sequence of length 0 does
        o[~allowed.any(dim=1).numpy()] = 0.0
        out[r0:r1] = o
    return out


@pytest.mark.parametrize("mode", ["decode", "prefill"])
def test_out_of_range_ids_contribute_nothing(mode):
    lens = [300, 200, 130]
    q_lens = [1, 1, 1] if mode == "decode" else [100, 200, 7]
    b = make_batch_from_lens(lens, q_lens, dtype="bf16", num_q_heads=8, num_kv_heads=2,
                             head_dim=128, block_size=16, seed=21, keep_contig=True)
    skipped = {0: [3], 1: [0, 5], 2: [8]}
    d = Dev(b)
    bt = b.block_table.copy()
    bt[0, 3] = b.num_blocks + 1000
    bt[1, 0] = -5
    bt[1, 5] = 1 << 30
    bt[2, 8] = b.num_blocks        # the last block of sequence 2 (a partial block)
    d.bt = torch.from_numpy(bt).cuda()
    say("bad ids", mode, skipped)
    out = d.decode() if mode == "decode" else d.prefill()
    torch.cuda.synchronize()
    assert torch.isfinite(out.float()).all()
    assert_parity(out, _expected(b, skipped), "bf16", f"{mode} with skipped blocks",
                  seq_bounds(b, decode=(mode == "decode")))
