"""Decode parity: the HIP split-K kernel through the C ABI against the oracle."""
import numpy as np
import pytest
import torch

from workloads import DECODE_B256, TINY_DECODE_F32, make_batch, make_batch_from_lens
from tests.gpu_helpers import seq_bounds, Dev, assert_parity, f64, oracle_decode, require_gpu, say

pytestmark = pytest.mark.gpu

RAGGED = [1, 15, 16, 17, 63, 64, 65, 511, 512, 513, 1023, 1024, 1025, 1500, 2049, 4097]


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def test_tiny_decode_f32_full():
    b = make_batch(TINY_DECODE_F32)
    say("decode tiny fp32", b.seq_lens.tolist())
    out = Dev(b).decode()
    torch.cuda.synchronize()
    assert_parity(out, oracle_decode(b), "f32", "tiny decode fp32", seq_bounds(b, decode=True))


@pytest.mark.parametrize("hq,hkv,d,dtype", [
    (32, 8, 128, "bf16"), (8, 8, 128, "bf16"), (16, 8, 128, "bf16"), (64, 8, 128, "bf16"),
    (8, 2, 64, "bf16"), (4, 4, 64, "bf16"), (8, 4, 64, "bf16"), (16, 2, 64, "bf16"),
    (12, 3, 128, "bf16"),
    (4, 2, 64, "f32"), (8, 8, 64, "f32"), (16, 4, 64, "f32"), (16, 2, 64, "f32"),
])
def test_ragged_lengths_full(hq, hkv, d, dtype):
    b = make_batch_from_lens(RAGGED, [1] * len(RAGGED), dtype=dtype, num_q_heads=hq,
                             num_kv_heads=hkv, head_dim=d, block_size=16, seed=101)
    say("decode ragged", hq, hkv, d, dtype)
    out = Dev(b).decode()
    torch.cuda.synchronize()
    assert_parity(out, oracle_decode(b), dtype, f"ragged {hq}/{hkv}/{d}/{dtype}",
                  seq_bounds(b, decode=True))


def test_decode_b256_full_size_every_sequence():
    """The full decode workload (256 sequences, lengths U[512, 4096]) against
    the oracle on every sequence, gated over the whole output and per
    sequence."""
    b = make_batch(DECODE_B256)
    say("decode 256 sequences, full size", b.num_seqs, int(b.seq_lens.sum()))
    out = Dev(b).decode()
    torch.cuda.synchronize()
    assert torch.isfinite(out.float()).all()
    assert_parity(out, oracle_decode(b), "bf16", "decode 256 sequences, all",
                  seq_bounds(b, decode=True))


def test_block_permutation_bitwise():
    kw = dict(dtype="bf16", num_q_heads=32, num_kv_heads=8, head_dim=128, block_size=16, seed=5)
    a = make_batch_from_lens(RAGGED, [1] * len(RAGGED), **kw)
    perm = np.random.default_rng(9).permutation(a.num_blocks).astype(np.int32)
    c = make_batch_from_lens(RAGGED, [1] * len(RAGGED), block_perm=perm, **kw)
    assert not np.array_equal(a.block_table, c.block_table)
    say("decode permutation")
    oa, oc = Dev(a).decode(), Dev(c).decode()
    torch.cuda.synchronize()
    assert torch.equal(oa.view(torch.int16), oc.view(torch.int16))


def _set_k_component(b, s, t, dim, value):
    """Write K[s][t][g=all][dim] in the stored layer (chunk-major K tile)."""
    tile = b.block_size * b.head_dim
    vec = 16 // b.esz
    blk = int(b.block_table[s, t // b.block_size])
    layer = b.kv_layer.view(b.num_blocks, 2, b.num_kv_heads, tile)
    layer[blk, 0, :, ((dim // vec) * b.block_size + t % b.block_size) * vec + dim % vec] = value


@pytest.mark.parametrize("j", [0, 517, 1499])
def test_one_hot_probe_exact(j):
    """q[0] = 16 and k_j[0] = 100: every other weight underflows to zero in
    fp32, so the output must be exactly v_j (checks the gather bit for bit)."""
    b = make_batch_from_lens([1500], [1], dtype="bf16", num_q_heads=32, num_kv_heads=8,
                             head_dim=128, block_size=16, seed=7, keep_contig=True)
    b.q[0, :, 0] = 16.0
    _set_k_component(b, 0, j, 0, 100.0)
    say("decode one-hot", j)
    out = Dev(b).decode()
    torch.cuda.synchronize()
    v = b.v_contig[0][j]                       # [Hkv, d] bf16
    want = v.repeat_interleave(4, dim=0)       # query head h reads kv head h // 4
    assert torch.equal(out[0].cpu().view(torch.int16), want.view(torch.int16))


def test_single_token_and_empty_sequences():
    b = make_batch_from_lens([1, 0, 1, 0], [1, 0, 1, 0], dtype="bf16", num_q_heads=8,
                             num_kv_heads=2, head_dim=128, block_size=16, seed=8,
                             keep_contig=True)
    d = Dev(b)
    q4 = torch.full((4, 8, 128), 3.0, dtype=torch.bfloat16, device="cuda")
    q4[0], q4[2] = d.q[0], d.q[1]       # decode: one query row per sequence, even if empty
    d.q = q4
    say("decode L=1 / L=0")
    out = d.decode().cpu()
    for s in (0, 2):
        want = b.v_contig[s][0].repeat_interleave(4, dim=0)
        assert torch.equal(out[s].view(torch.int16), want.view(torch.int16))
    assert (out[1] == 0).all() and (out[3] == 0).all()
