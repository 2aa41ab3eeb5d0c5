"""Seeded random sweeps of decode and prefill against the oracle: batch sizes,
lengths (with block, step and split boundaries mixed in), head layouts and
dtypes drawn per case, each case printed before it runs."""
import numpy as np
import pytest
import torch

from workloads import make_batch_from_lens
from tests.gpu_helpers import seq_bounds, Dev, assert_parity, oracle_decode, oracle_prefill, require_gpu, say

pytestmark = pytest.mark.gpu

# lengths that sit on a block (16), step (64) or split (1024) boundary
EDGES = [0, 1, 15, 16, 17, 63, 64, 65, 1023, 1024, 1025]
DECODE_SHAPES = [(32, 8, 128, "bf16"), (8, 8, 128, "bf16"), (16, 8, 128, "bf16"),
                 (64, 8, 128, "bf16"), (8, 2, 64, "bf16"), (16, 2, 64, "bf16"),
                 (4, 2, 64, "f32"), (16, 4, 64, "f32"), (12, 3, 128, "bf16"), (24, 6, 64, "bf16")]
PREFILL_HEADS = [(32, 8), (8, 8), (16, 8), (4, 1), (24, 6), (6, 3), (64, 8), (16, 2)]


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


@pytest.mark.parametrize("seed", range(6))
def test_decode_random(seed):
    rng = np.random.default_rng(1000 + seed)
    hq, hkv, d, dtype = DECODE_SHAPES[rng.integers(len(DECODE_SHAPES))]
    B = int(rng.integers(1, 13))
    lens = [int(x) for x in rng.integers(0, 2600, size=B)]
    lens[int(rng.integers(B))] = int(rng.choice(EDGES))
    say("decode random", seed, hq, hkv, d, dtype, lens)
    b = make_batch_from_lens(lens, [1] * B, dtype=dtype, num_q_heads=hq, num_kv_heads=hkv,
                             head_dim=d, block_size=16, seed=2000 + seed)
    out = Dev(b).decode()
    torch.cuda.synchronize()
    assert_parity(out, oracle_decode(b), dtype, f"decode random {seed}",
                  seq_bounds(b, decode=True))


@pytest.mark.parametrize("seed", range(6))
def test_prefill_random(seed):
    rng = np.random.default_rng(3000 + seed)
    hq, hkv = PREFILL_HEADS[rng.integers(len(PREFILL_HEADS))]
    B = int(rng.integers(1, 6))
    n = [int(x) for x in rng.integers(0, 400, size=B)]
    c = [int(x) for x in rng.integers(0, 1200, size=B)]
    k = int(rng.integers(B))
    n[k] = int(rng.choice(EDGES[1:]))
    L = [ci + ni for ci, ni in zip(c, n)]
    say("prefill random", seed, hq, hkv, "L", L, "n", n)
    b = make_batch_from_lens(L, n, dtype="bf16", num_q_heads=hq, num_kv_heads=hkv, head_dim=128,
                             block_size=16, seed=4000 + seed)
    out = Dev(b).prefill()
    torch.cuda.synchronize()
    assert out.shape[0] == sum(n)
    assert_parity(out, oracle_prefill(b), "bf16", f"prefill random {seed}", seq_bounds(b))


def test_many_short_sequences():
    """Wide batches: 4096 decode sequences and 1024 prefill chunks of 1 to 64
    tokens (the decode grid and the prefill work-tile list at many entries),
    each sequence gated on its own."""
    rng = np.random.default_rng(4096)
    lens = [int(x) for x in rng.integers(1, 65, size=4096)]
    say("decode, 4096 sequences")
    b = make_batch_from_lens(lens, [1] * len(lens), dtype="bf16", num_q_heads=32, num_kv_heads=8,
                             head_dim=128, block_size=16, seed=4097)
    out = Dev(b).decode()
    torch.cuda.synchronize()
    assert_parity(out, oracle_decode(b), "bf16", "decode, 4096 sequences", seq_bounds(b, decode=True))
    lens = [int(x) for x in rng.integers(1, 65, size=1024)]
    n = [int(rng.integers(1, L + 1)) for L in lens]
    say("prefill, 1024 chunks")
    b = make_batch_from_lens(lens, n, dtype="bf16", num_q_heads=32, num_kv_heads=8,
                             head_dim=128, block_size=16, seed=4098)
    out = Dev(b).prefill()
    torch.cuda.synchronize()
    assert_parity(out, oracle_prefill(b), "bf16", "prefill, 1024 chunks", seq_bounds(b))
