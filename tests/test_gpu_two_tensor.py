"""The two-tensor layer (the alternative the paper rejects): decode with the
top block ids in a second, separately allocated tensor gives bit for bit the
result of the one-range decode over the same bytes, and matches the oracle."""
import numpy as np
import pytest
import torch

import paper_2608_23658_amd.kvattn as K
from workloads import make_batch_from_lens
from tests.gpu_helpers import seq_bounds, Dev, assert_parity, oracle_decode, require_gpu, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


@pytest.mark.parametrize("hq,split", [(32, 0.8), (64, 0.5), (8, 0.9)])
def test_two_tensor_equals_one_range_bitwise(hq, split):
    lens = [1, 15, 16, 100, 700, 1500, 3333, 64]
    b = make_batch_from_lens(lens, [1] * len(lens), dtype="bf16", num_q_heads=hq,
                             num_kv_heads=8, head_dim=128, block_size=16, seed=hq)
    nb = b.num_blocks
    nbase = int(split * nb)
    ids = np.concatenate([b.block_table[s, :-(-L // 16)] for s, L in enumerate(lens)])
    assert (ids >= nbase).any() and (ids < nbase).any()
    say("two-tensor decode", hq, nb, nbase)
    dev = Dev(b)
    one = dev.decode()
    per_block = 2 * 8 * 16 * 128
    kv_base = dev.kv[:nbase * per_block]
    kv_el = dev.kv[nbase * per_block:].clone()          # a separate allocation
    two = K.decode_two_tensor(dev.q, kv_base, nbase, kv_el, nb - nbase, dev.bt, dev.sl,
                              num_kv_heads=8, max_seq_len=b.max_seq_len, scale=b.scale)
    torch.cuda.synchronize()
    assert torch.equal(one.view(torch.int16), two.view(torch.int16))
    assert_parity(two, oracle_decode(b), "bf16", "two-tensor decode", seq_bounds(b, decode=True))
