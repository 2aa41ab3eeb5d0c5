"""Long contexts: 131072 tokens (128 decode splits merged by the combine, 2048
prefill key steps per tile), next to a ragged 65543-token sequence and a
1-token one, on one paged layer. Decode in full and prefill on sampled rows
against the oracle (Section 5: a chunk attends to all prior context)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_23658_amd.kvattn as K
from workloads import make_batch_from_lens
from tests.gpu_helpers import Dev, assert_parity, oracle_decode, require_gpu, say, seq_bounds

pytestmark = pytest.mark.gpu

LENS = [131072, 65543, 1]


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


@pytest.fixture(scope="module")
def batch():
    b = make_batch_from_lens(LENS, [1] * len(LENS), dtype="bf16", num_q_heads=32,
                             num_kv_heads=8, head_dim=128, block_size=16, seed=131072)
    return b, Dev(b)


def test_long_context_decode(batch):
    b, dev = batch
    say("long-context decode", LENS, "splits", K.decode_split_tokens(max(LENS)))
    out = dev.decode()
    torch.cuda.synchronize()
    assert_parity(out, oracle_decode(b), "bf16", f"long-context decode {LENS}",
                  seq_bounds(b, decode=True))


def test_long_context_prefill_rows(batch):
    b, dev = batch
    news = [2048, 7, 1]
    cu = np.concatenate([[0], np.cumsum(news)]).astype(np.int32)
    g = torch.Generator().manual_seed(131073)
    q = torch.randn(int(cu[-1]), 32, 128, generator=g).to(torch.bfloat16)
    say("long-context prefill", news, "new rows of", LENS)
    out = K.prefill_chunk(q.cuda(), dev.kv, b.num_blocks, dev.bt, dev.sl,
                          torch.from_numpy(cu).cuda(), num_kv_heads=8,
                          max_seq_len=max(LENS), scale=b.scale)
    torch.cuda.synchronize()
    rng = np.random.default_rng(7)
    rows = sorted({0, 1, 255, 256, 2047} | set(rng.integers(0, 2048, 3).tolist())
                  | set(range(2048, int(cu[-1]))))
    qraw = q.view(torch.int16).numpy().view(np.uint16)
    ref = oracle.paged_attention_rows(qraw, b.kv_raw(), b.block_table, b.seq_lens, cu, rows,
                                      dtype="bf16", num_q_heads=32, num_kv_heads=8,
                                      head_dim=128, block_size=16, scale=b.scale)
    got = out[torch.tensor(rows, device="cuda")]
    # the sampled rows are sorted, so each sequence's rows are contiguous in them
    bounds = np.searchsorted(rows, cu)
    assert_parity(got, ref, "bf16", f"long-context prefill rows {rows}", bounds)
