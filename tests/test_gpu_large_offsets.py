"""A 5 GiB layer whose sequences live in blocks past the first 4 GiB, so that
every byte offset needs 64 bits: the write of the tokens' K/V (kv_append),
chunked prefill, decode and a block copy, each against the oracle run on
just the referenced blocks (Section 3, "The contiguity constraint": one
tensor per layer, addressed by block id through one base pointer)."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2608_23658_amd.kvattn as K
from tests.gpu_helpers import assert_parity, f64, require_gpu, say

pytestmark = pytest.mark.gpu

NB = 81920                          # 64 KiB blocks: 5 GiB
HQ, HKV, D, BS = 32, 8, 128, 16
BLOCK_ELEMS = 2 * HKV * BS * D      # bf16 elements per block
HIGH = (1 << 32) // (BLOCK_ELEMS * 2)   # first block id at or past 4 GiB
BF16_NAN = 0x7FC0


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _u16(t: torch.Tensor) -> np.ndarray:
    return t.cpu().view(torch.int16).numpy().view(np.uint16)


def test_offsets_past_4gib():
    rng = np.random.default_rng(4096)
    lens = np.array([2348, 1000], np.int32)
    news = np.array([777, 256], np.int32)
    nblk = [math.ceil(int(L) / BS) for L in lens]
    # distinct ids past 4 GiB; the first sequence also holds the layer's last block
    pick = rng.choice(np.arange(HIGH, NB - 1), size=sum(nblk) + 1, replace=False)
    ids = np.concatenate([pick[:nblk[0] - 1], [NB - 1], pick[nblk[0] - 1:sum(nblk) - 1]])
    spare = int(pick[-1])                     # an unreferenced block for the copy
    assert ids.min() * BLOCK_ELEMS * 2 >= 1 << 32
    bt = np.full((2, max(nblk)), -1, np.int32)
    bt[0, :nblk[0]] = ids[:nblk[0]]
    bt[1, :nblk[1]] = ids[nblk[0]:]
    compact = {int(b): i for i, b in enumerate(ids)}
    bt_c = np.where(bt >= 0, np.vectorize(lambda x: compact.get(int(x), -1))(bt), -1)
    bt_c = bt_c.astype(np.int32)

    # every token of both sequences, written through its slot
    g = torch.Generator().manual_seed(4097)
    ntok = int(lens.sum())
    k_new = torch.randn(ntok, HKV, D, generator=g).to(torch.bfloat16)
    v_new = torch.randn(ntok, HKV, D, generator=g).to(torch.bfloat16)
    slots, slots_c = [], []
    for s, L in enumerate(lens):
        t = np.arange(int(L))
        slots.append(bt[s, t // BS].astype(np.int64) * BS + t % BS)
        slots_c.append(bt_c[s, t // BS].astype(np.int64) * BS + t % BS)
    slots = np.concatenate(slots).astype(np.int32)
    slots_c = np.concatenate(slots_c).astype(np.int32)
    host = np.full(len(ids) * BLOCK_ELEMS, BF16_NAN, np.uint16)
    ref_layer = oracle.kv_append(host, _u16(k_new), _u16(v_new), slots_c, dtype="bf16",
                                 num_kv_heads=HKV, head_dim=D, block_size=BS)

    say("large offsets: 5 GiB layer, kv_append of", ntok, "tokens past 4 GiB")
    layer = torch.full((NB * BLOCK_ELEMS,), float("nan"), dtype=torch.bfloat16, device="cuda")
    K.kv_append(k_new.cuda(), v_new.cuda(), torch.from_numpy(slots).cuda(), layer, NB)
    torch.cuda.synchronize()
    ids_t = torch.from_numpy(ids.astype(np.int64)).cuda()
    got = _u16(layer.view(NB, BLOCK_ELEMS).index_select(0, ids_t))
    assert np.array_equal(got.reshape(-1), ref_layer)

    bt_t = torch.from_numpy(bt).cuda()
    sl_t = torch.from_numpy(lens).cuda()
    scale = 1.0 / math.sqrt(D)

    say("large offsets: prefill", news.tolist(), "new rows of", lens.tolist())
    cu = np.concatenate([[0], np.cumsum(news)]).astype(np.int32)
    q = torch.randn(int(cu[-1]), HQ, D, generator=g).to(torch.bfloat16)
    out = K.prefill_chunk(q.cuda(), layer, NB, bt_t, sl_t, torch.from_numpy(cu).cuda(),
                          num_kv_heads=HKV, max_seq_len=int(lens.max()), scale=scale)
    torch.cuda.synchronize()
    ref = oracle.paged_attention(_u16(q), ref_layer, bt_c, lens, cu, dtype="bf16",
                                 num_q_heads=HQ, num_kv_heads=HKV, head_dim=D,
                                 block_size=BS, scale=scale)
    assert_parity(f64(out), ref, "bf16", "prefill past 4 GiB", cu)

    say("large offsets: decode of", lens.tolist())
    qd = torch.randn(2, HQ, D, generator=g).to(torch.bfloat16)
    od = K.decode(qd.cuda(), layer, NB, bt_t, sl_t, num_kv_heads=HKV,
                  max_seq_len=int(lens.max()), scale=scale)
    torch.cuda.synchronize()
    refd = oracle.paged_decode(_u16(qd), ref_layer, bt_c, lens, dtype="bf16",
                               num_q_heads=HQ, num_kv_heads=HKV, head_dim=D,
                               block_size=BS, scale=scale)
    assert_parity(f64(od), refd, "bf16", "decode past 4 GiB", np.arange(3))

    say("large offsets: copy block", NB - 1, "->", spare)
    K.copy_blocks([layer], NB, BLOCK_ELEMS * 2,
                  torch.tensor([NB - 1], dtype=torch.int32, device="cuda"),
                  torch.tensor([spare], dtype=torch.int32, device="cuda"))
    torch.cuda.synchronize()
    moved = _u16(layer.view(NB, BLOCK_ELEMS)[spare])
    assert np.array_equal(moved, ref_layer.reshape(-1, BLOCK_ELEMS)[compact[NB - 1]])
    del layer
    torch.cuda.empty_cache()
