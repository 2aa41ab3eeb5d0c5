"""kv_append on the GPU: byte-for-byte against the CPU oracle (a copy has no
rounding), then inside the two engine flows it exists for: a decode step that
writes its token and attends to it, and a prompt prefilled chunk by chunk with
each chunk's K/V written just before it attends."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_23658_amd.kvattn as K
from workloads import make_batch_from_lens
from workloads.append import make_append, next_slots
from tests.gpu_helpers import seq_bounds, Dev, assert_parity, oracle_decode, oracle_prefill, require_gpu, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _np(t: torch.Tensor) -> np.ndarray:
    t = t.cpu()
    return t.view(torch.int16).numpy().view(np.uint16) if t.dtype == torch.bfloat16 else t.numpy()


@pytest.mark.parametrize("dtype,hkv,d,T,nb,pad", [
    ("bf16", 8, 128, 300, 64, 0.1),
    ("f32", 2, 64, 77, 16, 0.2),
    ("bf16", 4, 64, 1, 4, 0.0),
    ("bf16", 8, 128, 4096, 300, 0.0),
    ("bf16", 1, 256, 50, 8, 0.5),
])
def test_append_bitwise_vs_oracle(dtype, hkv, d, T, nb, pad):
    say("append", dtype, hkv, d, T, nb, pad)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    g = torch.Generator().manual_seed(1234 + T)
    n = nb * 2 * hkv * 16 * d
    layer = torch.randn(n, generator=g).to(tdt)
    a = make_append(T, num_kv_heads=hkv, head_dim=d, dtype=dtype, num_blocks=nb,
                    block_size=16, seed=T + 7, pad_fraction=pad)
    if T > 4:
        a.slot_mapping[1] = nb * 16            # one past the layer
        a.slot_mapping[3] = nb * 16 + 1000
    ref = oracle.kv_append(_np(layer), a.k_raw(), a.v_raw(), a.slot_mapping, dtype=dtype,
                           num_kv_heads=hkv, head_dim=d, block_size=16)
    dl = layer.cuda()
    K.kv_append(a.k_new.cuda(), a.v_new.cuda(), torch.from_numpy(a.slot_mapping).cuda(), dl, nb)
    torch.cuda.synchronize()
    got = _np(dl)
    assert np.array_equal(got.view(np.uint8), ref.view(np.uint8))


def test_append_empty_and_all_padding():
    say("append empty / all padding")
    layer = torch.randn(4 * 2 * 2 * 16 * 64).to(torch.bfloat16).cuda()
    before = layer.clone()
    e = torch.empty(0, 2, 64, dtype=torch.bfloat16, device="cuda")
    K.kv_append(e, e, torch.empty(0, dtype=torch.int32, device="cuda"), layer, 4)
    k = torch.randn(9, 2, 64).to(torch.bfloat16).cuda()
    K.kv_append(k, k, torch.full((9,), -1, dtype=torch.int32, device="cuda"), layer, 4)
    torch.cuda.synchronize()
    assert torch.equal(layer.view(torch.int16), before.view(torch.int16))


def test_decode_step_writes_its_token_then_attends():
    """Each sequence's new token goes to slot seq_len (its table already holds
    that block), then decode runs over seq_len + 1 tokens."""
    lens = np.array([15, 16, 100, 257, 1024, 3000], dtype=np.int32)
    b = make_batch_from_lens(lens + 1, np.ones_like(lens), dtype="bf16", num_q_heads=32,
                             num_kv_heads=8, head_dim=128, block_size=16, seed=77)
    a = make_append(len(lens), num_kv_heads=8, head_dim=128, dtype="bf16",
                    num_blocks=b.num_blocks, block_size=16, seed=78)
    slots = next_slots(b.block_table, lens, 16)
    assert (slots >= 0).all()
    say("decode step append", lens.tolist())
    dev = Dev(b)
    K.kv_append(a.k_new.cuda(), a.v_new.cuda(), torch.from_numpy(slots).cuda(), dev.kv,
                b.num_blocks)
    out = dev.decode()
    b.kv_layer = torch.from_numpy(
        oracle.kv_append(b.kv_raw(), a.k_raw(), a.v_raw(), slots, dtype="bf16",
                         num_kv_heads=8, head_dim=128, block_size=16).view(np.int16)
    ).view(torch.bfloat16)
    assert_parity(out, oracle_decode(b), "bf16", "decode after append",
                  seq_bounds(b, decode=True))


def test_prompt_prefilled_chunk_by_chunk_with_append():
    """A 1024-token prompt in four 256-token chunks: every chunk's K/V is
    appended into an empty (NaN) layer right before the chunk attends; the
    concatenated outputs match the oracle on the whole prompt, and the layer
    ends up holding exactly the prompt's rows."""
    L, n = 1024, 256
    b = make_batch_from_lens([L], [L], dtype="bf16", num_q_heads=32, num_kv_heads=8,
                             head_dim=128, block_size=16, seed=91, keep_contig=True)
    nan_layer = torch.full_like(b.kv_layer, float("nan")).cuda()
    bt = torch.from_numpy(b.block_table).cuda()
    q = b.q.cuda()
    k_all, v_all = b.k_contig[0].cuda(), b.v_contig[0].cuda()
    t = np.arange(L)
    slots_all = (b.block_table[0][t // 16].astype(np.int64) * 16 + t % 16).astype(np.int32)
    out = torch.empty_like(q)
    for c0 in range(0, L, n):
        say("chunk", c0)
        sl = torch.tensor([c0 + n], dtype=torch.int32, device="cuda")
        cu = torch.tensor([0, n], dtype=torch.int32, device="cuda")
        K.kv_append(k_all[c0:c0 + n].contiguous(), v_all[c0:c0 + n].contiguous(),
                    torch.from_numpy(slots_all[c0:c0 + n]).cuda(), nan_layer, b.num_blocks)
        out[c0:c0 + n] = K.prefill_chunk(q[c0:c0 + n].contiguous(), nan_layer, b.num_blocks, bt,
                                         sl, cu, num_kv_heads=8, max_seq_len=L, scale=b.scale)
    assert_parity(out, oracle_prefill(b), "bf16", "chunked prefill with append")
    got = _np(nan_layer)
    ref = b.kv_raw()
    assert np.array_equal(got.view(np.uint8), ref.view(np.uint8))
