"""Chunked-prefill parity: the HIP MFMA kernel through the C ABI against the oracle."""
import numpy as np
import pytest
import torch

from workloads import MIXED_STEP, PREFILL_L32768, make_batch, make_batch_from_lens
from tests.gpu_helpers import (seq_bounds, Dev, assert_parity, f64, oracle_decode, oracle_prefill,
                               oracle_rows, require_gpu, say)

pytestmark = pytest.mark.gpu

MIXED_L = [37, 100, 300, 513, 1, 64, 1000, 129, 2048]
MIXED_N = [37, 20, 1, 257, 1, 16, 300, 65, 2048]


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


# (24, 6) and (6, 3): kv head counts that are not powers of two, so the block
# size is not either and block offsets take the multiply path
@pytest.mark.parametrize("hq,hkv", [(32, 8), (8, 8), (16, 8), (4, 1), (24, 6), (6, 3),
                                    (64, 8), (8, 1), (48, 6)])
def test_mixed_chunks_full(hq, hkv):
    b = make_batch_from_lens(MIXED_L, MIXED_N, dtype="bf16", num_q_heads=hq, num_kv_heads=hkv,
                             head_dim=128, block_size=16, seed=31)
    say("prefill mixed", hq, hkv)
    out = Dev(b).prefill()
    torch.cuda.synchronize()
    assert_parity(out, oracle_prefill(b), "bf16", f"mixed {hq}/{hkv}", seq_bounds(b))


def test_sequences_without_new_rows():
    """Sequences that add no rows in this call (n = 0, with and without cached
    context, first, middle and last in the batch) produce nothing and leave
    their neighbours unchanged."""
    L = [0, 40, 300, 0, 17, 2000, 64, 500]
    N = [0, 0, 300, 0, 17, 0, 1, 0]
    b = make_batch_from_lens(L, N, dtype="bf16", num_q_heads=32, num_kv_heads=8,
                             head_dim=128, block_size=16, seed=41)
    say("prefill rowless sequences")
    out = Dev(b).prefill()
    torch.cuda.synchronize()
    assert out.shape[0] == sum(N)
    assert_parity(out, oracle_prefill(b), "bf16", "rowless sequences", seq_bounds(b))


def test_first_row_is_v0_exactly():
    b = make_batch_from_lens([70], [70], dtype="bf16", num_q_heads=32, num_kv_heads=8,
                             head_dim=128, block_size=16, seed=3, keep_contig=True)
    say("prefill first row")
    out = Dev(b).prefill().cpu()
    want = b.v_contig[0][0].repeat_interleave(4, dim=0)
    assert torch.equal(out[0].view(torch.int16), want.view(torch.int16))


def test_causality_bitwise():
    """Changing K/V after position p leaves rows up to p unchanged bit for bit."""
    b = make_batch_from_lens([700], [700], dtype="bf16", num_q_heads=32, num_kv_heads=8,
                             head_dim=128, block_size=16, seed=4)
    d = Dev(b)
    say("prefill causality")
    ref = d.prefill().clone()
    p = 450
    tile = b.block_size * b.head_dim
    layer = d.kv.view(b.num_blocks, 2, b.num_kv_heads, tile)
    for blk in b.block_table[0, (p + 1 + 15) // 16: (700 + 15) // 16]:
        layer[int(blk)] = 3.0
    # the partial block holding p + 1 .. : rewrite the slots after p
    blk = int(b.block_table[0, (p + 1) // 16])
    kt = layer[blk, 0].view(b.num_kv_heads, 16, 16, 8)
    vt = layer[blk, 1].view(b.num_kv_heads, 128, 16)
    for t in range(p + 1, (p // 16 + 1) * 16):
        kt[:, :, t % 16, :] = -2.0
        vt[:, :, t % 16] = 5.0
    got = d.prefill()
    torch.cuda.synchronize()
    assert torch.equal(got[:p + 1].view(torch.int16), ref[:p + 1].view(torch.int16))
    assert not torch.equal(got[p + 1:], ref[p + 1:])


def test_prefill_l32768_chunk_equivalence():
    """One 32768-token chunk versus four 8192-token chunks over the same cache:
    both match the oracle, and the row tiling makes them bitwise equal."""
    b = make_batch(PREFILL_L32768)
    d = Dev(b)
    say("prefill 32768 whole")
    whole = d.prefill(max_num_batched_tokens=32768)
    parts = []
    for k in range(4):
        say("prefill 32768 chunk", k)
        q = d.q[8192 * k: 8192 * (k + 1)]
        sl = torch.tensor([8192 * (k + 1)], dtype=torch.int32, device="cuda")
        cu = torch.tensor([0, 8192], dtype=torch.int32, device="cuda")
        import paper_2608_23658_amd.kvattn as K
        parts.append(K.prefill_chunk(q, d.kv, b.num_blocks, d.bt, sl, cu, num_kv_heads=8,
                                     max_seq_len=32768, max_num_batched_tokens=8192,
                                     scale=b.scale))
    chunked = torch.cat(parts)
    torch.cuda.synchronize()
    # one row in every 256-row tile (at a different offset in each), plus the
    # first and last rows of the chunks and of a few tiles
    rng = np.random.default_rng(1)
    rows = sorted(set([256 * t + int(o) for t, o in enumerate(rng.integers(0, 256, 128))]
                      + [0, 1, 63, 64, 255, 256, 8191, 8192, 16383, 24576, 32767]))
    assert len({r // 256 for r in rows}) == 128
    say("oracle rows", len(rows))
    ref = oracle_rows(b, rows)
    assert_parity(f64(whole)[rows], ref, "bf16", "32768 whole, sampled rows")
    assert_parity(f64(chunked)[rows], ref, "bf16", "32768 as 4x8192, sampled rows")
    assert torch.equal(whole.view(torch.int16), chunked.view(torch.int16))


def test_mixed_step_chunk_plus_decode():
    """The last 8192-token chunk of a 32768-token prompt plus 128 decode
    sequences: as one unified call, and as a prefill call plus a decode call."""
    b = make_batch(MIXED_STEP)
    d = Dev(b)
    say("mixed step, unified call")
    uni = d.prefill(max_num_batched_tokens=8192 + 128)
    torch.cuda.synchronize()
    # one chunk row in every 256-row tile, and every decode row
    rng = np.random.default_rng(2)
    rows = sorted(set([256 * t + int(o) for t, o in enumerate(rng.integers(0, 256, 32))]
                      + [0, 1, 4095, 8191] + list(range(8192, 8192 + 128))))
    say("oracle rows", len(rows))
    ref = oracle_rows(b, rows)
    assert_parity(f64(uni)[rows], ref, "bf16", "mixed step, unified")
    # decode part alone through the decode kernel
    import paper_2608_23658_amd.kvattn as K
    qd = d.q[8192:]
    say("mixed step, decode part")
    dec = K.decode(qd, d.kv, b.num_blocks, d.bt[1:], d.sl[1:], num_kv_heads=8,
                   max_seq_len=b.max_seq_len, scale=b.scale)
    torch.cuda.synchronize()
    drows = [r for r in rows if r >= 8192]
    assert_parity(f64(dec)[[r - 8192 for r in drows]], ref[[rows.index(r) for r in drows]],
                  "bf16", "mixed step, decode part")


def test_reference_moves_mid_sequence():
    """Scores that jump far above everything before them, late in the context
    and inside the chunk: every query row carries a shared direction u, and the
    keys at three positions are a * u with a growing, so each of those keys
    outgrows the rows' reference by more than 2^8. The kernel must move the
    reference, rescale O and the row sum, and redo the step's exponentials
    (prefill), or rescale its running state (decode), and still match the
    oracle. The keys are written into the layer by the oracle's own append."""
    import oracle
    import paper_2608_23658_amd.kvattn as K
    L, n = 2500, 600
    b = make_batch_from_lens([L], [n], dtype="bf16", num_q_heads=32, num_kv_heads=8,
                             head_dim=128, block_size=16, seed=77)
    g = torch.Generator().manual_seed(78)
    u = torch.randn(128, generator=g)
    u = u / u.norm()
    b.q = (b.q.float() + 2.0 * 128 ** 0.5 * u).to(torch.bfloat16)
    pos = np.array([900, 1700, 2400])
    amp = [4.0, 8.0, 16.0]
    k_new = torch.stack([a * u.expand(8, 128) for a in amp]).to(torch.bfloat16)
    v_new = torch.randn(3, 8, 128, generator=g).to(torch.bfloat16)
    slots = (b.block_table[0][pos // 16].astype(np.int64) * 16 + pos % 16).astype(np.int32)
    u16 = lambda t: t.view(torch.int16).numpy().view(np.uint16)
    raw = oracle.kv_append(b.kv_raw(), u16(k_new), u16(v_new), slots, dtype="bf16",
                           num_kv_heads=8, head_dim=128, block_size=16)
    b.kv_layer = torch.from_numpy(raw.view(np.int16)).view(torch.bfloat16)
    say("prefill with late score jumps at", pos.tolist())
    dev = Dev(b)
    out = dev.prefill()
    torch.cuda.synchronize()
    ref = oracle_prefill(b)
    # the rows at and after the last jump attend to it almost alone
    assert np.abs(ref[pos[2] - (L - n):, 0] - f64(v_new[2, 0])).max() < 1e-3
    assert_parity(out, ref, "bf16", "prefill with late score jumps", seq_bounds(b))
    say("decode over the same layer")
    qd = b.q[-1:].contiguous()
    od = K.decode(qd.cuda(), dev.kv, b.num_blocks, dev.bt, dev.sl, num_kv_heads=8,
                  max_seq_len=L, scale=b.scale)
    torch.cuda.synchronize()
    refd = oracle.paged_decode(u16(qd), raw, b.block_table, b.seq_lens, dtype="bf16",
                               num_q_heads=32, num_kv_heads=8, head_dim=128, block_size=16,
                               scale=b.scale)
    assert_parity(od, refd, "bf16", "decode with late score jumps")
