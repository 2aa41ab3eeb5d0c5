"""Pins for the fp64 oracle: each checks it against something other than itself.

* brute force: torch's scaled_dot_product_attention (fp64, CPU) on the
  contiguous, un-paged copy of each sequence, with an explicit bottom-right
  causal mask and grouped-query heads;
* closed forms: K = 0 gives the mean of the visible V, constant V gives that
  constant, one key gives its value, two keys give a logistic mix;
* invariants: block-table permutation, chunking (bit-exact), causality,
  NaN poison outside the sequences;
* planted mistakes: wrong variants of the oracle must fail these pins.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import oracle.paged_kv as opa
from workloads import TINY_DECODE_F32, make_batch, make_batch_from_lens
from tests.tolerance import compare


def _run(b, seqs=None):
    return oracle.paged_attention(
        b.q_raw(), b.kv_raw(), b.block_table, b.seq_lens, b.cu_seqlens_q,
        dtype=b.dtype, num_q_heads=b.num_q_heads, num_kv_heads=b.num_kv_heads,
        head_dim=b.head_dim, block_size=b.block_size, scale=b.scale, seqs=seqs)


def _sdpa(b):
    """Brute force on the contiguous copy: library attention with a mask."""
    T = b.total_q_tokens
    out = np.zeros((T, b.num_q_heads, b.head_dim))
    qf = b.q.to(torch.float64)
    for s in range(b.num_seqs):
        L = int(b.seq_lens[s])
        r0, r1 = int(b.cu_seqlens_q[s]), int(b.cu_seqlens_q[s + 1])
        n = r1 - r0
        if n == 0:
            continue
        k = b.k_contig[s].to(torch.float64).permute(1, 0, 2)[None]   # [1, Hkv, L, d]
        v = b.v_contig[s].to(torch.float64).permute(1, 0, 2)[None]
        q = qf[r0:r1].permute(1, 0, 2)[None]                        # [1, Hq, n, d]
        pos = torch.arange(L - n, L)[:, None]
        allowed = torch.arange(L)[None, :] <= pos                    # bottom-right causal
        o = torch.nn.functional.scaled_dot_product_attention(
            q, k, v, attn_mask=allowed, scale=b.scale, enable_gqa=True)
        out[r0:r1] = o[0].permute(1, 0, 2).numpy()
    return out


MIXED = dict(seq_lens=[37, 100, 300, 513, 1, 64], q_lens=[37, 20, 1, 257, 1, 16])


@pytest.mark.parametrize("dtype,hq,hkv,d", [("f32", 4, 2, 64), ("bf16", 8, 2, 128),
                                             ("bf16", 4, 4, 64), ("f32", 8, 1, 32)])
def test_bruteforce_sdpa_mixed_chunks(dtype, hq, hkv, d):
    b = make_batch_from_lens(MIXED["seq_lens"], MIXED["q_lens"], dtype=dtype,
                             num_q_heads=hq, num_kv_heads=hkv, head_dim=d, block_size=16,
                             seed=11, keep_contig=True)
    got = _run(b)
    ref = _sdpa(b)
    assert np.max(np.abs(got - ref)) <= 1e-12


def test_bruteforce_sdpa_tiny_decode():
    b = make_batch(TINY_DECODE_F32, keep_contig=True)
    got = oracle.paged_decode(b.q_raw(), b.kv_raw(), b.block_table, b.seq_lens,
                              dtype=b.dtype, num_q_heads=b.num_q_heads,
                              num_kv_heads=b.num_kv_heads, head_dim=b.head_dim,
                              block_size=b.block_size, scale=b.scale)
    ref = _sdpa(b)
    assert np.max(np.abs(got - ref)) <= 1e-12
    assert b.scale == 1.0 / 8.0


def _layer_parts(b):
    """K and V parts of the stored layer as views [Nb, Hkv, tile]."""
    tile = b.block_size * b.head_dim
    x = b.kv_layer.view(b.num_blocks, 2, b.num_kv_heads, tile)
    return x[:, 0], x[:, 1]


def test_k_zero_gives_mean_of_visible_v():
    # Chunks with cached context: a top-left causal mask would average over
    # the wrong number of keys.
    b = make_batch_from_lens([40, 77, 300], [40, 13, 45], dtype="f32", num_q_heads=4,
                             num_kv_heads=2, head_dim=32, block_size=16, seed=3,
                             keep_contig=True)
    kpart, _ = _layer_parts(b)
    kpart.zero_()
    got = _run(b)
    for s in range(b.num_seqs):
        L = int(b.seq_lens[s])
        r0, r1 = int(b.cu_seqlens_q[s]), int(b.cu_seqlens_q[s + 1])
        v = b.v_contig[s].double().numpy()        # [L, Hkv, d]
        for i in range(r1 - r0):
            p = L - (r1 - r0) + i
            mean = v[:p + 1].mean(axis=0)          # [Hkv, d]
            for h in range(b.num_q_heads):
                np.testing.assert_allclose(got[r0 + i, h], mean[h // 2], rtol=0, atol=1e-13)


def test_constant_v_gives_constant():
    b = make_batch_from_lens([130, 64], [10, 1], dtype="bf16", num_q_heads=8,
                             num_kv_heads=2, head_dim=64, block_size=16, seed=5)
    _, vpart = _layer_parts(b)
    vpart.fill_(0.75)
    got = _run(b)
    assert np.max(np.abs(got - 0.75)) <= 1e-15


def test_single_key_is_its_value_bit_exact():
    b = make_batch_from_lens([1, 17], [1, 1], dtype="f32", num_q_heads=2, num_kv_heads=1,
                             head_dim=16, block_size=16, seed=9, keep_contig=True)
    got = _run(b)
    v0 = b.v_contig[0].double().numpy()[0, 0]
    assert np.array_equal(got[0, 0], v0) and np.array_equal(got[0, 1], v0)
    # The first row of a prefill chunk at position 0 sees only key 0 as well.
    c = make_batch_from_lens([50], [50], dtype="bf16", num_q_heads=4, num_kv_heads=2,
                             head_dim=32, block_size=16, seed=10, keep_contig=True)
    got = _run(c)
    v = c.v_contig[0].double().numpy()
    for h in range(4):
        assert np.array_equal(got[0, h], v[0, h // 2])


def test_two_keys_logistic_mix():
    """Hand-built layer: q = (a, 0, ..), k0 = 0, k1 = (x, 0, ..). Then
    out = (v0 + e^s v1) / (1 + e^s) with s = scale * a * x."""
    d, bs = 16, 16
    b = make_batch_from_lens([2], [1], dtype="f32", num_q_heads=1, num_kv_heads=1,
                             head_dim=d, block_size=bs, seed=1, keep_contig=True)
    a, x = 1.5, 2.25
    b.q.zero_()
    b.q[0, 0, 0] = a
    kpart, _ = _layer_parts(b)
    blk = int(b.block_table[0, 0])
    kpart[blk].zero_()
    kpart[blk, 0, 1 * 4 + 0] = x           # slot 1, dim 0: chunk 0, slot 1, lane 0 (VEC 4)
    got = _run(b)
    v = b.v_contig[0].double().numpy()[:, 0]
    s = b.scale * a * x
    want = (v[0] + math.exp(s) * v[1]) / (1.0 + math.exp(s))
    np.testing.assert_allclose(got[0, 0], want, rtol=0, atol=1e-14)


def test_duplicate_heads_identical():
    b = make_batch_from_lens([90, 33], [5, 1], dtype="bf16", num_q_heads=8, num_kv_heads=2,
                             head_dim=64, block_size=16, seed=12)
    b.q[:, 1] = b.q[:, 0]
    b.q[:, 3] = b.q[:, 0]
    got = _run(b)
    assert np.array_equal(got[:, 0], got[:, 1]) and np.array_equal(got[:, 0], got[:, 3])
    assert not np.array_equal(got[:, 0], got[:, 4])      # another group differs


def test_block_permutation_invariance_bit_exact():
    lens, ql = [200, 31, 517], [1, 1, 60]
    kw = dict(dtype="bf16", num_q_heads=8, num_kv_heads=2, head_dim=64, block_size=16, seed=21)
    a = make_batch_from_lens(lens, ql, **kw)
    rng = np.random.default_rng(5)
    perm = rng.permutation(a.num_blocks).astype(np.int32)
    b = make_batch_from_lens(lens, ql, block_perm=perm, **kw)
    assert not np.array_equal(a.block_table, b.block_table)
    assert np.array_equal(_run(a), _run(b))


def test_chunk_equivalence_bit_exact():
    """One 1024-token pass equals four 256-token chunks, bit for bit."""
    kw = dict(dtype="bf16", num_q_heads=4, num_kv_heads=1, head_dim=64, block_size=16)
    whole = make_batch_from_lens([1024], [1024], seed=33, **kw)
    ref = _run(whole)
    q = whole.q_raw()
    for k in range(4):
        L = 256 * (k + 1)
        got = oracle.paged_attention(
            q[256 * k:L], whole.kv_raw(), whole.block_table, np.array([L], np.int32),
            np.array([0, 256], np.int32), dtype="bf16", num_q_heads=4, num_kv_heads=1,
            head_dim=64, block_size=16, scale=whole.scale)
        assert np.array_equal(got, ref[256 * k:L])


def test_causality_future_keys_do_not_matter():
    kw = dict(dtype="f32", num_q_heads=2, num_kv_heads=1, head_dim=32, block_size=16)
    b = make_batch_from_lens([300], [300], seed=44, **kw)
    ref = _run(b)
    kpart, vpart = _layer_parts(b)
    # Overwrite tokens 200..299 (blocks 12.5 .. 18) with new finite values.
    for t in range(200, 300):
        blk = int(b.block_table[0, t // 16])
        r = t % 16
        kview = kpart[blk].view(1, 32 // 4, 16, 4)
        vview = vpart[blk].view(1, 32, 16)
        kview[:, :, r, :] = 3.0
        vview[:, :, r] = -2.0
    got = _run(b)
    assert np.array_equal(got[:200], ref[:200])
    assert not np.allclose(got[200:], ref[200:])


def test_nan_poison_and_padding_never_read():
    b = make_batch(TINY_DECODE_F32)
    raw = b.kv_raw()
    assert np.isnan(raw).sum() > 0           # free blocks and tail slots are poisoned
    bt = b.block_table.copy()
    nblk = -(-b.seq_lens // 16)
    for s in range(b.num_seqs):
        bt[s, nblk[s]:] = 10 ** 9           # would raise if read
    got = oracle.paged_decode(b.q_raw(), raw, bt, b.seq_lens, dtype="f32", num_q_heads=4,
                              num_kv_heads=2, head_dim=64, block_size=16, scale=b.scale)
    assert np.all(np.isfinite(got))


def test_one_hot_probe():
    """A key aligned with a huge query component takes all the weight."""
    b = make_batch_from_lens([70], [1], dtype="bf16", num_q_heads=4, num_kv_heads=1,
                             head_dim=128, block_size=16, seed=50, keep_contig=True)
    j = 53
    b.q[0, :, 0] = 16.0
    kpart, _ = _layer_parts(b)
    blk = int(b.block_table[0, j // 16])
    kpart[blk].view(1, 16, 16, 8)[0, 0, j % 16, 0] = 100.0
    got = _run(b)
    vj = b.v_contig[0].double().numpy()[j, 0]
    for h in range(4):
        np.testing.assert_allclose(got[0, h], vj, rtol=0, atol=1e-12)


def test_decode_equals_prefill_with_one_row_and_empty_sequence():
    b = make_batch_from_lens([45, 0, 160], [1, 0, 1], dtype="bf16", num_q_heads=4,
                             num_kv_heads=2, head_dim=64, block_size=16, seed=60)
    pre = _run(b)
    q3 = torch.randn(3, 4, 64, generator=torch.Generator().manual_seed(1)).to(torch.bfloat16)
    q3[0] = b.q[0]
    q3[2] = b.q[1]
    qraw = q3.view(torch.int16).numpy().view(np.uint16)
    dec = oracle.paged_decode(qraw, b.kv_raw(), b.block_table, b.seq_lens, dtype="bf16",
                              num_q_heads=4, num_kv_heads=2, head_dim=64, block_size=16,
                              scale=b.scale)
    assert np.array_equal(dec[0], pre[0]) and np.array_equal(dec[2], pre[1])
    assert np.all(dec[1] == 0)


def test_row_sampler_agrees_with_full():
    b = make_batch_from_lens(MIXED["seq_lens"], MIXED["q_lens"], dtype="bf16",
                             num_q_heads=8, num_kv_heads=2, head_dim=64, block_size=16, seed=70)
    full = _run(b)
    rows = [0, 36, 37, 50, 57, 58, 100, 314, 315, 316]
    got = oracle.paged_attention_rows(b.q_raw(), b.kv_raw(), b.block_table, b.seq_lens,
                                      b.cu_seqlens_q, rows, dtype="bf16", num_q_heads=8,
                                      num_kv_heads=2, head_dim=64, block_size=16,
                                      scale=b.scale)
    assert np.max(np.abs(got - full[rows])) <= 1e-12


# ---- planted mistakes: each wrong variant must fail a pin above ------------

_ATTEND = opa.attend
_GATHER = opa.gather_kv

def _gqa_mod(qf, K, V, context, scale):
    """Mistake: query head h reads KV head h % Hkv instead of h // G."""
    n, hq, d = qf.shape
    hkv = K.shape[1]
    perm = [(h % hkv) * (hq // hkv) + h // hkv for h in range(hq)]
    return _ATTEND(qf[:, perm], K, V, context, scale)[:, np.argsort(perm)]


def _top_left(qf, K, V, context, scale):
    """Mistake: causal mask aligned top-left (row i sees keys 0..i)."""
    n = qf.shape[0]
    return _ATTEND(qf, K[:n], V[:n], 0, scale)


def _v_row_major(kv_raw, dtype, block_ids, seq_len, hkv, bs, d):
    """Mistake: V tile read as slot-major instead of dim-major."""
    K, _ = _GATHER(kv_raw, dtype, block_ids, seq_len, hkv, bs, d)
    tile = bs * d
    nb = kv_raw.size // (2 * hkv * tile)
    layer = kv_raw.reshape(nb, 2, hkv, tile)
    nblk = -(-seq_len // bs)
    V = np.concatenate([opa.storage_to_f64(layer[int(b), 1], dtype).reshape(hkv, bs, d)
                        .transpose(1, 0, 2) for b in block_ids[:nblk]])
    return K, V[:seq_len]


@pytest.mark.parametrize("mutant", ["gqa", "top_left", "v_layout"])
def test_planted_mistakes_are_caught(mutant, monkeypatch):
    if mutant == "gqa":
        monkeypatch.setattr(opa, "attend", _gqa_mod)
    elif mutant == "top_left":
        monkeypatch.setattr(opa, "attend", _top_left)
    else:
        monkeypatch.setattr(opa, "gather_kv", _v_row_major)
    b = make_batch_from_lens([40, 300], [40, 45], dtype="f32", num_q_heads=4,
                             num_kv_heads=2, head_dim=32, block_size=16, seed=3,
                             keep_contig=True)
    got = _run(b)
    assert not np.max(np.abs(got - _sdpa(b))) <= 1e-12     # the brute-force pin fails


# ---- the pass/fail rule: negative controls must fail -----------------------

def test_tolerance_negative_controls():
    b = make_batch_from_lens([600, 900, 1200], [1, 1, 1], dtype="bf16", num_q_heads=8,
                             num_kv_heads=2, head_dim=128, block_size=16, seed=80)
    ref = _run(b)
    assert compare(ref, ref, "bf16")["pass"]
    assert not compare(np.zeros_like(ref), ref, "bf16")["pass"]          # zeros
    assert not compare(ref[:, ::-1], ref, "bf16")["pass"]                # shuffled heads
    for variant in ("one_block_swapped_in", "all_blocks_plus_one"):
        bt = b.block_table.copy()
        if variant == "one_block_swapped_in":
            bt[0, 3] = bt[1, 3]                    # one block of another sequence
        else:
            n0 = -(-int(b.seq_lens[0]) // 16)
            bt[0, :n0] = (bt[0, :n0] + 1) % b.num_blocks     # address off by one block
        wrong = oracle.paged_attention(b.q_raw(), b.kv_raw(), bt, b.seq_lens,
                                       b.cu_seqlens_q, dtype="bf16", num_q_heads=8,
                                       num_kv_heads=2, head_dim=128, block_size=16,
                                       scale=b.scale)
        assert not compare(wrong, ref, "bf16")["pass"], variant


def test_per_sequence_gate_catches_what_the_whole_output_hides():
    """A 1-token sequence (output exactly v0, of unit size) next to a long one
    (output of size about 1/sqrt(L)): a 5% error in the long sequence's output,
    as a wrong normalisation would give, passes the gate over the whole output
    and fails it per sequence."""
    from tests.gpu_helpers import assert_parity
    lens = [1, 2000]
    b = make_batch_from_lens(lens, [1] * len(lens), dtype="bf16", num_q_heads=8,
                             num_kv_heads=2, head_dim=128, block_size=16, seed=81)
    ref = oracle.paged_decode(b.q_raw(), b.kv_raw(), b.block_table, b.seq_lens, dtype="bf16",
                              num_q_heads=8, num_kv_heads=2, head_dim=128, block_size=16,
                              scale=b.scale)
    wrong = ref.copy()
    wrong[1] *= 1.05
    assert compare(wrong, ref, "bf16")["pass"]            # hidden by the short row
    assert not compare(wrong[1:], ref[1:], "bf16")["pass"]
    bounds = np.arange(len(lens) + 1)
    with pytest.raises(AssertionError):
        assert_parity(wrong, ref, "bf16", "negative control", bounds)
    assert_parity(ref, ref, "bf16", "positive control", bounds)
