"""Pins for the K/V append oracle: each checks it against something other than itself.

* the generator's own scatter (a different code path: torch advanced
  indexing on a 5-D view) must come out of the oracle byte for byte;
* gather after append returns the appended rows exactly (the gather is pinned
  by the attention brute force in test_oracle.py);
* padding and out-of-range slots leave the layer untouched;
* planted mistakes in the oracle fail these pins.
"""
import numpy as np
import pytest
import torch

import oracle
import oracle.append as oap
from workloads import make_batch_from_lens
from workloads.append import make_append, next_slots


def _raw(t):
    return t.view(torch.int16).numpy().view(np.uint16) if t.dtype == torch.bfloat16 else t.numpy()


def _all_slots(bt_row, L, bs):
    t = np.arange(L)
    return (bt_row[t // bs].astype(np.int64) * bs + t % bs).astype(np.int32)


@pytest.mark.parametrize("dtype,hkv,d", [("bf16", 2, 128), ("f32", 2, 64), ("bf16", 4, 64)])
def test_append_reproduces_generator_pool(dtype, hkv, d):
    b = make_batch_from_lens([37, 100, 16, 1], [1, 1, 1, 1], dtype=dtype, num_q_heads=hkv,
                             num_kv_heads=hkv, head_dim=d, block_size=16, seed=5,
                             keep_contig=True)
    empty = np.full_like(b.kv_raw(), b.kv_raw().flat[-1])   # the generator's NaN fill
    out = empty
    for s in range(b.num_seqs):
        L = int(b.seq_lens[s])
        slots = _all_slots(b.block_table[s], L, 16)
        out = oracle.kv_append(out, _raw(b.k_contig[s]), _raw(b.v_contig[s]), slots,
                               dtype=dtype, num_kv_heads=hkv, head_dim=d, block_size=16)
    assert np.array_equal(out.view(np.uint8), b.kv_raw().view(np.uint8))


@pytest.mark.parametrize("dtype,d", [("bf16", 128), ("f32", 64)])
def test_gather_after_append_round_trip(dtype, d):
    hkv, bs, nb = 2, 16, 12
    a = make_append(70, num_kv_heads=hkv, head_dim=d, dtype=dtype, num_blocks=nb,
                    block_size=bs, seed=11)
    esz = {"bf16": 2, "f32": 4}[dtype]
    layer = np.zeros(nb * 2 * hkv * bs * d, dtype=np.uint16 if esz == 2 else np.float32)
    out = oracle.kv_append(layer, a.k_raw(), a.v_raw(), a.slot_mapping, dtype=dtype,
                           num_kv_heads=hkv, head_dim=d, block_size=bs)
    # read every token back through a one-block "table" pointing at its block
    for t, slot in enumerate(a.slot_mapping):
        blk, r = divmod(int(slot), bs)
        K, V = oracle.gather_kv(out, dtype, np.array([blk]), bs, hkv, bs, d)
        assert np.array_equal(K[r], oracle.storage_to_f64(a.k_raw()[t], dtype))
        assert np.array_equal(V[r], oracle.storage_to_f64(a.v_raw()[t], dtype))


def test_padding_and_out_of_range_slots_are_skipped():
    hkv, d, bs, nb = 2, 64, 16, 4
    a = make_append(8, num_kv_heads=hkv, head_dim=d, dtype="bf16", num_blocks=nb,
                    block_size=bs, seed=3)
    a.slot_mapping[:] = [-1, nb * bs, nb * bs + 5, -7, -1, 10 ** 6, -1, -2]
    layer = np.arange(nb * 2 * hkv * bs * d, dtype=np.uint16)
    out = oracle.kv_append(layer, a.k_raw(), a.v_raw(), a.slot_mapping, dtype="bf16",
                           num_kv_heads=hkv, head_dim=d, block_size=bs)
    assert np.array_equal(out, layer)


def test_next_slots_follow_the_table():
    bt = np.array([[3, 7, -1], [2, -1, -1]], dtype=np.int32)
    assert next_slots(bt, np.array([17, 16]), 16).tolist() == [7 * 16 + 1, -1]
    assert next_slots(bt, np.array([0, 5]), 16).tolist() == [3 * 16, 2 * 16 + 5]


_ORIG = oap.kv_append


def _swap_kv(kv_raw, k_new, v_new, slot_mapping, **kw):
    return _ORIG(kv_raw, v_new, k_new, slot_mapping, **kw)


def _off_by_one(kv_raw, k_new, v_new, slot_mapping, **kw):
    sm = np.where(slot_mapping >= 0, slot_mapping + 1, slot_mapping)
    return _ORIG(kv_raw, k_new, v_new, sm, **kw)


def _v_slot_major(kv_raw, k_new, v_new, slot_mapping, *, dtype, num_kv_heads, head_dim,
                  block_size):
    out = np.array(kv_raw, copy=True)
    layer = out.reshape(-1).reshape(-1, 2, num_kv_heads, block_size * head_dim)
    vec = 16 // {"bf16": 2, "f32": 4}[dtype]
    j = np.arange(head_dim)
    for t, slot in enumerate(slot_mapping):
        if slot < 0 or slot >= layer.shape[0] * block_size:
            continue
        b, r = divmod(int(slot), block_size)
        for g in range(num_kv_heads):
            layer[b, 0, g, ((j // vec) * block_size + r) * vec + j % vec] = k_new[t, g]
            layer[b, 1, g, r * head_dim + j] = v_new[t, g]      # wrong: slot-major V
    return out


@pytest.mark.parametrize("mutant", [_swap_kv, _off_by_one, _v_slot_major])
def test_planted_mistakes_are_caught(mutant, monkeypatch):
    monkeypatch.setattr(oracle, "kv_append", mutant)
    failed = 0
    for pin in (lambda: test_append_reproduces_generator_pool("bf16", 2, 128),
                lambda: test_gather_after_append_round_trip("bf16", 128)):
        try:
            pin()
        except AssertionError:
            failed += 1
    assert failed >= 1, mutant.__name__


def test_copy_blocks_moves_whole_blocks():
    """After copying, gathering the destination block returns the source
    block's rows (the gather is pinned by the attention brute force), other
    blocks are untouched, and invalid pairs are skipped."""
    hkv, d, bs, nb = 2, 64, 16, 8
    rng = np.random.default_rng(5)
    layer = rng.integers(0, 1 << 16, size=nb * 2 * hkv * bs * d, dtype=np.uint16)
    out = oracle.copy_blocks(layer, [5, 2, 9, 3], [1, 6, 0, 3], num_blocks=nb)
    for s, t in ((5, 1), (2, 6)):
        Ks, Vs = oracle.gather_kv(layer, "bf16", np.array([s]), bs, hkv, bs, d)
        Kt, Vt = oracle.gather_kv(out, "bf16", np.array([t]), bs, hkv, bs, d)
        assert np.array_equal(Ks, Kt, equal_nan=True) and np.array_equal(Vs, Vt, equal_nan=True)
    blk = layer.reshape(nb, -1)
    for b in (0, 2, 3, 4, 5, 7):
        assert np.array_equal(out.reshape(nb, -1)[b], blk[b])
