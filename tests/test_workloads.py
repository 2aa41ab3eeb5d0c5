"""The seeded generator: documented layout, poison, determinism, config shapes."""
import numpy as np
import torch

from workloads import (DECODE_B256, MIXED_STEP, PREFILL_L32768, TINY_DECODE_F32, layout_offsets,
                       make_batch, make_batch_from_lens)
from workloads.configs import ELASTIC, pool_blocks_rule


def _check_layout(b):
    raw = b.kv_layer.to(torch.float64).numpy()
    written = 0
    for s in range(b.num_seqs):
        L = int(b.seq_lens[s])
        if L == 0:
            continue
        t = np.arange(L)
        blocks = b.block_table[s, t // b.block_size]
        slots = t % b.block_size
        k = b.k_contig[s].to(torch.float64).numpy()
        v = b.v_contig[s].to(torch.float64).numpy()
        for g in range(b.num_kv_heads):
            for j in range(b.head_dim):
                ko = layout_offsets(0, blocks, g, slots, j, b.num_kv_heads, b.block_size,
                                    b.head_dim, b.esz)
                vo = layout_offsets(1, blocks, g, slots, j, b.num_kv_heads, b.block_size,
                                    b.head_dim, b.esz)
                assert np.array_equal(raw[ko], k[:, g, j])
                assert np.array_equal(raw[vo], v[:, g, j])
        written += 2 * L * b.num_kv_heads * b.head_dim
    # every other element is NaN poison
    assert int(np.isfinite(raw).sum()) == written


def test_layout_matches_documented_offsets_f32_and_bf16():
    for dtype in ("f32", "bf16"):
        b = make_batch_from_lens([37, 16, 5], [1, 16, 5], dtype=dtype, num_q_heads=4,
                                 num_kv_heads=2, head_dim=32, block_size=16, seed=2,
                                 keep_contig=True)
        _check_layout(b)


def test_same_seed_same_bytes_and_seed_matters():
    a = make_batch(TINY_DECODE_F32)
    b = make_batch(TINY_DECODE_F32)
    assert np.array_equal(a.kv_raw().view(np.uint32), b.kv_raw().view(np.uint32))
    assert np.array_equal(a.q_raw(), b.q_raw()) and np.array_equal(a.block_table, b.block_table)
    c = make_batch_from_lens([37, 64, 101, 130], [1] * 4, dtype="f32", num_q_heads=4,
                             num_kv_heads=2, head_dim=64, block_size=16, seed=7, num_blocks=64)
    assert not np.array_equal(a.q_raw(), c.q_raw())


def test_tiny_decode_shapes():
    b = make_batch(TINY_DECODE_F32)
    assert b.seq_lens.tolist() == [37, 64, 101, 130]
    nblk = [-(-int(L) // 16) for L in b.seq_lens]
    assert sum(nblk) == 23 and b.num_blocks == 64
    ids = np.concatenate([b.block_table[s, :n] for s, n in enumerate(nblk)])
    assert len(set(ids.tolist())) == 23 and ids.min() >= 0 and ids.max() < 64
    assert (b.block_table[0, 3:] == -1).all()
    assert b.q.shape == (4, 4, 64) and b.q.dtype == torch.float32


def test_config_length_ranges_and_pool_rule():
    g = torch.Generator().manual_seed(DECODE_B256.seed)
    r = torch.randint(512, 4097, (256,), generator=g)
    assert r.min() >= 512 and r.max() <= 4096
    assert pool_blocks_rule(2048) == 2272          # 2048 * 1.1 -> 2253 -> multiple of 32
    assert pool_blocks_rule(32) == 64
    s3 = MIXED_STEP
    assert s3.fixed_prefix == ((32768, 8192),) and s3.rand_count == 128
    assert s3.max_num_batched_tokens == 8192 + 128
    assert PREFILL_L32768.num_blocks == 2272


def test_elastic_sizes():
    # 3 GiB over 32 layers is 96 MiB per layer, 1536 blocks of 64 KiB,
    # a whole number of 2 MiB granules (48).
    assert ELASTIC.block_bytes == 64 * 1024
    assert ELASTIC.elastic_bytes_per_layer == 96 << 20
    assert ELASTIC.elastic_blocks == 1536
    assert ELASTIC.elastic_bytes_per_layer % (2 << 20) == 0
    assert (ELASTIC.base_blocks * ELASTIC.block_bytes) % (2 << 20) == 0
