"""The elastic per-layer pool: lifecycle, kernels over base + elastic ids,
bit-identical results across a decommit/recommit cycle, commit failure under
memory pressure, and decommit with work still in flight."""
import numpy as np
import pytest
import torch

import paper_2608_23658_amd.kvattn as K
from workloads import make_batch_from_lens
from tests.gpu_helpers import seq_bounds, Dev, assert_parity, oracle_decode, require_gpu, say

pytestmark = pytest.mark.gpu

BLOCK = 2 * 8 * 16 * 128 * 2      # one block at 8 kv heads of 128, bf16: 64 KiB


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _elastic_batch(base_blocks, elastic_blocks, lens, seed, frac=0.3):
    """A batch whose tables mix base and elastic block ids (>= frac elastic)."""
    nb = base_blocks + elastic_blocks
    need = sum(-(-L // 16) for L in lens)
    n_el = min(elastic_blocks, max(1, int(np.ceil(frac * need))))
    rng = np.random.default_rng(seed)
    el = rng.choice(np.arange(base_blocks, nb), n_el, replace=False)
    ba = rng.choice(np.arange(base_blocks), need - n_el, replace=False)
    used = rng.permutation(np.concatenate([el, ba]))
    rest = np.setdiff1d(np.arange(nb), used)
    perm = np.concatenate([used, rest]).astype(np.int32)
    b = make_batch_from_lens(lens, [1] * len(lens), dtype="bf16", num_q_heads=32,
                             num_kv_heads=8, head_dim=128, block_size=16, seed=seed,
                             num_blocks=nb, block_perm=perm)
    ids = np.concatenate([b.block_table[s, :-(-L // 16)] for s, L in enumerate(lens)])
    assert (ids >= base_blocks).mean() >= 0.15 and ids.max() >= base_blocks
    return b


def test_granularity_and_lifecycle():
    g = K.ElasticPool.granularity()
    say("pool granularity", g)
    assert g > 0 and (2 << 20) % g == 0 or g % (2 << 20) == 0
    gran = max(g, 2 << 20)
    pool = K.ElasticPool(3, 4 * gran, 2 * gran)
    try:
        ptrs = [pool.layer_ptr(l) for l in range(3)]
        assert len(set(ptrs)) == 3
        assert not pool.is_committed
        assert pool.decommit() >= 0           # no-op
        ms = pool.commit()
        assert pool.is_committed and ms > 0
        assert pool.commit() >= 0             # no-op
        assert [pool.layer_ptr(l) for l in range(3)] == ptrs
        v = pool.layer_view(1)
        v.fill_(7)
        torch.cuda.synchronize()
        assert int(v[-1]) == 7 and int(v[0]) == 7
        pool.decommit()
        assert not pool.is_committed
        assert [pool.layer_ptr(l) for l in range(3)] == ptrs
        base = pool.layer_view(1, committed_part=False)
        assert int(base[0]) == 7              # base contents survive a toggle
        bd = pool.last_breakdown()
        assert set(bd) == {"create_ms", "map_ms", "access_ms", "sync_ms", "unmap_ms"}
    finally:
        pool.close()


def test_decode_over_base_and_elastic_ids_and_bit_identical_toggle():
    gran = max(K.ElasticPool.granularity(), 2 << 20)
    base_blocks, el_blocks = 256, 128            # 16 MiB base, 8 MiB elastic per layer
    assert (base_blocks * BLOCK) % gran == 0 and (el_blocks * BLOCK) % gran == 0
    lens = [100, 700, 1, 1025, 2000, 333]
    b = _elastic_batch(base_blocks, el_blocks, lens, seed=41)
    pool = K.ElasticPool(2, base_blocks * BLOCK, el_blocks * BLOCK)
    try:
        pool.commit()
        layer = pool.layer_view(1, dtype=torch.bfloat16)
        layer.copy_(b.kv_layer.cuda())
        d = Dev(b, kv=pool.layer_ptr(1))
        say("pool decode committed")
        out1 = d.decode().clone()
        torch.cuda.synchronize()
        assert_parity(out1, oracle_decode(b), "bf16", "pool decode, base + elastic ids",
                      seq_bounds(b, decode=True))
        say("pool decommit / recommit")
        pool.decommit()
        pool.commit()
        # elastic contents are undefined after recommit: refill them
        layer = pool.layer_view(1, dtype=torch.bfloat16)
        n_base = base_blocks * BLOCK // 2
        layer[n_base:].copy_(b.kv_layer[n_base:].cuda())
        out2 = d.decode()
        torch.cuda.synchronize()
        assert torch.equal(out1.view(torch.int16), out2.view(torch.int16))
    finally:
        pool.close()


def test_commit_failure_rolls_back():
    """When the second layer's elastic handle cannot be created the commit
    fails with KV_ERR_OOM, keeps nothing and leaves base contents intact."""
    gran = max(K.ElasticPool.granularity(), 2 << 20)
    torch.cuda.empty_cache()
    free, _ = torch.cuda.mem_get_info()
    per_layer = (int(free * 0.6) // gran) * gran
    pool = K.ElasticPool(2, gran, per_layer)
    try:
        base = pool.layer_view(0, committed_part=False)
        base.fill_(42)
        torch.cuda.synchronize()
        say("pool commit expecting OOM", per_layer)
        with pytest.raises(K.KvAttnError) as e:
            pool.commit()
        assert e.value.code == K.KV_ERR_OOM
        assert not pool.is_committed
        free_after, _ = torch.cuda.mem_get_info()
        assert free_after > free - 4 * gran - (64 << 20)
        assert int(base[0]) == 42 and int(base[-1]) == 42
    finally:
        pool.close()


def test_decommit_waits_for_work_in_flight():
    gran = max(K.ElasticPool.granularity(), 2 << 20)
    base_blocks, el_blocks = 8192, 2048
    lens = [4000] * 40
    b = _elastic_batch(base_blocks, el_blocks, lens, seed=43, frac=0.2)
    pool = K.ElasticPool(1, base_blocks * BLOCK, el_blocks * BLOCK)
    try:
        pool.commit()
        pool.layer_view(0, dtype=torch.bfloat16).copy_(b.kv_layer.cuda())
        d = Dev(b, kv=pool.layer_ptr(0))
        ref = d.decode().clone()
        torch.cuda.synchronize()
        say("pool decode then immediate decommit")
        outs = [d.decode() for _ in range(20)]       # enqueued, not waited for
        pool.decommit()                               # must drain before unmapping
        for o in outs:
            assert torch.equal(o.view(torch.int16), ref.view(torch.int16))
    finally:
        pool.close()


def test_whole_handle_commit_decodes_and_keeps_base_bit_for_bit():
    """The naive toggle: one whole handle per layer over base + elastic with
    the base contents copied in. The layer pointer does not move, base bytes
    survive it and its decommit, a decode over base and elastic ids matches
    the oracle, and it refuses to run over a two-handle commit."""
    base_blocks, el_blocks = 256, 128
    lens = [90, 1500, 1, 640, 2048]
    b = _elastic_batch(base_blocks, el_blocks, lens, seed=47)
    n_base = base_blocks * BLOCK // 2                   # bf16 elements of the base part
    pool = K.ElasticPool(2, base_blocks * BLOCK, el_blocks * BLOCK)
    try:
        ptrs = [pool.layer_ptr(l) for l in range(2)]
        kv = b.kv_layer.cuda()
        for l in range(2):
            pool.layer_view(l, committed_part=False, dtype=torch.bfloat16).copy_(kv[:n_base])
        torch.cuda.synchronize()
        say("pool whole-handle commit")
        ms = pool.commit_whole()
        steps = pool.last_steps()
        say("whole-handle commit ms", round(ms, 3),
            {k: round(v, 3) for k, v in steps.items() if k.startswith("commit")})
        assert pool.is_committed and ms > 0 and steps["commit_copy_ms"] > 0
        assert [pool.layer_ptr(l) for l in range(2)] == ptrs
        for l in range(2):
            layer = pool.layer_view(l, dtype=torch.bfloat16)
            assert torch.equal(layer[:n_base].view(torch.int16), kv[:n_base].view(torch.int16))
            layer[n_base:].copy_(kv[n_base:])
        d = Dev(b, kv=pool.layer_ptr(1))
        out = d.decode()
        torch.cuda.synchronize()
        assert_parity(out, oracle_decode(b), "bf16", "decode over whole-handle layers",
                      seq_bounds(b, decode=True))
        assert pool.commit_whole() >= 0                 # no-op while committed this way
        assert pool.commit() >= 0                       # so is the two-handle commit
        say("pool whole-handle decommit")
        pool.decommit()
        steps = pool.last_steps()
        assert not pool.is_committed and steps["decommit_copy_ms"] > 0
        assert [pool.layer_ptr(l) for l in range(2)] == ptrs
        for l in range(2):
            base = pool.layer_view(l, committed_part=False, dtype=torch.bfloat16)
            assert torch.equal(base.view(torch.int16), kv[:n_base].view(torch.int16))
        pool.commit()                                   # the two-handle path still works
        with pytest.raises(K.KvAttnError) as e:
            pool.commit_whole()
        assert e.value.code == K.KV_ERR_STATE
        pool.decommit()
        base = pool.layer_view(0, committed_part=False, dtype=torch.bfloat16)
        assert torch.equal(base.view(torch.int16), kv[:n_base].view(torch.int16))
    finally:
        pool.close()
