"""The toggle controller on a real elastic pool, end to end: block copies are
byte-exact against the CPU oracle; the controller commits after decode-only
steps, refuses to decommit while elastic blocks are live, and decommits once
they are drained by migration; a decode captured in a HIP graph while
committed is replayed after the drain and decommit (its table now holds base
ids only) and after the recommit (new elastic blocks refilled), matching the
eager result bit for bit each time, with results also checked against the
oracle."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_23658_amd.kvattn as K
from tests.gpu_helpers import assert_parity, require_gpu, say

pytestmark = pytest.mark.gpu

BLOCK = 2 * 8 * 16 * 128 * 2      # one block at 8 kv heads of 128, bf16: 64 KiB
HKV, D = 8, 128


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _np_u8(t):
    return t.cpu().numpy()


def test_copy_blocks_bitwise_vs_oracle():
    nb, nl = 16, 3
    g = torch.Generator().manual_seed(3)
    layers = [torch.randint(0, 256, (nb * BLOCK,), generator=g, dtype=torch.uint8).cuda()
              for _ in range(nl)]
    before = [_np_u8(t) for t in layers]
    src = np.array([3, 12, 5, 20, -1, 9], dtype=np.int32)
    dst = np.array([7, 0, 5, 1, 2, 15], dtype=np.int32)
    say("copy_blocks", src.tolist(), dst.tolist())
    K.copy_blocks([t.data_ptr() for t in layers], nb, BLOCK, torch.from_numpy(src).cuda(),
                  torch.from_numpy(dst).cuda())
    torch.cuda.synchronize()
    for l in range(nl):
        ref = oracle.copy_blocks(before[l], src, dst, num_blocks=nb)
        assert np.array_equal(_np_u8(layers[l]), ref)


class _Engine:
    """A minimal engine over two layers: sequences own block ids from the
    gated pool; their K/V rows are written with kv_append."""

    def __init__(self, pool, bp, nb_total, rng):
        self.pool, self.bp, self.nb, self.rng = pool, bp, nb_total, rng

    def fill(self, ids, L, seed):
        g = torch.Generator().manual_seed(seed)
        t = np.arange(L)
        slots = torch.from_numpy((ids[t // 16].astype(np.int64) * 16 + t % 16).astype(np.int32))
        for layer in range(self.pool.num_layers):
            k = torch.randn(L, HKV, D, generator=g).to(torch.bfloat16).cuda()
            v = torch.randn(L, HKV, D, generator=g).to(torch.bfloat16).cuda()
            K.kv_append(k, v, slots.cuda(), self.pool.layer_ptr(layer), self.nb)

    def oracle_decode(self, q, bt, sl):
        raw = _np_u8(self.pool.layer_view(0)).view(np.uint16)
        qraw = q.cpu().view(torch.int16).numpy().view(np.uint16)
        return oracle.paged_decode(qraw, raw, bt, sl, dtype="bf16", num_q_heads=32,
                                   num_kv_heads=HKV, head_dim=D, block_size=16,
                                   scale=1.0 / np.sqrt(D))


def test_controller_drain_decommit_and_graph_replay_across_toggles():
    nb_base, nb_el = 64, 32
    nb = nb_base + nb_el
    gran = max(K.ElasticPool.granularity(), 2 << 20)
    assert (nb_base * BLOCK) % gran == 0 and (nb_el * BLOCK) % gran == 0
    say("controller pool", nb_base, nb_el)
    pool = K.ElasticPool(2, nb_base * BLOCK, nb_el * BLOCK)
    bp = K.BlockPool(nb_base, nb_el)
    ctl = K.Controller(pool, bp, hysteresis=2)
    eng = _Engine(pool, bp, nb, np.random.default_rng(0))
    try:
        assert ctl.before_step(False)[0] == K.KVCTL_NONE
        act, ms = ctl.before_step(False)
        assert act == K.KVCTL_COMMIT and pool.is_committed and bp.admitted
        say("committed in", round(ms, 3), "ms")
        # five sequences of 240 tokens (15 blocks each): 64 base + 11 elastic blocks
        L, B, maxb = 240, 5, 15
        tables = [bp.alloc(maxb) for _ in range(B)]
        assert bp.live_elastic == 11
        for s in range(B):
            eng.fill(tables[s], L, 100 + s)
        bt_np = np.stack(tables).astype(np.int32)
        sl_np = np.full(B, L, dtype=np.int32)
        q_s = torch.randn(B, 32, D, generator=torch.Generator().manual_seed(9)).to(
            torch.bfloat16).cuda()
        bt_s = torch.from_numpy(bt_np).cuda()
        sl_s = torch.from_numpy(sl_np).cuda()
        out_s = torch.empty_like(q_s)
        ws_s = K.workspace(K.decode_workspace_bytes(B, 32, D, L))

        def run():
            K.decode(q_s, pool.layer_ptr(0), nb, bt_s, sl_s, num_kv_heads=HKV, max_seq_len=L,
                     out=out_s, ws=ws_s)

        run()
        eager = out_s.clone()
        torch.cuda.synchronize()
        assert_parity(eager, eng.oracle_decode(q_s, bt_np, sl_np), "bf16", "committed decode")
        # capture the decode while committed
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            run()
        torch.cuda.current_stream().wait_stream(side)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            run()
        for r in range(3):
            out_s.fill_(0)
            torch.cuda.synchronize()
            graph.replay()
            torch.cuda.synchronize()
            assert torch.equal(out_s.view(torch.int16), eager.view(torch.int16)), r
        # a prefill is next: refused while elastic blocks are live
        with pytest.raises(K.KvAttnError) as e:
            ctl.before_step(True)
        assert e.value.code == K.KV_ERR_STATE and pool.is_committed
        # sequence 0 finishes; drain the elastic blocks of the others by migration
        bp.free(tables[0])
        sl_s[0] = 0
        f, t = bp.plan_drain()
        assert len(f) == 11 and (f >= nb_base).all() and (t < nb_base).all()
        K.copy_blocks([pool.layer_ptr(0), pool.layer_ptr(1)], nb, BLOCK,
                      torch.from_numpy(f).cuda(), torch.from_numpy(t).cuda())
        remap = dict(zip(f.tolist(), t.tolist()))
        bt_np = np.vectorize(lambda x: remap.get(int(x), int(x)))(bt_np).astype(np.int32)
        bt_np[0] = -1
        bt_s.copy_(torch.from_numpy(bt_np))
        bp.free(f)
        sl_np[0] = 0
        run()
        after_drain = out_s.clone()
        torch.cuda.synchronize()
        # migration moved bytes, not values: the other sequences are unchanged
        assert torch.equal(after_drain[1:].view(torch.int16), eager[1:].view(torch.int16))
        assert not after_drain[0].float().abs().any()
        act, ms = ctl.before_step(True)
        assert act == K.KVCTL_DECOMMIT and not pool.is_committed and not bp.admitted
        say("decommitted in", round(ms, 3), "ms")
        assert (bt_np < nb_base).all()
        for r in range(3):
            out_s.fill_(1)
            torch.cuda.synchronize()
            graph.replay()
            torch.cuda.synchronize()
            assert torch.equal(out_s.view(torch.int16), after_drain.view(torch.int16)), r
        # decode-only again: recommit, a new sequence takes the elastic blocks
        assert ctl.before_step(False)[0] == K.KVCTL_NONE
        act, ms = ctl.before_step(False)
        assert act == K.KVCTL_COMMIT and pool.is_committed
        say("recommitted in", round(ms, 3), "ms")
        new = bp.alloc(maxb)
        assert (new >= nb_base).sum() == 11
        eng.fill(new, L, 555)
        bt_np[0] = new
        sl_np[0] = L
        bt_s.copy_(torch.from_numpy(bt_np))
        sl_s.copy_(torch.from_numpy(sl_np))
        run()
        eager2 = out_s.clone()
        torch.cuda.synchronize()
        assert torch.equal(eager2[1:].view(torch.int16), eager[1:].view(torch.int16))
        for r in range(3):
            out_s.fill_(0)
            torch.cuda.synchronize()
            graph.replay()
            torch.cuda.synchronize()
            assert torch.equal(out_s.view(torch.int16), eager2.view(torch.int16)), r
        assert_parity(eager2, eng.oracle_decode(q_s, bt_np, sl_np), "bf16", "after recommit")
        assert ctl.counts() == (2, 1)
        del graph
    finally:
        ctl.close()
        pool.close()
