"""Host logic of the elastic gate and the toggle controller (no device):
the block pool hands out elastic ids only while admitted, base ids first;
failures change nothing; the drain plan moves every live elastic id to a
free base id; the controller commits after `hysteresis` decode-only steps,
decommits before a prefill, and refuses to decommit while elastic blocks are
live. A randomized scheduler checks the gate invariant over many steps."""
import numpy as np
import pytest

import paper_2608_23658_amd.kvattn as K

KVCTL_NONE, KVCTL_COMMIT, KVCTL_DECOMMIT = K.KVCTL_NONE, K.KVCTL_COMMIT, K.KVCTL_DECOMMIT


def test_gate_hands_out_elastic_ids_only_while_admitted():
    bp = K.BlockPool(4, 3)
    assert not bp.admitted and bp.num_admitted == 4 and bp.num_free == 4
    assert bp.alloc(4).tolist() == [0, 1, 2, 3]          # lowest base ids first
    with pytest.raises(K.KvAttnError) as e:
        bp.alloc(1)
    assert e.value.code == K.KV_ERR_OOM
    bp.set_elastic(True)
    assert bp.num_admitted == 7 and bp.num_free == 3
    assert bp.alloc(2).tolist() == [4, 5]
    assert bp.live_elastic == 2
    bp.free([1])
    assert bp.alloc(2).tolist() == [1, 6]                # base before elastic
    bp.set_elastic(False)
    assert bp.num_free == 0 and bp.live_elastic == 3


def test_failures_change_nothing():
    bp = K.BlockPool(3, 2)
    ids = bp.alloc(2)
    for bad in ([7], [2], [ids[0], ids[0]], [-1]):
        with pytest.raises(K.KvAttnError) as e:
            bp.free(bad)
        assert e.value.code == K.KV_ERR_INVALID
    assert bp.num_free == 1
    with pytest.raises(K.KvAttnError):
        bp.alloc(2)                                      # only 1 free, none taken
    assert bp.num_free == 1
    bp.free(ids)
    assert bp.num_free == 3


def test_drain_plan_moves_live_elastic_ids_to_free_base_ids():
    bp = K.BlockPool(6, 4)
    bp.set_elastic(True)
    base = bp.alloc(6)
    el = bp.alloc(3)
    assert el.tolist() == [6, 7, 8]
    bp.free(base[:2])                                    # 3 live elastic, 2 free base
    with pytest.raises(K.KvAttnError) as e:
        bp.plan_drain()
    assert e.value.code == K.KV_ERR_OOM
    assert bp.num_free == 3 and bp.live_elastic == 3     # nothing allocated
    bp.free(base[3:4])
    f, t = bp.plan_drain()
    assert f.tolist() == [6, 7, 8] and sorted(t.tolist()) == sorted([0, 1, 3])
    assert bp.live_elastic == 3 and bp.num_free == 1     # destinations are now allocated
    bp.free(f)
    assert bp.live_elastic == 0


def test_controller_hysteresis_and_prefill_boundary():
    bp = K.BlockPool(8, 4)
    ctl = K.Controller(None, bp, hysteresis=3)
    assert not ctl.committed and not bp.admitted
    acts = [ctl.before_step(p)[0] for p in (False, False, True, False, False, False, False)]
    assert acts == [KVCTL_NONE, KVCTL_NONE, KVCTL_NONE, KVCTL_NONE, KVCTL_NONE, KVCTL_COMMIT,
                    KVCTL_NONE]
    assert ctl.committed and bp.admitted and bp.num_admitted == 12
    assert ctl.before_step(True)[0] == KVCTL_DECOMMIT
    assert not bp.admitted and ctl.counts() == (1, 1)
    assert ctl.before_step(True)[0] == KVCTL_NONE        # already decommitted


def test_controller_refuses_to_decommit_over_live_elastic_blocks():
    bp = K.BlockPool(2, 2)
    ctl = K.Controller(None, bp, hysteresis=1)
    assert ctl.before_step(False)[0] == KVCTL_COMMIT
    ids = bp.alloc(3)
    with pytest.raises(K.KvAttnError) as e:
        ctl.before_step(True)
    assert e.value.code == K.KV_ERR_STATE
    assert ctl.committed and bp.admitted                 # nothing changed
    bp.free(ids[2:])
    assert ctl.before_step(True)[0] == KVCTL_DECOMMIT


def test_would_commit_predicts_the_next_call():
    bp = K.BlockPool(2, 2)
    ctl = K.Controller(None, bp, hysteresis=2)
    for p in (False, False, True, False, False, False):
        predicted = K.lib().kvctl_would_commit(ctl._h, int(p)) == 1
        act, _ = ctl.before_step(p)
        assert predicted == (act == KVCTL_COMMIT)


def test_randomized_scheduler_keeps_the_gate():
    """Sequences grow and finish; steps are decode-only or carry a prefill;
    before each prefill the scheduler drains by migration. At every point no
    elastic id is live while the range is withdrawn."""
    rng = np.random.default_rng(7)
    nb, ne = 64, 32
    bp = K.BlockPool(nb, ne)
    ctl = K.Controller(None, bp, hysteresis=4)
    seqs = {}
    nxt = 0
    for step in range(2000):
        prefill = rng.random() < 0.08
        try:
            act, _ = ctl.before_step(prefill)
        except K.KvAttnError as e:
            assert e.code == K.KV_ERR_STATE and prefill
            # migrate what fits into free base ids; preempt the rest
            while True:
                try:
                    f, t = bp.plan_drain()
                    break
                except K.KvAttnError as e2:
                    assert e2.code == K.KV_ERR_OOM
                    victim = next(s for s, v in seqs.items() if any(b >= nb for b in v))
                    bp.free(seqs.pop(victim))
            remap = dict(zip(f.tolist(), t.tolist()))
            for s in seqs:
                seqs[s] = [remap.get(b, b) for b in seqs[s]]
            bp.free(f)
            act, _ = ctl.before_step(prefill)
            assert act == KVCTL_DECOMMIT
        if not bp.admitted:
            assert bp.live_elastic == 0
        live = [b for v in seqs.values() for b in v]
        assert len(live) == len(set(live))
        assert all(b < bp.num_admitted for b in live)
        # the step: new sequences (prefill), growth, finishes
        if prefill:
            try:
                seqs[nxt] = bp.alloc(int(rng.integers(1, 6))).tolist()
                nxt += 1
            except K.KvAttnError:
                pass
        for s in list(seqs):
            if rng.random() < 0.3:
                try:
                    seqs[s] += bp.alloc(1).tolist()
                except K.KvAttnError:
                    pass
            if rng.random() < 0.05:
                bp.free(seqs.pop(s))
    c, d = ctl.counts()
    assert c >= 10 and d >= 10
