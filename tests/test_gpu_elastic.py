"""Elastic-pool decode at full size: 32 layers of 6 GiB (96 MiB elastic each),
512 sequences U[8192, 32768] over one shared table with 15% elastic
references. Sampled outputs against the oracle (the referenced blocks are
copied to the host), one kernel call spanning base and elastic ids, and
bit-identical results across a decommit / recommit cycle."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2608_23658_amd.kvattn as K
from workloads.configs import ELASTIC as E
from workloads.elastic import elastic_queries, elastic_tables, fill_layer, remap_elastic_to_base
from tests.gpu_helpers import assert_parity, f64, require_gpu, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _oracle_row(view_u8, bt_row, L, q_row):
    """The oracle on the blocks one sequence references, copied to the host."""
    bb = E.block_bytes
    nblk = math.ceil(L / E.block_size)
    ids = bt_row[:nblk]
    uniq, inv = np.unique(ids, return_inverse=True)
    idx = torch.from_numpy(uniq.astype(np.int64)).cuda()
    blocks = view_u8.view(-1, bb).index_select(0, idx).cpu()
    raw = blocks.numpy().view(np.uint16).reshape(-1)
    table = inv.astype(np.int32)[None]
    qraw = q_row.view(torch.int16).numpy().view(np.uint16)[None]
    return oracle.paged_decode(qraw, raw, table, np.array([L], np.int32), dtype="bf16",
                               num_q_heads=E.num_q_heads, num_kv_heads=E.num_kv_heads,
                               head_dim=E.head_dim, block_size=E.block_size, scale=E.scale)[0]


def test_elastic_decode_full_size():
    torch.cuda.empty_cache()
    bb = E.block_bytes
    base, el = E.base_blocks * bb, E.elastic_bytes_per_layer
    nb_all = E.base_blocks + E.elastic_blocks
    lens, bt_np, el_mask = elastic_tables(E)
    assert el_mask.sum() / (bt_np >= 0).sum() >= 0.15
    bt = torch.from_numpy(bt_np).cuda()
    sl = torch.from_numpy(lens).cuda()
    q_cpu = elastic_queries(E)
    q = q_cpu.cuda()
    msl = int(lens.max())
    ws = K.workspace(K.decode_workspace_bytes(E.batch, 32, 128, msl))
    layers = [0, 15, 31]
    say("elastic pool create", E.num_layers, base, el)
    pool = K.ElasticPool(E.num_layers, base, el)
    try:
        pool.commit()
        for l in layers:
            fill_layer(pool.layer_view(l, dtype=torch.bfloat16), l, base // 2)
        outs = {}
        for l in layers:
            say("elastic decode committed, layer", l)
            outs[l] = K.decode(q, pool.layer_ptr(l), nb_all, bt, sl, num_kv_heads=8,
                               max_seq_len=msl, scale=E.scale, ws=ws)
        torch.cuda.synchronize()
        # the sequences with the most elastic references, the longest and the
        # shortest, and ten drawn at random
        rng = np.random.default_rng(5)
        seqs = sorted(set(np.argsort(-el_mask.sum(1))[:4].tolist()
                          + [int(np.argmax(lens)), int(np.argmin(lens))]
                          + rng.choice(E.batch, 10, replace=False).tolist()))
        for l in layers:
            view = pool.layer_view(l)
            ref = np.stack([_oracle_row(view, bt_np[s], int(lens[s]), q_cpu[s]) for s in seqs])
            assert_parity(f64(outs[l])[seqs], ref, "bf16", f"elastic layer {l} seqs {seqs}")
        # decommit: the same reuse structure on base ids only; ids at or past
        # the base range are out of bounds for the call and never read
        say("elastic decommit")
        pool.decommit()
        bt_base = torch.from_numpy(remap_elastic_to_base(bt_np, E)).cuda()
        o = K.decode(q, pool.layer_ptr(0), E.base_blocks, bt_base, sl, num_kv_heads=8,
                     max_seq_len=msl, scale=E.scale, ws=ws)
        torch.cuda.synchronize()
        assert torch.isfinite(o.float()).all()
        bt_base_np = bt_base.cpu().numpy()
        view = pool.layer_view(0, committed_part=False)
        dseqs = seqs[:6]
        ref = np.stack([_oracle_row(view, bt_base_np[s], int(lens[s]), q_cpu[s]) for s in dseqs])
        assert_parity(f64(o)[dseqs], ref, "bf16", f"elastic layer 0 decommitted, seqs {dseqs}")
        say("elastic recommit and refill")
        pool.commit()
        for l in layers:
            fill_layer(pool.layer_view(l, dtype=torch.bfloat16), l, base // 2, part="elastic")
        for l in layers:
            o = K.decode(q, pool.layer_ptr(l), nb_all, bt, sl, num_kv_heads=8,
                         max_seq_len=msl, scale=E.scale, ws=ws)
            torch.cuda.synchronize()
            assert torch.equal(o.view(torch.int16), outs[l].view(torch.int16)), l
    finally:
        pool.close()
