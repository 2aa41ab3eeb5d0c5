"""The rate probes do the work they are timed for: the read probe reads
exactly the K/V tiles of the blocks a decode batch holds (its per-lane word
sums match a host computation over the same bytes), and the matrix probe
multiplies the operands it states (its sums match the closed form
sum(A B) = sum_k colsum(A)[k] rowsum(B)[k])."""
import numpy as np
import pytest
import torch

import paper_2608_23658_amd.kvattn as K
from workloads import make_batch_from_lens
from tests.gpu_helpers import require_gpu, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def test_read_probe_reads_every_tile_of_the_batch():
    # lengths across block and 1024-token split edges, an empty sequence, and
    # one table entry out of range (skipped, like the decode kernel does)
    lens = [0, 1, 15, 16, 17, 1023, 1024, 1025, 2600, 333]
    b = make_batch_from_lens(lens, [min(1, L) for L in lens], dtype="bf16", num_q_heads=32,
                             num_kv_heads=8, head_dim=128, block_size=16, seed=5)
    bt_np = b.block_table.copy()
    bt_np[8, 7] = b.num_blocks + 3
    kv = b.kv_layer.cuda()
    bt = torch.from_numpy(bt_np).cuda()
    sl = torch.from_numpy(b.seq_lens).cuda()
    say("read probe", lens)
    out = K.probe_read_blocks(kv, b.num_blocks, bt, sl, num_kv_heads=8, head_dim=128,
                              dtype=torch.bfloat16, max_seq_len=b.max_seq_len)
    torch.cuda.synchronize()
    got = out.cpu().numpy().view(np.uint32).astype(np.int64)

    # lane l of a wavefront reads words [256 c + 4 l, 256 c + 4 l + 4) of each
    # 4 KiB tile: per (block, K/V, head, lane) sums over c and the 4 words
    words = b.kv_layer.contiguous().view(torch.int32).numpy().view(np.uint32).astype(np.int64)
    tiles = words.reshape(b.num_blocks, 2, 8, 4, 64, 4).sum(axis=(3, 5))   # [blk, kv, g, lane]
    nsplit = -(-b.max_seq_len // 1024)
    B = len(lens)
    want = np.zeros((nsplit, B, 8, 64), dtype=np.int64)
    for s, L in enumerate(lens):
        for sp in range(nsplit):
            t0, t1 = 1024 * sp, min(L, 1024 * (sp + 1))
            for blk in range(t0 // 16, -(-t1 // 16)):
                if t0 >= L:
                    break
                i = int(bt_np[s, blk])
                if 0 <= i < b.num_blocks:
                    want[sp, s] += tiles[i, 0] + tiles[i, 1]
    want %= 1 << 32
    assert got.shape == (nsplit * B * 8 * 64,)
    assert np.array_equal(got.reshape(nsplit, B, 8, 64), want)


def _probe_operands(gid):
    """bf16 A and B fragments [4][8] of the thread with global index gid, as
    the probe draws them (returned as float64 of the rounded bf16 values)."""
    h = (gid * 2654435761) & 0xffffffff
    a = np.zeros((4, 8), dtype=np.float32)
    b = np.zeros((4, 8), dtype=np.float32)
    for j in range(4):
        for i in range(8):
            h = (h * 1664525 + 1013904223) & 0xffffffff
            a[j, i] = ((h >> 8) & 0xffff) / 32768.0 - 1.0
            h = (h * 1664525 + 1013904223) & 0xffffffff
            b[j, i] = ((h >> 8) & 0xffff) / 32768.0 - 1.0
    rnd = lambda x: torch.from_numpy(x).to(torch.bfloat16).double().numpy()
    return rnd(a), rnd(b)


def test_matrix_probe_multiplies_its_operands():
    wg, iters = 3, 5
    threads = K.lib().kvattn_probe_mfma_threads()
    say("matrix probe", wg, iters)
    clocks = torch.zeros(wg * 8 * 4, dtype=torch.int64, device="cuda")
    out = K.probe_mfma(wg, iters, clocks=clocks)
    torch.cuda.synchronize()
    # every wavefront recorded increasing counters, and a clock in a sane range
    c = clocks.view(-1, 4).cpu()
    assert bool((c[:, 1] > c[:, 0]).all()) and bool((c[:, 3] >= c[:, 2]).all())
    ck = K.probe_mfma_clock(clocks, iters)
    assert 0.3 < ck["clock_ghz_realtime_median"] < 3.0, ck
    assert 0.0 < ck["matrix_busy_median"] <= 1.05, ck
    got = out.double().cpu().numpy().reshape(wg, threads // 64, 64)
    for w in range(wg):
        for v in range(threads // 64):
            ops = [_probe_operands(w * threads + v * 64 + l) for l in range(64)]
            A = np.stack([o[0] for o in ops])   # [lane, frag, 8]
            Bm = np.stack([o[1] for o in ops])
            # A fragment: lane l holds row l % 32, k = 8 (l // 32) + i;
            # B fragment: lane l holds column l % 32, k = 8 (l // 32) + i
            colA = np.stack([A[:32].sum(0), A[32:].sum(0)], 1).reshape(4, 16)   # [frag, k]
            rowB = np.stack([Bm[:32].sum(0), Bm[32:].sum(0)], 1).reshape(4, 16)
            total = iters * sum(colA[m % 4] @ rowB[(m + m // 4) % 4] for m in range(8))
            absA = np.stack([np.abs(A[:32]).sum(0), np.abs(A[32:]).sum(0)], 1).reshape(4, 16)
            absB = np.stack([np.abs(Bm[:32]).sum(0), np.abs(Bm[32:]).sum(0)], 1).reshape(4, 16)
            bound = iters * sum(absA[m % 4] @ absB[(m + m // 4) % 4] for m in range(8))
            assert abs(got[w, v].sum() - total) <= 1e-5 * bound, (w, v, got[w, v].sum(), total)
