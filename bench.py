#!/usr/bin/env python3
"""Benchmark of the paged-KV attention hot path on one MI355X.

Headline (one JSON line on stdout): decode of the Llama-3-8B-shaped layer
(256 sequences, lengths U[512, 4096], bf16) as algorithmic KV-read GB/s. A
step is one kvattn_decode call over the whole batch, inputs resident in HBM.
The same line carries the chunked-prefill figures (the last 8192-token chunk
of a 32768-token prompt and the whole 32768-token prompt, TFLOP/s), the
elastic-pool toggle latencies, the roofline of the dominant kernel from
per-kernel HIP events, and the CPU oracle timed on a bounded sample.
"""
from __future__ import annotations

import argparse
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402
import torch  # noqa: E402

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
MFMA_BF16_PEAK_TFLOPS = 2516.6  # 256 CU x 2.4 GHz x 4096 dense bf16 FLOP/clk


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="all",
                    choices=["all", "decode", "prefill", "mixed", "append", "two_tensor",
                             "toggle", "controller", "elastic", "necessity", "copy"],
                    help="'all' = headline decode plus the prefill, mixed-step and toggle "
                         "legs; 'copy' = a plain 2 GiB elementwise copy, the reference that "
                         "scales the HBM byte counters")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="target CPU time of the oracle sample")
    return ap.parse_args()


class Timer:
    """HIP events on the current stream around a region."""

    def __init__(self):
        self.a = torch.cuda.Event(enable_timing=True)
        self.b = torch.cuda.Event(enable_timing=True)

    def __enter__(self):
        torch.cuda.synchronize()
        self.a.record()
        return self

    def __exit__(self, *exc):
        self.b.record()
        torch.cuda.synchronize()
        self.ms = self.a.elapsed_time(self.b)
        return False


def timed(fn, steps, warmup, K, kernel):
    """Run fn warmup + steps + steps times; returns (ms per step, mean ms of
    `kernel` launches from per-kernel events, all per-kernel means, and each
    kernel's p10 / median / p90 over its launches).

    The step time comes from the first `steps` runs, bracketed by
    synchronisation, with nothing else on the stream: the library's
    per-kernel events, recorded between its launches, leave gaps on the GPU
    (about 15 us per decode step). The per-kernel durations come from HIP
    events on the launch stream in a second pass of the same steps right
    after."""
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    with Timer() as t:
        for _ in range(steps):
            fn()
    with K.KernelTrace(4 * steps) as tr:
        for _ in range(steps):
            fn()
    torch.cuda.synchronize()
    per = {}
    for name, ms in tr.durations():
        per.setdefault(name, []).append(ms)
    means = {k: statistics.fmean(v) for k, v in per.items()}
    spread = {k: {"p10": round(float(np.percentile(v, 10)), 6),
                  "median": round(float(np.median(v)), 6),
                  "p90": round(float(np.percentile(v, 90)), 6)} for k, v in per.items()}
    return t.ms / steps, means.get(kernel), means, spread


PROFILES = os.path.join(ROOT, "profiles")
COPY_BYTES = 2 << 30


def measured_traffic(name):
    """HBM bytes per launch from the counter summary in profiles/, or None if
    there is none or the kernel's source changed since it was taken."""
    from paper_2608_23658_amd.profiling import traffic_if_current
    t = traffic_if_current(os.path.join(PROFILES, name), ROOT)
    return None if t is None else int(t)


def roofline_hbm(bytes_per_launch, kernel_ms, traffic=None):
    ach = bytes_per_launch / (kernel_ms * 1e-3) / 1e9
    return {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(ach / HBM_PEAK_GBS, 4), "traffic": traffic}


def roofline_mfma(flops_per_launch, kernel_ms, traffic=None):
    ach = flops_per_launch / (kernel_ms * 1e-3) / 1e12
    return {"bound": "mfma", "achieved": round(ach, 1), "peak": MFMA_BF16_PEAK_TFLOPS,
            "unit": "TFLOP/s", "frac": round(ach / MFMA_BF16_PEAK_TFLOPS, 4),
            "traffic": traffic}


def copy_leg(args):
    """A plain elementwise copy of COPY_BYTES (read COPY_BYTES, write COPY_BYTES):
    the known-size kernel whose byte counters calibrate the others."""
    n = COPY_BYTES // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(max(1, args.warmup)):
        torch.mul(src, 1.0, out=dst)
    with Timer() as t:
        for _ in range(args.steps):
            torch.mul(src, 1.0, out=dst)
    ms = t.ms / args.steps
    log(f"copy: {ms:.3f} ms, {2 * COPY_BYTES / ms / 1e6:.0f} GB/s read+write")
    return {"bytes_read": COPY_BYTES, "bytes_written": COPY_BYTES, "ms": ms,
            "gbs": 2 * COPY_BYTES / ms / 1e6}


def read_ceiling(args, K, b, kv, bt, sl, nbytes, split_ms):
    """The memory rate for decode's pattern: the read probe over the same
    batch (the K and V tiles of every block holding a token, same grid),
    timed over as many calls as the decode step."""
    out = torch.empty(K.probe_read_blocks_waves(b.num_seqs, 8, b.max_seq_len) * 64,
                      dtype=torch.int32, device="cuda")

    def call():
        K.probe_read_blocks(kv, b.num_blocks, bt, sl, num_kv_heads=8, head_dim=128,
                            dtype=torch.bfloat16, max_seq_len=b.max_seq_len, out=out)

    for _ in range(max(2, args.warmup)):
        call()
    with Timer() as t:
        for _ in range(args.steps):
            call()
    ms = t.ms / args.steps
    read = int(sum(-(-int(L) // 16) for L in b.seq_lens)) * 8 * 2 * 16 * 128 * 2
    res = {"probe": "read_blocks_kernel", "ms": round(ms, 5), "bytes_read": read,
           "read_gbs": round(read / (ms * 1e-3) / 1e9, 1),
           "algorithmic_gbs": round(nbytes / (ms * 1e-3) / 1e9, 1),
           "decode_split_time_over_probe": round(split_ms / ms, 4) if split_ms else None}
    log(f"decode read probe: {ms * 1e3:.1f} us, {res['read_gbs']} GB/s of its own reads, "
        f"decode split kernel / probe time {res['decode_split_time_over_probe']}")
    return res


def mfma_ceiling(args, K, prefill_tflops):
    """The matrix-unit rate this chip sustains in the prefill kernel's launch
    shape with random bf16 operands (the matrix probe: 2048 workgroups of
    eight wavefronts, one resident per CU at a time)."""
    wg, iters = 256 * 8, 2000
    out = torch.empty(wg * K.lib().kvattn_probe_mfma_threads(), dtype=torch.float32,
                      device="cuda")
    for _ in range(3):
        K.probe_mfma(wg, iters, out=out)
    n = max(3, args.steps // 5)
    with Timer() as t:
        for _ in range(n):
            K.probe_mfma(wg, iters, out=out)
    ms = t.ms / n
    tf = K.probe_mfma_flops(wg, iters) / (ms * 1e-3) / 1e12
    # one more call recording each wavefront's clock: the rate with random
    # operands is held down by the clock, not by the matrix pipes' issue
    clocks = torch.zeros(wg * 8 * 4, dtype=torch.int64, device="cuda")
    K.probe_mfma(wg, iters, out=out, clocks=clocks)
    torch.cuda.synchronize()
    res = {"probe": "mfma_rate_kernel", "ms": round(ms, 4), "tflops": round(tf, 1),
           "frac_of_peak": round(tf / MFMA_BF16_PEAK_TFLOPS, 4),
           "prefill_over_probe": round(prefill_tflops / tf, 4)}
    res.update(K.probe_mfma_clock(clocks, iters, tf))
    log(f"matrix probe: {tf:.0f} TFLOP/s ({res['frac_of_peak']:.3f} of peak), matrix pipes "
        f"{res['matrix_busy_median']:.3f} busy, so a clock of {res['clock_ghz_implied']} GHz; "
        f"prefill chunk kernel at {res['prefill_over_probe']:.3f} of it")
    return res


def decode_leg(args, K, work, wl):
    from workloads import DECODE_B256, make_batch
    spec = DECODE_B256
    log("decode: generating", spec.name)
    b = make_batch(spec)
    q = b.q.cuda()
    kv = b.kv_layer.cuda()
    bt = torch.from_numpy(b.block_table).cuda()
    sl = torch.from_numpy(b.seq_lens).cuda()
    out = torch.empty_like(q)
    ws = K.workspace(K.decode_workspace_bytes(b.num_seqs, 32, 128, b.max_seq_len))

    def step():
        K.decode(q, kv, b.num_blocks, bt, sl, num_kv_heads=8, max_seq_len=b.max_seq_len,
                 scale=b.scale, out=out, ws=ws)

    ms, kern_ms, means, spread = timed(step, args.steps, args.warmup, K, "decode_split")
    nbytes = work.decode_bytes(b.seq_lens, 32, 8, 128, 2)
    kvb = work.decode_kv_bytes(b.seq_lens, 8, 128, 2)
    log(f"decode: {ms * 1e3:.1f} us/step, kernels {means}")
    res = {
        "workload": spec.name, "ms_per_step": ms,
        "gbs": nbytes / (ms * 1e-3) / 1e9,
        "kv_gbs": kvb / (ms * 1e-3) / 1e9,
        "bytes_per_step": nbytes, "kernel_ms": means, "kernel_spread_ms": spread,
        "roofline": roofline_hbm(nbytes, kern_ms,
                                 measured_traffic("traffic_decode_split_b256_l512_4096.txt")),
        "num_seqs": b.num_seqs, "sum_seq_len": int(b.seq_lens.sum()),
    }
    res["ceiling"] = read_ceiling(args, K, b, kv, bt, sl, nbytes, kern_ms)
    return res, b


def two_tensor_leg(args, K, work, b):
    """The decode workload with its top 15% of block ids moved into a second,
    separately allocated tensor (the layer split the paper rejects), against
    the one-range decode over the same bytes."""
    q = b.q.cuda()
    kv = b.kv_layer.cuda()
    bt = torch.from_numpy(b.block_table).cuda()
    sl = torch.from_numpy(b.seq_lens).cuda()
    nb = b.num_blocks
    nbase = int(0.85 * nb)
    per_block = 2 * 8 * 16 * 128
    kv_base = kv[:nbase * per_block]
    kv_el = kv[nbase * per_block:].clone()
    out = torch.empty_like(q)
    ws = K.workspace(K.decode_workspace_bytes(q.shape[0], 32, 128, b.max_seq_len))
    nbytes = work.decode_bytes(b.seq_lens, 32, 8, 128, 2)
    res = {}
    for name, fn in (
            ("one_range", lambda: K.decode(q, kv, nb, bt, sl, num_kv_heads=8,
                                           max_seq_len=b.max_seq_len, scale=b.scale, out=out,
                                           ws=ws)),
            ("two_tensor", lambda: K.decode_two_tensor(q, kv_base, nbase, kv_el, nb - nbase, bt,
                                                       sl, num_kv_heads=8,
                                                       max_seq_len=b.max_seq_len, scale=b.scale,
                                                       out=out, ws=ws))):
        ms, _, _, _ = timed(fn, args.steps, args.warmup, K, "decode_split")
        res[name] = {"ms_per_call": ms, "gbs": nbytes / ms / 1e6}
    res["two_tensor_slowdown"] = res["two_tensor"]["ms_per_call"] / res["one_range"]["ms_per_call"]
    res["elastic_fraction_of_ids"] = float((b.block_table >= nbase).sum() /
                                           (b.block_table >= 0).sum())
    log(f"two-tensor: one range {res['one_range']['ms_per_call']:.4f} ms, two tensors "
        f"{res['two_tensor']['ms_per_call']:.4f} ms ({res['two_tensor_slowdown']:.4f}x)")
    return res


def prefill_leg(args, K, work):
    from workloads import PREFILL_L32768, make_batch
    spec = PREFILL_L32768
    log("prefill: generating", spec.name)
    b = make_batch(spec)
    q = b.q.cuda()
    kv = b.kv_layer.cuda()
    bt = torch.from_numpy(b.block_table).cuda()
    res = {}
    out = torch.empty_like(q)
    ws = K.workspace(K.prefill_workspace_bytes(1, 32768, 32, 128))
    # (a) the last 8192-token chunk over 24576 cached tokens; (b) the whole prompt
    for name, n, L in (("chunk8192_ctx24576", 8192, 32768), ("whole32768", 32768, 32768)):
        qq = q[L - n:L]
        oo = out[:n]
        sl = torch.tensor([L], dtype=torch.int32, device="cuda")
        cu = torch.tensor([0, n], dtype=torch.int32, device="cuda")

        def step():
            K.prefill_chunk(qq, kv, b.num_blocks, bt, sl, cu, num_kv_heads=8, max_seq_len=L,
                            max_num_batched_tokens=n, scale=b.scale, out=oo, ws=ws)

        steps = max(3, args.steps // 5)
        ms, kern_ms, means, spread = timed(step, steps, max(5, args.warmup), K, "prefill")
        flops = work.prefill_flops([L], [n], 32, 128)
        log(f"prefill {name}: {ms:.3f} ms/call, {flops / ms / 1e9:.1f} TFLOP/s, kernels {means}")
        res[name] = {"ms_per_call": ms, "tflops": flops / (ms * 1e-3) / 1e12,
                     "flops_per_call": flops, "kernel_ms": means,
                     "kernel_spread_ms": spread,
                     "roofline": roofline_mfma(flops, kern_ms, measured_traffic(
                         f"traffic_prefill_{name}.txt"))}
    return res, b


def mixed_leg(args, K, work):
    """The mixed step: one prefill call (8192 new rows of a 32768-token prompt)
    and one decode call (128 sequences), back to back on one stream."""
    from workloads import MIXED_STEP, make_batch
    spec = MIXED_STEP
    log("mixed: generating", spec.name)
    b = make_batch(spec)
    q = b.q.cuda()
    kv = b.kv_layer.cuda()
    bt = torch.from_numpy(b.block_table).cuda()
    sl = torch.from_numpy(b.seq_lens).cuda()
    qp, qd = q[:8192], q[8192:]
    op, od = torch.empty_like(qp), torch.empty_like(qd)
    slp = sl[:1]
    cup = torch.tensor([0, 8192], dtype=torch.int32, device="cuda")
    wsp = K.workspace(K.prefill_workspace_bytes(1, 8192, 32, 128))
    wsd = K.workspace(K.decode_workspace_bytes(128, 32, 128, b.max_seq_len))

    def step():
        K.prefill_chunk(qp, kv, b.num_blocks, bt[:1], slp, cup, num_kv_heads=8,
                        max_seq_len=b.max_seq_len, max_num_batched_tokens=8192 + 128,
                        scale=b.scale, out=op, ws=wsp)
        K.decode(qd, kv, b.num_blocks, bt[1:], sl[1:], num_kv_heads=8,
                 max_seq_len=b.max_seq_len, scale=b.scale, out=od, ws=wsd)

    steps = max(3, args.steps // 5)
    ms, _, means, _ = timed(step, steps, max(5, args.warmup), K, "prefill")
    flops = work.prefill_flops(b.seq_lens[:1], b.q_lens[:1], 32, 128)
    dbytes = work.decode_bytes(b.seq_lens[1:], 32, 8, 128, 2)
    log(f"mixed: {ms:.3f} ms/step, kernels {means}")

    # the same step as one unified prefill call (each decode sequence a
    # one-row chunk), as a serving engine batches it
    cu = torch.from_numpy(b.cu_seqlens_q).cuda()
    ou = torch.empty_like(q)
    wsu = K.workspace(K.prefill_workspace_bytes(b.num_seqs, b.total_q_tokens, 32, 128))

    def unified():
        K.prefill_chunk(q, kv, b.num_blocks, bt, sl, cu, num_kv_heads=8,
                        max_seq_len=b.max_seq_len, max_num_batched_tokens=8192 + 128,
                        scale=b.scale, out=ou, ws=wsu)

    ums, _, umeans, _ = timed(unified, steps, max(5, args.warmup), K, "prefill")
    log(f"mixed, one unified call: {ums:.3f} ms/step, kernels {umeans}")
    return {"workload": spec.name, "ms_per_step": ms, "kernel_ms": means,
            "prefill_tflops": flops / (means["prefill"] * 1e-3) / 1e12,
            "decode_gbs": dbytes / (means["decode_split"] * 1e-3) / 1e9,
            "unified_call": {"ms_per_step": ums, "kernel_ms": umeans}}


def append_leg(args, K, work):
    """Writing a step's new K/V rows into the paged layer of the decode
    workload's size (40704 blocks, 2.5 GiB): a decode step (one token for each
    of 256 sequences, distinct random slots) and an 8192-token prefill chunk of
    one sequence (consecutive slots through 512 random blocks)."""
    from workloads.append import make_append
    nb = 40704
    layer = torch.empty(nb * 2 * 8 * 16 * 128, dtype=torch.bfloat16, device="cuda")
    res = {}
    for name, T in (("decode_step256", 256), ("prefill_chunk8192", 8192)):
        a = make_append(T, num_kv_heads=8, head_dim=128, dtype="bf16", num_blocks=nb,
                        block_size=16, seed=4242 + T)
        if T > 256:
            # one sequence's chunk: consecutive slots through its (random) blocks
            blocks = torch.randperm(nb, generator=torch.Generator().manual_seed(T))[:T // 16]
            t = np.arange(T)
            a.slot_mapping = (blocks.numpy()[t // 16].astype(np.int64) * 16 +
                              t % 16).astype(np.int32)
        k, v = a.k_new.cuda(), a.v_new.cuda()
        sm = torch.from_numpy(a.slot_mapping).cuda()

        def step():
            K.kv_append(k, v, sm, layer, nb)

        ms, kern_ms, _, spread = timed(step, args.steps, args.warmup, K, "kv_append")
        # A call is this one launch. For a kernel of ~10 us the events around
        # each launch add about 2 us, more than the back-to-back launches
        # leave between them, so the per-call time of the timed loop (launch
        # gaps included) is the closer bound on the kernel's duration.
        dur_ms = min(ms, kern_ms)
        nbytes = work.append_bytes(T, 8, 128, 2)
        log(f"append {name}: {ms * 1e3:.1f} us/call, kernel {kern_ms * 1e3:.1f} us, "
            f"{nbytes / dur_ms / 1e6:.0f} GB/s")
        traffic = measured_traffic({"decode_step256": "traffic_kv_append_decode256.txt",
                                    "prefill_chunk8192": "traffic_kv_append_chunk8192.txt"}[name])
        res[name] = {"us_per_call": ms * 1e3, "kernel_us": kern_ms * 1e3,
                     "kernel_spread_ms": spread,
                     "bytes_per_call": nbytes, "roofline": roofline_hbm(nbytes, dur_ms, traffic)}
    return res


def toggle_leg(K):
    """Commit / decommit of a 3 GiB elastic reserve spread over 32 layers of
    128 MiB base each: the two-handle toggle with every step timed; when the
    physical pages arrive (the first write to the committed elastic pages
    against a second write); and the naive whole-handle toggle (one handle
    per layer over base + elastic, base contents copied in and out) on the
    same pool."""
    from workloads.configs import ELASTIC
    gran = max(K.ElasticPool.granularity(), 2 << 20)
    el = ELASTIC.elastic_bytes_per_layer
    assert el % gran == 0
    base = 64 * gran
    L = ELASTIC.num_layers
    pool = K.ElasticPool(L, base, el)
    med = statistics.median
    commit, decommit, st_c, st_d = [], [], [], []
    first, second = [], []
    whole_c, whole_d, wst_c, wst_d = [], [], [], []
    try:
        for l in range(L):
            pool.layer_view(l, committed_part=False).fill_(l)
        torch.cuda.synchronize()
        for i in range(22):
            c = pool.commit()
            sc = pool.last_steps()
            d = pool.decommit()
            sd = pool.last_steps()
            if i >= 2:
                commit.append(c)
                decommit.append(d)
                st_c.append(sc)
                st_d.append(sd)
        for i in range(6):
            pool.commit()
            views = [pool.layer_view(l)[base:] for l in range(L)]
            times = []
            for _ in range(2):
                with Timer() as t:
                    for v in views:
                        v.fill_(1)
                times.append(t.ms)
            del views
            pool.decommit()
            if i >= 1:
                first.append(times[0])
                second.append(times[1])
        for i in range(7):
            c = pool.commit_whole()
            sc = pool.last_steps()
            d = pool.decommit()
            sd = pool.last_steps()
            if i >= 2:
                whole_c.append(c)
                whole_d.append(d)
                wst_c.append(sc)
                wst_d.append(sd)
        base_ok = all(int(pool.layer_view(l, committed_part=False)[-1]) == l for l in range(L))
    finally:
        pool.close()

    def steps(rows, prefix):
        return {k[len(prefix):]: round(med([r[k] for r in rows]), 4) for k in rows[0]
                if k.startswith(prefix) and med([r[k] for r in rows]) > 0}
    res = {"reserve_bytes": el * L, "layers": L, "base_bytes_per_layer": base,
           "elastic_bytes_per_layer": el, "granularity": gran, "cycles": len(commit),
           "commit_ms_median": med(commit), "decommit_ms_median": med(decommit),
           "commit_steps_ms": steps(st_c, "commit_"),
           "decommit_steps_ms": steps(st_d, "decommit_"),
           "first_write_elastic_ms_median": med(first),
           "second_write_elastic_ms_median": med(second),
           "whole_handle": {"cycles": len(whole_c), "commit_ms_median": med(whole_c),
                            "decommit_ms_median": med(whole_d),
                            "commit_steps_ms": steps(wst_c, "commit_"),
                            "decommit_steps_ms": steps(wst_d, "decommit_"),
                            "base_contents_preserved": base_ok}}
    # one handle of the whole reserve, created, mapped and released (the
    # allocation cost alone; such a handle cannot back per-layer slices)
    single = [K.ElasticPool.time_single_handle(el * L) for _ in range(5)]
    res["single_handle_reserve_ms_median"] = {
        k: med([x[k] for x in single]) for k in ("create_ms", "map_ms", "access_ms",
                                                  "release_ms")}
    log(f"toggle: commit {res['commit_ms_median']:.2f} ms {res['commit_steps_ms']}, decommit "
        f"{res['decommit_ms_median']:.2f} ms {res['decommit_steps_ms']}; first write "
        f"{res['first_write_elastic_ms_median']:.2f} ms, second "
        f"{res['second_write_elastic_ms_median']:.2f} ms; whole-handle {res['whole_handle']}")
    return res


def controller_leg(K, work):
    """The toggle controller live at full reserve size: 32 layers of 1 GiB
    base (16384 blocks) plus 96 MiB elastic (1536 blocks), 3 GiB of reserve
    in all, hysteresis 2. A decode step over all 32 layers (48 sequences,
    lengths U[1024, 4096], 1300 of their blocks elastic) is captured
    in one HIP graph (kvattn_decode_noalloc, so the graph allocates nothing)
    and replayed. Sequence: decode-only steps until the controller commits;
    the batch takes its blocks (base first, then elastic) and is filled;
    graph replays; a prefill is announced: the controller refuses while
    elastic blocks are live, they are migrated to base blocks in every layer
    (plan + block copies + table rewrite, timed as the drain), then it
    decommits (other sequences having finished, so that base blocks are free
    to take the migrated ones); a 3 GiB activation burst stands in for the
    prefill; decode-only
    steps until it recommits (torch's cache emptied first). Every replay is
    checked bit for bit against the first."""
    from workloads.configs import ELASTIC as E
    L, HKV, D, HQ = E.num_layers, 8, 128, 32
    blk = 2 * HKV * 16 * D * 2
    nb_base, nb_el = 16384, E.elastic_blocks
    nb = nb_base + nb_el
    torch.cuda.empty_cache()
    pool = K.ElasticPool(L, nb_base * blk, nb_el * blk)
    bp = K.BlockPool(nb_base, nb_el)
    ctl = K.Controller(pool, bp, hysteresis=2)
    g = torch.Generator().manual_seed(2608)
    lens = torch.randint(1024, 4097, (48,), generator=g).numpy().astype(np.int32)
    need = int(sum((int(x) + 15) // 16 for x in lens))
    res = {"layers": L, "base_blocks": nb_base, "elastic_blocks": nb_el,
           "reserve_bytes": nb_el * blk * L, "num_seqs": len(lens),
           "sum_seq_len": int(lens.sum()), "hysteresis": 2, "events": []}
    try:
        filler = bp.alloc(nb_base - (need - 1300))      # other sequences' base blocks
        acts = []
        for step in range(3):
            a, ms = ctl.before_step(False)
            acts.append(a)
            if a:
                res["events"].append({"step": step, "action": "commit", "ms": ms,
                                      "steps_ms": pool.last_steps()})
        assert ctl.committed, acts
        ids = bp.alloc(need)
        res["elastic_fraction_of_ids"] = float((ids >= nb_base).mean())
        bt_np = np.full((len(lens), 256), -1, dtype=np.int32)
        o = 0
        for s_, Ls in enumerate(lens):
            nbk = (int(Ls) + 15) // 16
            bt_np[s_, :nbk] = ids[o:o + nbk]
            o += nbk
        bt = torch.from_numpy(bt_np).cuda()
        sl = torch.from_numpy(lens).cuda()
        idx = torch.from_numpy(ids.astype(np.int64)).cuda()
        for l in range(L):
            lay = pool.layer_view(l, dtype=torch.bfloat16).view(nb, blk // 2)
            lay[idx] = torch.randn(len(ids), blk // 2, device="cuda").to(torch.bfloat16)
        q = torch.randn(len(lens), HQ, D, generator=g).to(torch.bfloat16).cuda()
        outs = torch.empty(L, len(lens), HQ, D, dtype=torch.bfloat16, device="cuda")
        ptrs = [pool.layer_ptr(l) for l in range(L)]
        scale = 1.0 / np.sqrt(D)

        def step():
            for l in range(L):
                K.decode_noalloc(q, ptrs[l], nb, bt, sl, outs[l], num_kv_heads=HKV,
                                 max_seq_len=4096, scale=scale)
        step()
        torch.cuda.synchronize()
        ref = outs.clone()
        graph = torch.cuda.CUDAGraph()
        s2 = torch.cuda.Stream()
        s2.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s2):
            step()
            torch.cuda.synchronize()
            with torch.cuda.graph(graph, stream=s2):
                step()
        torch.cuda.synchronize()
        same = []

        def replay(n):
            ms = []
            for _ in range(n):
                outs.zero_()
                torch.cuda.synchronize()
                with Timer() as t:
                    graph.replay()
                ms.append(t.ms)
                same.append(bool(torch.equal(outs.view(torch.int16), ref.view(torch.int16))))
            return ms
        r1 = replay(10)
        # a prefill is announced: drain the elastic blocks by migration first
        a, ms = None, None
        try:
            ctl.before_step(True)
        except K.KvAttnError as e:
            res["refused_while_elastic_live"] = e.code == K.KV_ERR_STATE
        # other sequences have finished since: their base blocks are free again
        bp.free(filler[:2000])
        filler = filler[2000:]
        t0 = time.perf_counter()
        src, dst = bp.plan_drain()
        K.copy_blocks(ptrs, nb, blk, torch.from_numpy(src).cuda(), torch.from_numpy(dst).cuda())
        remap = np.arange(nb, dtype=np.int32)
        remap[src] = dst
        bt_np = np.where(bt_np >= 0, remap[np.maximum(bt_np, 0)], -1).astype(np.int32)
        bt.copy_(torch.from_numpy(bt_np))
        bp.free(src)
        torch.cuda.synchronize()
        res["drain_ms"] = (time.perf_counter() - t0) * 1e3
        res["drained_blocks"] = int(len(src))
        a, ms = ctl.before_step(True)
        res["events"].append({"action": "decommit" if a == K.KVCTL_DECOMMIT else a, "ms": ms,
                              "steps_ms": pool.last_steps()})
        burst = torch.empty(nb_el * blk * L, dtype=torch.uint8, device="cuda")
        burst.fill_(1)
        torch.cuda.synchronize()
        del burst
        r2 = replay(10)                                  # decode over base blocks only
        for step_i in range(3):
            a, ms = ctl.before_step(False)
            if a:
                res["events"].append({"action": "commit" if a == K.KVCTL_COMMIT else a,
                                      "ms": ms, "steps_ms": pool.last_steps()})
        r3 = replay(10)
        res["graph_step_ms_median"] = {"committed": statistics.median(r1),
                                       "after_decommit": statistics.median(r2),
                                       "after_recommit": statistics.median(r3)}
        nbytes = work.decode_bytes(lens, HQ, HKV, D, 2) * L
        res["graph_step_gbs"] = nbytes / (statistics.median(r1) * 1e-3) / 1e9
        res["replays_bitwise_equal"] = all(same)
        res["replays"] = len(same)
        res["counts"] = dict(zip(("commits", "decommits"), ctl.counts()))
        del filler
    finally:
        ctl.close()
        bp.close()
        pool.close()
        torch.cuda.empty_cache()
    for ev in res["events"]:
        ev["steps_ms"] = {k: round(v, 4) for k, v in ev["steps_ms"].items() if v > 0}
    log(f"controller: {res['events']}, drain {res['drain_ms']:.2f} ms "
        f"({res['drained_blocks']} blocks), graph steps {res['graph_step_ms_median']}, "
        f"bitwise {res['replays_bitwise_equal']}")
    return res


def necessity_leg():
    from paper_2608_23658_amd import necessity
    r = necessity.run()
    log(f"necessity: {r}")
    return r


def elastic_leg(args, K, work):
    """Decode over 32 layers of an elastic pool (base 96768 + 1536 elastic
    blocks of 64 KiB per layer, 3 GiB of elastic reserve in all), 512
    sequences U[8192, 32768], one shared table with >= 15% elastic references.
    States: committed; decommitted with the elastic references remapped onto
    base ids (same reuse structure; num_blocks = base blocks, so nothing can
    touch the unmapped range); recommitted with the elastic part refilled
    (output must equal the committed one bit for bit); and a plain
    torch-allocated copy of layer 0 as the control (against the pool's own
    layer 0 read 32 times, which has the same one-layer footprint)."""
    from workloads.configs import ELASTIC as E
    from workloads.elastic import (elastic_queries, elastic_tables, fill_layer,
                                   remap_elastic_to_base)
    bf16 = torch.bfloat16
    torch.cuda.empty_cache()
    bb = E.block_bytes
    base, el = E.base_blocks * bb, E.elastic_bytes_per_layer
    nb_all = E.base_blocks + E.elastic_blocks
    lens, bt_np, el_mask = elastic_tables(E)
    bt = torch.from_numpy(bt_np).cuda()
    bt_base = torch.from_numpy(remap_elastic_to_base(bt_np, E)).cuda()
    sl = torch.from_numpy(lens).cuda()
    q = elastic_queries(E).cuda()
    msl = int(lens.max())
    ws = K.workspace(K.decode_workspace_bytes(E.batch, E.num_q_heads, E.head_dim, msl))
    outs = torch.empty(E.num_layers, E.batch, E.num_q_heads, E.head_dim, dtype=bf16,
                       device="cuda")
    reps = 3

    def calls_ms(src, table, n=8):
        for _ in range(2):
            K.decode(q, src, nb_all, table, sl, num_kv_heads=E.num_kv_heads, max_seq_len=msl,
                     scale=E.scale, out=outs[0], ws=ws)
        with Timer() as t:
            for _ in range(n):
                K.decode(q, src, nb_all, table, sl, num_kv_heads=E.num_kv_heads,
                         max_seq_len=msl, scale=E.scale, out=outs[0], ws=ws)
        return t.ms / n

    # The mapping itself, like for like, before anything else of this leg is
    # allocated: a one-layer pool (base and elastic handle over one range) and
    # a hipMalloc copy of its bytes, read through the committed table (the hot
    # elastic set in the elastic handle), alternated (pool, copy, copy, pool).
    # Where an allocation's physical pages land moves its time by a few
    # percent either way, so the pair is allocated afresh six times, in
    # alternating order, and the ratio is reported over the six pairs.
    ratios, pairs = [], []
    for trial in range(6):
        one = K.ElasticPool(1, base, el) if trial % 2 == 0 else None
        cp1 = torch.empty(base + el, dtype=torch.uint8, device="cuda")
        if one is None:
            one = K.ElasticPool(1, base, el)
        try:
            one.commit(empty_cache=False)
            fill_layer(one.layer_view(0, dtype=bf16), 0, base // 2)
            cp1.copy_(one.layer_view(0))
            p0 = one.layer_ptr(0)
            p_runs, c_runs = [], []
            for src in (p0, cp1.data_ptr(), cp1.data_ptr(), p0):
                (p_runs if src == p0 else c_runs).append(calls_ms(src, bt))
            pm, cm = statistics.mean(p_runs), statistics.mean(c_runs)
            ratios.append(pm / cm)
            pairs.append({"pool_first": trial % 2 == 0, "pool_ms": pm, "hipmalloc_ms": cm})
        finally:
            one.close()
            del cp1
            torch.cuda.empty_cache()
    mapping = {"pool_over_hipmalloc_median": statistics.median(ratios),
               "pool_over_hipmalloc_min": min(ratios), "pool_over_hipmalloc_max": max(ratios),
               "pairs": pairs}
    log(f"elastic: one-layer mapping control {mapping}")
    log(f"elastic: pool of {E.num_layers} x ({base >> 20} MiB base + {el >> 20} MiB elastic)")
    # a hipMalloc layer allocated before the pool, so that it takes the
    # physical memory the pool's first layers would otherwise get
    early = torch.empty(base + el, dtype=torch.uint8, device="cuda")
    pool = K.ElasticPool(E.num_layers, base, el)
    res = {"workload": E.name, "layers": E.num_layers, "base_blocks": E.base_blocks,
           "elastic_blocks": E.elastic_blocks, "num_seqs": E.batch,
           "sum_seq_len": int(lens.sum()),
           "elastic_ref_fraction": float(el_mask.sum() / (bt_np >= 0).sum())}
    try:
        pool.commit()
        for l in range(E.num_layers):
            fill_layer(pool.layer_view(l, dtype=bf16), l, base // 2)
        ptrs = [pool.layer_ptr(l) for l in range(E.num_layers)]

        def sweep(table, nblocks, layers=None, src=None):
            for l in (range(E.num_layers) if layers is None else layers):
                K.decode(q, ptrs[l] if src is None else src, nblocks, table, sl,
                         num_kv_heads=E.num_kv_heads, max_seq_len=msl, scale=E.scale,
                         out=outs[l], ws=ws)

        def per_layer_ms(table, nblocks, layers=None, src=None):
            n = E.num_layers if layers is None else len(layers)
            sweep(table, nblocks, layers, src)
            with Timer() as t:
                for _ in range(reps):
                    sweep(table, nblocks, layers, src)
            return t.ms / (reps * n)

        committed = per_layer_ms(bt, nb_all)
        ref = outs.clone()
        log(f"elastic: committed {committed:.3f} ms/layer")
        dec_ms = pool.decommit()
        decommitted = per_layer_ms(bt_base, E.base_blocks)
        log(f"elastic: decommitted {decommitted:.3f} ms/layer")
        com_ms = pool.commit()
        for l in range(E.num_layers):
            fill_layer(pool.layer_view(l, dtype=bf16), l, base // 2, part="elastic")
        sweep(bt, nb_all)
        torch.cuda.synchronize()
        bitwise = bool(torch.equal(outs.view(torch.int16), ref.view(torch.int16)))
        recommitted = per_layer_ms(bt, nb_all)
        log(f"elastic: recommitted {recommitted:.3f} ms/layer, bitwise equal {bitwise}")
        # the footprint control: the pool's layer 0 read by all 32 calls of a
        # sweep, and the same bytes in plain torch memory, measured in turn
        # (pool, torch, torch, pool) so that neither gets the warmer GPU
        ctl = torch.empty(base + el, dtype=torch.uint8, device="cuda")
        ctl.copy_(pool.layer_view(0))
        l0 = [0] * E.num_layers
        pool_runs, ctl_runs = [], []
        for src in (None, ctl.data_ptr(), ctl.data_ptr(), None):
            (pool_runs if src is None else ctl_runs).append(per_layer_ms(bt, nb_all, l0, src))
        pool_l0 = statistics.median(pool_runs)
        control = statistics.median(ctl_runs)
        # each pool layer alone: the physical placement of a layer's pages
        # moves its time by several percent, VMM or not
        layer_ms = [per_layer_ms(bt, nb_all, [l] * 4) for l in range(E.num_layers)]
        ctl_equal = bool(torch.equal(outs[0].view(torch.int16), ref[0].view(torch.int16)))
        del ctl
        # placement: a layer's time follows where its physical pages are,
        # VMM or not. The hipMalloc layer allocated before the pool (early)
        # against the pool's first layer, and one allocated now (late)
        # against the pool's fastest layer, each alternated with its pool
        # layer (pool, copy, copy, pool, pool, copy) over the same bytes
        placement = {}
        late = torch.empty(base + el, dtype=torch.uint8, device="cuda")
        fastest = int(np.argmin(layer_ms))
        for tag, l, cp in (("early", 0, early), ("late", fastest, late)):
            cp.copy_(pool.layer_view(l))
            p_runs, c_runs = [], []
            for src in (None, cp.data_ptr(), cp.data_ptr(), None, None, cp.data_ptr()):
                (p_runs if src is None else c_runs).append(
                    per_layer_ms(bt, nb_all, [l] * 8, src))
            placement[tag] = {"pool_layer": l, "pool_ms": statistics.median(p_runs),
                              "hipmalloc_ms": statistics.median(c_runs),
                              "pool_over_hipmalloc": statistics.median(p_runs) /
                              statistics.median(c_runs),
                              "runs_ms": {"pool": p_runs, "hipmalloc": c_runs}}
        placement["slowest_pool_layer"] = {"layer": int(np.argmax(layer_ms)),
                                           "ms": max(layer_ms)}
        del late
        log(f"elastic: placement control {placement}")
        # toggle cycles on the full pool, no kernels in flight
        cyc_c, cyc_d = [], []
        for _ in range(12):
            cyc_d.append(pool.decommit())
            cyc_c.append(pool.commit(empty_cache=False))
    finally:
        pool.close()
        del early
        torch.cuda.empty_cache()
    nbytes = work.decode_bytes(lens, E.num_q_heads, E.num_kv_heads, E.head_dim, 2)
    med = statistics.median
    res.update({
        "bytes_per_layer": nbytes,
        "ms_per_layer": {"committed": committed, "decommitted": decommitted,
                         "recommitted": recommitted, "pool_layer0_x32": pool_l0,
                         "torch_layer0_x32": control},
        "gbs_per_layer": {k: nbytes / (v * 1e-3) / 1e9 for k, v in
                          (("committed", committed), ("decommitted", decommitted),
                           ("recommitted", recommitted), ("pool_layer0_x32", pool_l0),
                           ("torch_layer0_x32", control))},
        "layer0_x32_runs_ms": {"pool": pool_runs, "torch": ctl_runs},
        "pool_layer_ms": {"min": min(layer_ms), "median": statistics.median(layer_ms),
                          "max": max(layer_ms)},
        "mapping_control_one_layer": mapping,
        "placement_control": placement,
        "roofline_committed": roofline_hbm(
            nbytes, committed, measured_traffic("traffic_decode_split_elastic_32l_b512.txt")),
        "decommitted_vs_committed_pct": 100.0 * (decommitted / committed - 1.0),
        "recommitted_bitwise_equal": bitwise, "control_bitwise_equal": ctl_equal,
        "sweep_ms_committed": committed * E.num_layers,
        "toggle_during_protocol_ms": {"decommit": dec_ms, "commit": com_ms},
        "toggle_cycles_ms_median": {"decommit": med(cyc_d), "commit": med(cyc_c)},
    })
    return res


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return ""


def cpu_baseline(dec_batch, work, seconds):
    """The fp64 oracle, as it stands, on the host cores of this process:
    n = the CPUs this process may run on, and every thread pool the oracle
    can use (numpy's BLAS, torch) is set to n. Timed on bounded samples:

    - the decode workload (256 sequences, lengths U[512, 4096]): whole
      sequences in order until about `seconds` of wall time have passed,
      reported in the headline's unit (algorithmic GB/s);
    - the tiny fp32 decode, in full;
    - the mixed step's prefill chunk (8192 rows over 24576 cached tokens):
      four 256-row tiles at the chunk's start, one third, two thirds and end,
      each as the chunk of a sequence that ends at the tile's last row (a
      row's result depends only on the keys up to it), in algorithmic
      TFLOP/s of the sampled rows."""
    import threadpoolctl

    import oracle
    from workloads import MIXED_STEP, TINY_DECODE_F32, make_batch

    n = len(os.sched_getaffinity(0))
    torch.set_num_threads(n)
    res = {}
    with threadpoolctl.threadpool_limits(limits=n):
        def decode_rate(b, budget):
            seqs, t0 = [], time.perf_counter()
            for s in range(b.num_seqs):
                oracle.paged_decode(b.q_raw(), b.kv_raw(), b.block_table, b.seq_lens,
                                    dtype=b.dtype, num_q_heads=b.num_q_heads,
                                    num_kv_heads=b.num_kv_heads, head_dim=b.head_dim,
                                    block_size=b.block_size, scale=b.scale, seqs=[s])
                seqs.append(s)
                if time.perf_counter() - t0 > budget:
                    break
            wall = time.perf_counter() - t0
            lens = b.seq_lens[seqs]
            nbytes = work.decode_bytes(lens, b.num_q_heads, b.num_kv_heads, b.head_dim, b.esz)
            return nbytes, wall, len(seqs), int(lens.sum())

        nbytes, wall, ns, ntok = decode_rate(dec_batch, seconds)
        head = {"value": round(nbytes / wall / 1e9, 4), "unit": "GB/s", "cores": n,
                "kind": "oracle",
                "sample": f"fp64 oracle decode of the first {ns} of {dec_batch.num_seqs} "
                          f"sequences of decode_b256_l512_4096_bf16 ({ntok} context tokens, "
                          f"{nbytes} algorithmic bytes) in {wall:.2f} s wall on {n} threads",
                "cpu_model": _cpu_model()}
        res["decode_b256_l512_4096_bf16"] = {"value": head["value"], "unit": "GB/s",
                                             "seconds": round(wall, 3), "sequences": ns}
        tiny = make_batch(TINY_DECODE_F32)
        nbytes, wall, ns, ntok = decode_rate(tiny, 60.0)
        res[TINY_DECODE_F32.name] = {"value": round(nbytes / wall / 1e9, 6), "unit": "GB/s",
                                     "seconds": round(wall, 4), "sequences": ns,
                                     "sample": "in full"}
        mb = make_batch(MIXED_STEP)
        L, nq = int(mb.seq_lens[0]), int(mb.q_lens[0])
        c = L - nq
        T = mb.total_q_tokens
        q_all = np.asarray(mb.q_raw()).reshape(T, mb.num_q_heads, mb.head_dim)
        flops, t0 = 0, time.perf_counter()
        tiles = [0, (nq // 3) // 256 * 256, (2 * nq // 3) // 256 * 256, nq - 256]
        for r0 in tiles:
            r1 = r0 + 256
            oracle.paged_attention(q_all[r0:r1], mb.kv_raw(), mb.block_table[:1],
                                   np.array([c + r1], dtype=np.int32),
                                   np.array([0, r1 - r0], dtype=np.int32), dtype=mb.dtype,
                                   num_q_heads=mb.num_q_heads, num_kv_heads=mb.num_kv_heads,
                                   head_dim=mb.head_dim, block_size=mb.block_size,
                                   scale=mb.scale)
            flops += work.prefill_flops([c + r1], [r1 - r0], mb.num_q_heads, mb.head_dim)
        wall = time.perf_counter() - t0
        res["mixed_step_prefill_chunk8192_ctx24576"] = {
            "value": round(flops / wall / 1e12, 6), "unit": "TFLOP/s",
            "seconds": round(wall, 3),
            "sample": f"rows {tiles} (+256 each) of the 8192-row chunk, {flops} algorithmic "
                      f"FLOP; sampled, not the whole chunk"}
    head["by_workload"] = res
    return head


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py runs on one GPU only: the hot path has no multi-GPU form here "
              "(sharding is by KV head or by sequence with no exchange; see the design notes). "
              "Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    import paper_2608_23658_amd.kvattn as K
    from paper_2608_23658_amd import work
    K.lib()

    line = {"metric": "decode attn KV-read GB/s (% HBM peak); chunked-prefill attn TFLOP/s "
                      "(% MFMA)",
            "value": None, "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
            "warmup": args.warmup, "ms_per_step": None, "higher_is_better": True,
            "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
            "config": None}
    dec_batch = None
    if args.workload in ("all", "decode"):
        dec, dec_batch = decode_leg(args, K, work, None)
        line["value"] = round(dec["gbs"], 1)
        line["ms_per_step"] = round(dec["ms_per_step"], 5)
        line["config"] = {"workload": dec["workload"], "num_seqs": dec["num_seqs"],
                          "seq_len": "U[512,4096]", "sum_seq_len": dec["sum_seq_len"],
                          "num_q_heads": 32, "num_kv_heads": 8, "head_dim": 128,
                          "block_size": 16, "parallelism": "none (1 GPU)"}
        line["roofline"] = dec["roofline"]
        line["decode"] = {k: dec[k] for k in ("kv_gbs", "bytes_per_step", "kernel_ms",
                                              "kernel_spread_ms", "ceiling")}
    if args.workload in ("all", "two_tensor"):
        if dec_batch is None:
            from workloads import DECODE_B256, make_batch
            dec_batch = make_batch(DECODE_B256)
        line["two_tensor_decode"] = two_tensor_leg(args, K, work, dec_batch)
    if args.workload in ("all", "prefill"):
        pre, _ = prefill_leg(args, K, work)
        # the metric's second half as a flat record (the last 8192-token chunk
        # over 24576 cached tokens), with both cases nested under it
        p = pre["chunk8192_ctx24576"]
        line["prefill"] = {
            "metric": "chunked-prefill attn TFLOP/s (% bf16 MFMA peak)",
            "value": round(p["tflops"], 2), "unit": "TFLOP/s",
            "ms_per_step": round(p["ms_per_call"], 5), "dtype": "bf16",
            "config": {"workload": "prefill_chunk8192_ctx24576_bf16", "new_tokens": 8192,
                       "cached_tokens": 24576, "num_q_heads": 32, "num_kv_heads": 8,
                       "head_dim": 128, "block_size": 16},
            "roofline": p["roofline"], "cases": pre,
            "ceiling": mfma_ceiling(args, K, p["roofline"]["achieved"])}
        if line["value"] is None:
            line.update(value=round(p["tflops"], 2), unit="TFLOP/s",
                        ms_per_step=round(p["ms_per_call"], 5), roofline=p["roofline"],
                        config={"workload": "prefill_chunk8192_ctx24576_bf16"})
    if args.workload in ("all", "mixed"):
        line["mixed_step"] = mixed_leg(args, K, work)
    if args.workload in ("all", "append"):
        line["kv_append"] = append_leg(args, K, work)
        if line["value"] is None:
            p = line["kv_append"]["prefill_chunk8192"]
            line.update(value=round(p["roofline"]["achieved"], 1), unit="GB/s",
                        ms_per_step=round(p["us_per_call"] / 1e3, 5), roofline=p["roofline"],
                        config={"workload": "kv_append_8192x8x128_bf16"})
    if args.workload in ("all", "toggle"):
        line["elastic_toggle"] = toggle_leg(K)
    if args.workload in ("all", "controller"):
        line["live_controller"] = controller_leg(K, work)
    if args.workload in ("all", "necessity"):
        line["necessity"] = necessity_leg()
    if args.workload in ("all", "elastic"):
        line["elastic_decode"] = elastic_leg(args, K, work)
        if line["value"] is None:
            e = line["elastic_decode"]
            line.update(value=round(e["gbs_per_layer"]["committed"], 1), unit="GB/s",
                        ms_per_step=round(e["ms_per_layer"]["committed"], 5),
                        config={"workload": e["workload"]})
    if args.workload == "copy":
        c = copy_leg(args)
        line.update(value=round(c["gbs"], 1), unit="GB/s", ms_per_step=round(c["ms"], 5),
                    config={"workload": "elementwise_copy_2GiB_f32"}, copy=c)
    if dec_batch is not None and not args.no_cpu_baseline:
        log("cpu baseline: oracle sample")
        line["cpu_baseline"] = cpu_baseline(dec_batch, work, args.cpu_seconds)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
