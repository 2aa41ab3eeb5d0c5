"""Static reclamation versus the dynamic toggle under an activation burst
(the paper, Section 4, "Static Reclamation is Unsafe"): with device memory
otherwise full, a reserve committed to KV leaves no room for a large
prefill's activations, while decommitting first lets the same burst run; and
a recommit right after the burst fails while the caching allocator still
holds the burst's memory, until that memory is returned (empty_cache).

Device memory is filled with a placeholder so that only reserve + margin is
free; everything is released on return.
"""
from __future__ import annotations

import time

import torch

from . import kvattn as K


def run(num_layers: int = 32, reserve_bytes: int = 3 << 30, margin_bytes: int = 1 << 30,
        device: int = 0) -> dict:
    gran = max(K.ElasticPool.granularity(device), 2 << 20)
    el = reserve_bytes // num_layers // gran * gran
    reserve = el * num_layers
    burst = reserve                      # the activations need what was lent to KV
    pool = K.ElasticPool(num_layers, gran, el, device)
    filler = None
    res = {"reserve_bytes": reserve, "burst_bytes": burst, "margin_bytes": margin_bytes}
    try:
        torch.cuda.empty_cache()
        free0, _ = torch.cuda.mem_get_info(device)
        fill = (free0 - burst - margin_bytes) // (2 << 20) * (2 << 20)
        res["filler_bytes"] = int(fill)
        filler = torch.empty(fill, dtype=torch.uint8, device=f"cuda:{device}")
        # static: the reserve is committed to KV when the burst arrives
        pool.commit()
        try:
            act = torch.empty(burst, dtype=torch.uint8, device=f"cuda:{device}")
            del act
            res["static_burst_oom"] = False
        except torch.OutOfMemoryError:
            res["static_burst_oom"] = True
        torch.cuda.empty_cache()
        # dynamic: decommit at the prefill boundary, run the burst, recommit
        res["decommit_ms"] = pool.decommit()
        try:
            act = torch.empty(burst, dtype=torch.uint8, device=f"cuda:{device}")
            act.fill_(1)
            torch.cuda.synchronize()
            del act
            res["dynamic_burst_ok"] = True
        except torch.OutOfMemoryError:
            res["dynamic_burst_ok"] = False
        # the freed burst is still cached by torch: a recommit cannot get it
        try:
            pool.commit(empty_cache=False)
            res["recommit_without_empty_cache"] = "ok"
        except K.KvAttnError as e:
            res["recommit_without_empty_cache"] = "oom" if e.code == K.KV_ERR_OOM else str(e)
        res["pool_consistent_after_failed_commit"] = not pool.is_committed
        # the recommit once torch has returned its cache: emptying the cache
        # and the commit's own steps, each timed
        torch.cuda.synchronize(device)
        t0 = time.perf_counter()
        torch.cuda.empty_cache()
        res["empty_cache_ms"] = (time.perf_counter() - t0) * 1e3
        res["recommit_ms"] = pool.commit(empty_cache=False)
        res["recommit_steps_ms"] = {k: v for k, v in pool.last_steps().items()
                                    if k.startswith("commit")}
        res["recommit_ok"] = pool.is_committed
        # the same recommit once more in steady state (nothing to return)
        pool.decommit()
        res["steady_recommit_ms"] = pool.commit(empty_cache=False)
        res["steady_recommit_steps_ms"] = {k: v for k, v in pool.last_steps().items()
                                           if k.startswith("commit")}
        pool.decommit()
    finally:
        del filler
        pool.close()
        torch.cuda.empty_cache()
    return res
