"""Offline calibration of the minimum retention ratio (App. B, "Calibration
Setting": rho_min is calibrated to match the target average KV compression
ratio) on the library's dynamic-budget run.

Host-side control only: every probe runs the whole dynamic chain
(``runner.DynamicRun``: attention, type masses, device-side budget
decisions, selection, re-quantisation) on the GPU, and the realized
compression comes from the decisions through the C ABI's byte-accounting
helpers.  The bisection follows the same probe sequence as the oracle's."""
from __future__ import annotations

from typing import Dict, List, Optional

import torch

from . import NAME_DT, uc_dense_bytes, uc_evicted_bytes, uc_packed_bytes
from .runner import DynamicRun


def realized_compression(w, decisions: Dict[int, Dict]) -> float:
    """1 - the mean over timesteps 1 .. steps-1 of stored / original bytes of
    the cached (kept, eviction- and quantisation-managed) segments, each
    timestep under the decision of the last boundary before it (App. B,
    "Compression Ratio"); protected segments are no part of the cache."""
    D = w.D
    cached = [s for s in w.segments if s.policy != "protect"]
    orig = sum(uc_dense_bytes(s.n, D, NAME_DT[s.dtype]) for s in cached)
    bounds = sorted(decisions)
    tot = 0.0
    for t in range(1, w.steps):
        d = decisions[max(b for b in bounds if b < t)]
        stored = 0
        for s in cached:
            dt = NAME_DT[s.dtype]
            if s.policy == "keep":
                stored += uc_dense_bytes(s.n, D, dt)
            elif s.policy == "evict":
                stored += uc_evicted_bytes(d["k"], D, dt)
            else:
                stored += uc_packed_bytes(s.n, D, d["group"], d["bits"], dt)
        tot += stored / orig
    return 1.0 - tot / (w.steps - 1)


def run_decisions(w, inp: Dict, b: int) -> Dict[int, Dict]:
    """The boundary decisions of one request's dynamic run on the GPU."""
    seg_k = [t[b:b + 1].contiguous() for t in inp["seg_k"]]
    seg_v = [t[b:b + 1].contiguous() for t in inp["seg_v"]]
    run = DynamicRun(w, seg_k, seg_v)
    o = torch.empty(1, w.Hq, w.M, w.D, device=seg_k[0].device)
    for t in range(w.steps):
        run.step(t, inp["q_pre"](t)[b:b + 1].contiguous(), o)
    torch.cuda.synchronize()
    return run.decisions


def calibrate_rho_min(w, inp: Dict, target: float, requests: Optional[List[int]] = None,
                      iters: int = 12) -> Dict:
    """rho_min whose average realized compression over the requests matches
    the target, by bisection on [0, rho_init] (the compression does not
    increase with rho_min); returns the probe closest to the target and all
    probes (rho_min, compression)."""
    import workloads as gen
    requests = [0] if requests is None else requests

    def f(x):
        wx = gen.scaled(w, rho_min=x)
        return sum(realized_compression(wx, run_decisions(wx, inp, b))
                   for b in requests) / len(requests)

    lo, hi = 0.0, w.rho_init
    probes = []
    for _ in range(iters):
        x = 0.5 * (lo + hi)
        c = f(x)
        probes.append((x, c))
        if c > target:
            lo = x
        else:
            hi = x
    best = min(probes, key=lambda p: abs(p[1] - target))
    return {"rho_min": best[0], "compression": best[1], "probes": probes}
