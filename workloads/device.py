"""Device copies of a workload's seeded inputs (torch tensors in the shapes
the runner expects).  Input recipes only; no method arithmetic."""
from __future__ import annotations

from typing import Dict, Optional

import numpy as np
import torch

from . import T_QDEC, T_QOBS, T_QPRE, Workload, decode_kv, queries, segment_kv

TORCH = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}


def to_device(a: np.ndarray, dtype: str, device) -> torch.Tensor:
    a = np.ascontiguousarray(a)
    if dtype == "bf16":
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(device)
    return torch.from_numpy(a).to(device)


def device_inputs(w: Workload, device="cuda", steps: Optional[int] = None) -> Dict:
    B, Hq, Hkv, D = w.B, w.Hq, w.Hkv, w.D
    inp: Dict = {"seg_k": [], "seg_v": []}
    for i, s in enumerate(w.segments):
        for which in ("k", "v"):
            a = segment_kv(w, i, which)
            inp["seg_" + which].append(to_device(a, s.dtype, device).view(B, Hkv, s.n, D))
    inp["q_obs"] = to_device(queries(w, T_QOBS, w.W), w.q_dtype, device).view(B, Hq, w.W, D)
    if w.mode == "decode":
        n = w.steps if steps is None else steps
        q = queries(w, T_QDEC, n).reshape(B, Hq, n, D).transpose(2, 0, 1, 3)
        inp["q_dec"] = to_device(q, w.q_dtype, device).view(n, B, Hq, 1, D)
        tdt = "bf16" if w.q_dtype == "bf16" else w.q_dtype
        for which in ("k", "v"):
            a = decode_kv(w, which, 0, n).reshape(B, Hkv, n, D).transpose(2, 0, 1, 3)
            inp[which + "_dec"] = to_device(a, tdt, device).view(n, B, Hkv, 1, D)
    else:
        def q_pre(t: int) -> torch.Tensor:
            return to_device(queries(w, T_QPRE, w.M, step=t), w.q_dtype, device).view(B, Hq, w.M, D)
        inp["q_pre"] = q_pre
    return inp


class DenoiseInputs:
    """Device inputs of a denoising workload whose latent keys and query block
    drift as a seeded random walk across timesteps (text-to-image): text K/V
    and latent V stay fixed; latent K and the 4096-row query block of every
    query head take X_t = X_{t-1} + sigma * eps_t on fp64 masters, rounded to
    the storage dtype each step.  Input recipes only."""

    def __init__(self, w: Workload, device="cuda", latent: int = 1):
        from . import T_DRIFT_K, T_DRIFT_Q, Drift
        B, Hq, Hkv, D = w.B, w.Hq, w.Hkv, w.D
        self.w, self.device, self.latent = w, device, latent
        self.seg_k, self.seg_v = [], []
        for i, s in enumerate(w.segments):
            if i == latent:
                k, mk = segment_kv(w, i, "k", master=True)
                self.drift_k = Drift(w, T_DRIFT_K, mk, s.dtype)
            else:
                k = segment_kv(w, i, "k")
            self.seg_k.append(to_device(k, s.dtype, device).view(B, Hkv, s.n, D))
            self.seg_v.append(to_device(segment_kv(w, i, "v"), s.dtype, device).view(B, Hkv, s.n, D))
        q, mq = queries(w, T_QPRE, w.M, step=0, master=True)
        self.drift_q = Drift(w, T_DRIFT_Q, mq, w.q_dtype)
        self.q = to_device(q, w.q_dtype, device).view(B, Hq, w.M, D)
        self.t = 0

    def advance(self):
        """Step t -> t+1: drift the latent keys and the queries (device copies
        updated in place)."""
        w = self.w
        self.t += 1
        k = self.drift_k.step()
        self.seg_k[self.latent].copy_(to_device(k, w.segments[self.latent].dtype, self.device)
                                      .view(self.seg_k[self.latent].shape))
        self.q.copy_(to_device(self.drift_q.step(), w.q_dtype, self.device).view(self.q.shape))
