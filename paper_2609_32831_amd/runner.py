"""Drives one workload through the C ABI: importance scoring, budget ->
policy configuration, top-k eviction with compaction, quantization, then the
decode loop (append, attend) or the prefill timesteps.

Host-side control flow only (Sec. 3.3-3.4 order of operations); every
step on the data runs in libunicache's kernels.  Inputs are device tensors
prepared by the caller (the benchmark and the tests use the seeded
generators in ``workloads``).
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import Dict, List, Optional

import numpy as np
import torch

from . import (NAME_DT, TORCH_DT, dense_segment, make_shape, packed_layout, packed_segment,
               uc_append_rows, uc_assign_bits, uc_attend_mixed, uc_attend_workspace_size,
               uc_dense_bytes, uc_evict_rows_for_budget, uc_packed_bytes, uc_quantize_segment,
               uc_score_importance, uc_score_workspace_size, uc_segment_mass, uc_select_keep)

TORCH = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}


def sm_scale(D: int) -> float:
    return float(np.float32(1.0 / math.sqrt(D)))


@dataclass
class Policy:
    kind: str                  # keep | evict | quant
    k: int = 0                 # rows kept (evict)
    bits: Optional[int] = None  # code width (quant); None = per head from the budget
    group: int = 0


def plan_policies(w) -> List[Policy]:
    """Budget -> policy configuration for every segment (Sec. 3.4): rows kept
    by an eviction policy, code width and group of a quantization policy.
    Budgets count stored bytes of one (b, h_kv); the original size is counted
    at the workload's I/O element type."""
    D = w.D
    io = NAME_DT[w.q_dtype]
    orig = sum(uc_dense_bytes(s.n, D, io) for s in w.segments)
    budget = orig / w.budget_ratio if w.budget_ratio else None
    pols: List[Policy] = []
    fixed = 0
    for s in w.segments:
        if s.policy == "keep":
            pols.append(Policy("keep"))
            fixed += uc_dense_bytes(s.n, D, NAME_DT[s.dtype])
        elif s.policy == "quant":
            pols.append(Policy("quant", bits=s.bits, group=s.group))
            if s.bits:
                fixed += uc_packed_bytes(s.n, D, s.group, s.bits, NAME_DT[s.dtype])
        else:
            pols.append(Policy("evict"))
    for s, p in zip(w.segments, pols):
        if p.kind != "evict":
            continue
        if s.keep_ratio is not None:
            p.k = int(math.floor(s.keep_ratio * s.n))
        else:
            p.k = int(uc_evict_rows_for_budget(budget, fixed, s.n, D, NAME_DT[s.dtype]))
    return pols


class Run:
    """One workload on the GPU.  inp holds device tensors:
      seg_k[i], seg_v[i]   [B, Hkv, n_i, D] pre-compression segment rows
      q_obs                [B, Hq, W, D]    observation queries for scoring
      decode: q_dec [steps, B, Hq, 1, D], k_dec / v_dec [steps, B, Hkv, 1, D]
      prefill: q_pre(t) -> [B, Hq, M, D] (callable)"""

    def __init__(self, w, inp: Dict, device="cuda", head_bits: Optional[List[int]] = None):
        self.w, self.inp, self.device = w, inp, device
        self.shape = make_shape(w.B, w.Hq, w.Hkv, w.D)
        self.sm = sm_scale(w.D)
        self.pol = plan_policies(w)
        B, Hkv, D = w.B, w.Hkv, w.D
        BH = B * Hkv
        self.full = [dense_segment(inp["seg_k"][i], inp["seg_v"][i]) for i in range(len(w.segments))]
        self.scores: Dict[int, torch.Tensor] = {}
        self.keep: Dict[int, torch.Tensor] = {}
        self.mixed = []
        for i, (s, p) in enumerate(zip(w.segments, self.pol)):
            dt = TORCH[s.dtype]
            if p.kind == "keep":
                self.mixed.append(self.full[i])
            elif p.kind == "evict":
                self.scores[i] = torch.empty(B, Hkv, s.n, device=device)
                self.keep[i] = torch.empty(BH, max(p.k, 1), dtype=torch.int32, device=device)
                kc = torch.empty(B, Hkv, max(p.k, 1), D, dtype=dt, device=device)
                vc = torch.empty_like(kc)
                seg = dense_segment(kc, vc, n_rows=p.k, idx=self.keep[i])
                self.mixed.append(seg)
            else:
                hb = head_bits if p.bits is None else None
                if p.bits is None and hb is None:
                    hb = [4] * BH
                self.mixed.append(packed_segment(B, Hkv, s.n, D, s.group, dt,
                                                 bits=p.bits or 4, head_bits=hb, device=device))
        self.tail = None
        if w.mode == "decode" and w.tail_capacity:
            tk = torch.zeros(B, Hkv, w.tail_capacity, D, dtype=TORCH["bf16"] if w.q_dtype == "bf16"
                             else TORCH[w.q_dtype], device=device)
            self.tail = dense_segment(tk, torch.zeros_like(tk), n_rows=0)
            self.mixed.append(self.tail)
        self.n_score = len(w.segments)
        self.mass = torch.empty(B, Hkv, self.n_score, device=device)
        self.ws_score = torch.empty(max(uc_score_workspace_size(self.shape, self.full, w.W), 256),
                                    dtype=torch.uint8, device=device)
        if self.tail is not None:
            self.tail.n_rows = w.tail_capacity
        M = w.M
        q_dt = NAME_DT[w.q_dtype]
        self.ws_attend = torch.empty(max(uc_attend_workspace_size(self.shape, self.mixed, q_dt, M), 256),
                                     dtype=torch.uint8, device=device)
        if self.tail is not None:
            self.tail.n_rows = 0

    # -- compression (once per prefill / per chunk) --------------------------
    def score(self, q_obs=None, W=None):
        q_obs = self.inp["q_obs"] if q_obs is None else q_obs
        W = self.w.W if W is None else W
        outs = [self.scores.get(i) for i in range(self.n_score)]
        uc_score_importance(self.shape, self.full, q_obs, W, self.sm, outs, self.mass,
                            ws=self.ws_score)

    def select(self):
        w = self.w
        BH = w.B * w.Hkv
        for i, p in enumerate(self.pol):
            if p.kind != "evict":
                continue
            n = w.segments[i].n
            seg = self.mixed[i]
            uc_select_keep(self.scores[i].view(BH, n), p.k, 0, self.keep[i],
                           self.inp["seg_k"][i].view(BH, n, w.D), self.inp["seg_v"][i].view(BH, n, w.D),
                           seg.t["k"].view(BH, -1, w.D), seg.t["v"].view(BH, -1, w.D))

    def quantize(self, k_src=None, v_src=None):
        for i, p in enumerate(self.pol):
            if p.kind == "quant":
                k = self.inp["seg_k"][i] if k_src is None else k_src
                v = self.inp["seg_v"][i] if v_src is None else v_src
                uc_quantize_segment(self.shape, k, v, self.w.segments[i].n, self.mixed[i])

    def compress(self):
        if self.scores:
            self.score()
        self.select()
        self.quantize()
        if self.tail is not None:
            self.tail.n_rows = 0

    # -- hot loop --------------------------------------------------------------
    def decode_step(self, t: int, o: torch.Tensor, lse=None, seg_lse=None):
        inp = self.inp
        if self.tail is not None:
            uc_append_rows(self.shape, inp["k_dec"][t], inp["v_dec"][t], 1, self.tail, t)
            self.tail.n_rows = t + 1
        uc_attend_mixed(self.shape, self.mixed, inp["q_dec"][t], 1, self.sm, o, lse, seg_lse,
                        ws=self.ws_attend)

    def prefill_step(self, q: torch.Tensor, o: torch.Tensor, lse=None, seg_lse=None):
        uc_attend_mixed(self.shape, self.mixed, q, self.w.M, self.sm, o, lse, seg_lse,
                        ws=self.ws_attend)

    # -- bookkeeping -----------------------------------------------------------
    def stored_bytes_per_head(self) -> int:
        w = self.w
        tot = 0
        for s, p in zip(w.segments, self.pol):
            if p.kind == "keep":
                tot += uc_dense_bytes(s.n, w.D, NAME_DT[s.dtype])
            elif p.kind == "evict":
                tot += p.k * (2 * w.D * (4 if s.dtype == "f32" else 2) + 4)
            else:
                tot += uc_packed_bytes(s.n, w.D, s.group, p.bits or 4, NAME_DT[s.dtype])
        return tot

    def attended_bytes(self, tail_rows: int = 0) -> int:
        """Algorithmic HBM bytes one attention call reads: every stored row it
        attends (dense rows, codes, float scales/minima, tails; not the index
        arrays) for all (b, h_kv), plus queries and fp32 outputs."""
        w = self.w
        BH = w.B * w.Hkv
        per = 0
        for s, p, seg in zip(w.segments, self.pol, self.mixed):
            eb = 4 if s.dtype == "f32" else (2)
            if p.kind == "keep":
                per += s.n * 2 * w.D * eb
            elif p.kind == "evict":
                per += p.k * 2 * w.D * eb
            else:
                per += uc_packed_bytes(s.n, w.D, s.group, p.bits or 4, NAME_DT[s.dtype])
        per += tail_rows * 2 * w.D * 2
        qb = 4 if w.q_dtype == "f32" else 2
        M = w.M if w.mode == "prefill" else 1
        return BH * per + w.B * w.Hq * M * w.D * (qb + 4)


class DenoiseRun:
    """A denoising workload whose quantised latent gets per-head code widths
    from its attention mass (text-to-image): a kept text segment plus one
    latent segment under a shared storage budget per batch element.

    Timestep t: at t = 0 (no widths yet) the latent is attended dense, as the
    first full-KV step that initialises the statistics (Sec. 3.3); afterwards
    the current latent keys are re-quantised with the current widths
    (int2/int4 per KV head) and attended packed.  Every rescore_every steps
    the step's per-segment log-sum-exps give each KV head's latent mass
    (Eq. 1 bracket at head granularity), and the widths for the next steps are
    assigned greedily: all heads at 2 bits, heads raised to 4 bits in
    descending mass order while the batch element's stored bytes stay within
    its budget.  Host-side control flow only."""

    def __init__(self, w, seg_k, seg_v, device="cuda"):
        self.w, self.device = w, device
        B, Hkv, D = w.B, w.Hkv, w.D
        self.BH = B * Hkv
        self.shape = make_shape(w.B, w.Hq, w.Hkv, D)
        self.sm = sm_scale(D)
        self.lat = next(i for i, s in enumerate(w.segments) if s.policy == "quant")
        ls = w.segments[self.lat]
        self.G, self.N = ls.group, ls.n
        self.dt = NAME_DT[ls.dtype]
        self.dense = [dense_segment(seg_k[i], seg_v[i]) for i in range(len(w.segments))]
        self.packed = packed_segment(B, Hkv, self.N, D, self.G, TORCH[ls.dtype], bits=4,
                                     head_bits=[4] * self.BH, device=device)
        self.bits = None
        io = NAME_DT[w.q_dtype]
        orig = sum(uc_dense_bytes(s.n, D, io) for s in w.segments)
        fixed = sum(uc_dense_bytes(s.n, D, NAME_DT[s.dtype]) for i, s in enumerate(w.segments)
                    if i != self.lat)
        self.budget_b = Hkv * orig / w.budget_ratio   # per batch element
        self.fixed_b = Hkv * fixed
        q_dt = NAME_DT[w.q_dtype]
        ws = max(uc_attend_workspace_size(self.shape, self.dense, q_dt, w.M),
                 uc_attend_workspace_size(self.shape, self._segs_packed(), q_dt, w.M))
        self.ws = torch.empty(max(ws, 256), dtype=torch.uint8, device=device)
        nseg = len(w.segments)
        self.lse = torch.empty(B, w.Hq, w.M, device=device)
        self.seg_lse = torch.empty(B, w.Hq, w.M, nseg, device=device)
        self.mass = torch.empty(B, Hkv, nseg, device=device)

    def _segs_packed(self):
        return [self.packed if i == self.lat else d for i, d in enumerate(self.dense)]

    def set_bits(self, bits):
        """Per-(b, h_kv) code widths; codes of consecutive heads are packed
        back to back."""
        off, total = packed_layout(self.BH, self.N, self.w.D, self.G, bits)
        t = self.packed.t
        assert total <= t["codes_k"].numel()
        t["head_bits"].copy_(torch.tensor(bits, dtype=torch.uint8))
        t["code_off"].copy_(torch.tensor(off, dtype=torch.int64))
        self.packed.desc.bits = max(bits)
        self.bits = list(bits)

    def assign(self, mass_latent):
        """Greedy int2/int4 widths of every batch element from [B, Hkv] masses."""
        w = self.w
        out = []
        for b in range(w.B):
            out += uc_assign_bits(list(mass_latent[b]), self.N, w.D, self.G, self.dt,
                                  self.budget_b, self.fixed_b)
        return out

    def step(self, t: int, q: torch.Tensor, o: torch.Tensor, want_stats: bool = False):
        """One timestep over the current latent keys (already in seg_k).  With
        want_stats (and at every rescoring step) lse / seg_lse are produced;
        at a rescoring step the widths for the following steps are assigned
        and returned."""
        w = self.w
        if self.bits is None:
            segs = self.dense
        else:
            segs = self._segs_packed()
            uc_quantize_segment(self.shape, self.dense[self.lat].t["k"],
                                self.dense[self.lat].t["v"], self.N, self.packed)
        rescore = w.rescore_every and t % w.rescore_every == 0
        stats = want_stats or rescore
        uc_attend_mixed(self.shape, segs, q, w.M, self.sm, o, self.lse if stats else None,
                        self.seg_lse if stats else None, ws=self.ws)
        if not rescore:
            return None
        uc_segment_mass(self.shape, w.M, len(w.segments), self.lse, self.seg_lse, self.mass)
        m = self.mass[:, :, self.lat].cpu().numpy()
        new = self.assign(m)
        self.set_bits(new)
        return new
