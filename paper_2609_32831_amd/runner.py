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

from . import (NAME_DT, TORCH_DT, budget_state_tensor, dense_segment,
               make_shape, packed_layout, packed_segment, uc_assign_bits, uc_attend_append,
               uc_attend_mixed, uc_attend_workspace_size, uc_budget_params, uc_budget_step,
               uc_calibrate_policy, uc_dense_bytes, uc_dequantize_segment,
               uc_evict_rows_for_budget, uc_evicted_bytes, uc_packed_bytes, uc_quantize_segment,
               uc_score_columns, uc_score_importance, uc_score_workspace_size, uc_segment_mass,
               uc_select_keep, uc_stream_append, uc_topk_mass, uc_budget_state, AttendPlan,
               packed_storage, uc_evict_step)

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
        # streaming tail: decode rows join the first quantised segment
        self.stream = None
        if w.mode == "decode" and w.stream_tail:
            self.stream = next(i for i, p in enumerate(self.pol) if p.kind == "quant")
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
                cap = s.n + w.steps if i == self.stream else 0
                self.mixed.append(packed_segment(B, Hkv, s.n, D, s.group, dt,
                                                 bits=p.bits or 4, head_bits=hb, device=device,
                                                 capacity=cap))
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
        # workspaces are sized with the growing segments at full length
        if self.tail is not None:
            self.tail.n_rows = w.tail_capacity
        if self.stream is not None:
            self.mixed[self.stream].n_rows = w.segments[self.stream].n + w.steps
        M = w.M
        q_dt = NAME_DT[w.q_dtype]
        self.ws_attend = torch.empty(max(uc_attend_workspace_size(self.shape, self.mixed, q_dt, M), 256),
                                     dtype=torch.uint8, device=device)
        if self.tail is not None:
            self.tail.n_rows = 0
        if self.stream is not None:
            self.mixed[self.stream].n_rows = w.segments[self.stream].n

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
                self.mixed[i].n_rows = self.w.segments[i].n  # a streamed segment restarts
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
        if self.tail is not None:  # row t joins the protected tail in the same launch
            assert self.tail.n_rows == t
            uc_attend_append(self.shape, self.mixed, len(self.mixed) - 1, inp["k_dec"][t],
                             inp["v_dec"][t], 1, inp["q_dec"][t], 1, self.sm, o, lse, seg_lse,
                             ws=self.ws_attend)
            return
        if self.stream is not None:  # the row joins the quantised segment's tail
            uc_stream_append(self.shape, self.mixed[self.stream], inp["k_dec"][t], inp["v_dec"][t], 1)
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
                tot += uc_evicted_bytes(p.k, w.D, NAME_DT[s.dtype])
            else:
                tot += uc_packed_bytes(s.n, w.D, s.group, p.bits or 4, NAME_DT[s.dtype])
        return tot

    def attended_bytes(self, tail_rows: int = 0) -> int:
        """Algorithmic HBM bytes of one decode step's attention launch: every
        stored row it attends (dense rows, codes, float scales/minima, tails;
        not the index arrays) for all (b, h_kv), queries and fp32 outputs, and
        with a protected tail the new row it also stores there."""
        w = self.w
        BH = w.B * w.Hkv
        per = 0
        for i, (s, p) in enumerate(zip(w.segments, self.pol)):
            eb = 4 if s.dtype == "f32" else (2)
            if p.kind == "keep":
                per += s.n * 2 * w.D * eb
            elif p.kind == "evict":
                per += p.k * 2 * w.D * eb
            else:
                n = s.n + (tail_rows if i == self.stream else 0)  # streamed rows join it
                per += uc_packed_bytes(n, w.D, s.group, p.bits or 4, NAME_DT[s.dtype])
        if self.stream is None:
            per += (tail_rows + (1 if tail_rows else 0)) * 2 * w.D * 2
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


class DynamicRun:
    """One request (batch element) of a prefill workload under the dynamic
    budget of Sec. 3.3 (Eq. 1-3) with the Sec. 3.4 translation, on the
    library's kernels; host-side control flow only.

    Timestep 0 attends the uncompressed cache (the first full-KV step): its
    per-segment log-sum-exps give the type masses, and scores over the whole
    context from the step's query block select the kept rows of the evicting
    type.  Later timesteps attend the compressed cache and record their type
    masses; after every chunk of chunk_steps timesteps (if a timestep
    follows) uc_budget_step turns the chunk's masses into the next
    retention ratio (Eq. 3), type budgets (Eq. 2) and their translation on
    the device: a row count for the evicting type (fewer rows are chosen
    among those still kept, scored by the last obs_window query rows of each
    query head over the current cache, and their logical indices composed)
    and a (bits, group) configuration for the quantised type (a change
    re-quantises its dequantised rows).  The host reads the decision once per
    boundary, because the row count and the configuration size the next
    launches.  Eviction and re-quantisation are irreversible.

    Scores come from the row normalisers of the timestep's own attention
    pass (uc_score_columns): the observation rows are rows of that query
    block over the same cache, so its log-sum-exps are the softmax
    normalisers of Eq. 1's P.  Between boundaries the layout is frozen, so
    the timesteps run on an execution plan (App. E, cached metadata and
    execution plans) that prepares the packed rows once per layout."""

    def __init__(self, w, seg_k, seg_v, device="cuda"):
        """seg_k / seg_v: per segment, the request's rows [1, Hkv, n, D]."""
        self.w, self.device = w, device
        Hq, Hkv, D, M = w.Hq, w.Hkv, w.D, w.M
        self.shape = make_shape(1, Hq, Hkv, D)
        self.sm = sm_scale(D)
        segs = w.segments
        self.nseg = len(segs)
        self.ev = next(i for i, s in enumerate(segs) if s.policy == "evict")
        self.qt = next(i for i, s in enumerate(segs) if s.policy == "quant")
        self.cand = [self.ev, self.qt]
        self.dt = NAME_DT[segs[self.ev].dtype]
        self.tdt = TORCH[segs[self.ev].dtype]
        self.n_ev, self.n_qt = segs[self.ev].n, segs[self.qt].n
        self.dense = [dense_segment(seg_k[i], seg_v[i]) for i in range(self.nseg)]
        q_dt = NAME_DT[w.q_dtype]
        self.q_torch_dt = TORCH[w.q_dtype]
        # workspaces sized for the largest configuration: every row present,
        # the quantised type at the finest grouping
        biggest = packed_segment(1, Hkv, self.n_qt, D, 32, self.tdt, bits=8, device=device)
        full = list(self.dense)
        mixed = [biggest if i == self.qt else d for i, d in enumerate(self.dense)]
        ws_att = max(uc_attend_workspace_size(self.shape, full, q_dt, M),
                     uc_attend_workspace_size(self.shape, mixed, q_dt, M))
        ws_sc = max(uc_score_workspace_size(self.shape, full, M),
                    uc_score_workspace_size(self.shape, full, max(1, w.obs_window)))
        del biggest
        self.ws_att = torch.empty(max(ws_att, 256), dtype=torch.uint8, device=device)
        self.ws_sc = torch.empty(max(ws_sc, 256), dtype=torch.uint8, device=device)
        self.lse = torch.empty(1, Hq, M, device=device)
        self.lse_ptr = self.lse.data_ptr()
        self.seg_lse = torch.empty(1, Hq, M, self.nseg, device=device)
        # raw per-segment masses of every timestep (uc_segment_mass)
        self.mass = torch.zeros(w.steps, 1, Hkv, self.nseg, device=device)
        self.scores = torch.empty(1, Hkv, self.n_ev, device=device)
        # budget decisions on the device
        self.params = uc_budget_params(Hq, Hkv, D, M, self.nseg, self.ev, self.qt, self.n_ev,
                                       self.n_qt, self.dt, w.rho_init, w.rho_min)
        self.state = budget_state_tensor(device)
        self.state_host = torch.empty(self.state.numel(), dtype=torch.uint8, pin_memory=True)
        self.state_ready = torch.cuda.Event()
        self.falling = True
        # the kept rows of the evicting type and their logical indices: two
        # sets of buffers with a row capacity of every row, alternating (a
        # boundary keeps rows of one set in the other)
        cap = self.n_ev
        self.kept = [dense_segment(torch.empty(1, Hkv, cap, D, dtype=self.tdt, device=device),
                                   torch.empty(1, Hkv, cap, D, dtype=self.tdt, device=device),
                                   n_rows=0,
                                   idx=torch.empty(1, Hkv, cap, dtype=torch.int32, device=device))
                     for _ in range(2)]
        self.set = 1  # the set the first boundary fills is 0
        self.k_dev = self.state.data_ptr() + uc_budget_state.k.offset
        # the quantised type: two storage sets for its packed form (a
        # re-quantisation reads one and writes the other) and a buffer for
        # its decoded rows
        self.pstore = [packed_storage(1, Hkv, self.n_qt, D, self.tdt, device) for _ in range(2)]
        self.pset = 1
        self.deq_k = torch.empty(1, Hkv, self.n_qt, D, dtype=self.tdt, device=device)
        self.deq_v = torch.empty_like(self.deq_k)
        self.plan: Optional[AttendPlan] = None  # plan of the current layout
        # storage state
        self.compact = None     # dense segment of the kept rows of the evicting type
        self.packed = None      # packed segment of the quantised type
        self.cfg = None         # (index, bits, group)
        self.decisions: Dict[int, Dict] = {}

    # ---- helpers -----------------------------------------------------------
    @property
    def idx(self) -> torch.Tensor:
        """[Hkv, k] int32 logical positions of the evicting type's kept rows."""
        c = self.compact
        if c is None or c.t.get("idx") is None:
            n = self.n_ev
            return torch.arange(n, dtype=torch.int32, device=self.device).expand(self.w.Hkv, n)
        return c.t["idx"][0, :, :c.n_rows]

    def segments(self):
        if self.compact is None:
            return list(self.dense)
        out = list(self.dense)
        out[self.ev] = self.compact
        out[self.qt] = self.packed
        return out

    def _score(self, q, W):
        """Scores of the evicting type's current rows from the last W rows of
        q [1, Hq, M, D], the query block the last attention pass ran, over
        the current cache (the quantised type in its packed form); the
        normalisers are that pass's row log-sum-exps."""
        Hkv, M = self.w.Hkv, self.w.M
        segs = self.segments()
        n_cur = segs[self.ev].n_rows
        outs = [None] * self.nseg
        outs[self.ev] = self.scores.view(-1)[: Hkv * n_cur].view(1, Hkv, n_cur)
        uc_score_columns(self.shape, segs, q[:, :, M - W:], W, self.sm, self.lse_ptr + 4 * (M - W),
                         M, outs, None, ws=self.ws_sc, q_ld=M)

    def _evict(self):
        """Keep the best k rows of the evicting type's current rows in the
        other buffer set, k read from the budget state on the device (nothing
        is written when k is not below the current count)."""
        cur = self.segments()[self.ev]
        uc_evict_step(self.shape, self.scores, cur, self.k_dev, self.kept[1 - self.set])

    def _decode(self):
        """The quantised type's current rows, decoded into deq_k / deq_v."""
        uc_dequantize_segment(self.shape, self.packed, self.deq_k, self.deq_v)

    def _quantize(self, cfg, decoded: bool):
        """(Re-)quantise the quantised type with configuration cfg into the
        other storage set, from its original rows the first time, else from
        its current rows decoded into deq_k / deq_v (decoded: already done).
        The packed segment is all that stays resident."""
        w = self.w
        _, bits, group = cfg
        self.pset = 1 - self.pset
        pk = packed_segment(1, w.Hkv, self.n_qt, w.D, group, self.tdt, bits=bits,
                            device=self.device, storage=self.pstore[self.pset])
        if self.packed is None:
            src_k, src_v = self.dense[self.qt].t["k"], self.dense[self.qt].t["v"]
        else:
            if not decoded:
                self._decode()
            src_k, src_v = self.deq_k, self.deq_v
        uc_quantize_segment(self.shape, src_k, src_v, self.n_qt, pk)
        self.packed, self.cfg = pk, cfg

    def _boundary(self, t, t0, n, q, W):
        """Boundary after timestep t over the chunk t0 .. t0+n-1: the device
        decides (uc_budget_step), the host reads the decision and applies it
        from the next timestep on.  When the retention ratio was still above
        its floor at the last boundary (so the budget is likely to shrink
        again), the work that does not depend on the host knowing the
        decision is queued before the host waits for it: scoring the current
        cache, the eviction step (its row count is read on the device, and
        it writes nothing if the count did not fall) and decoding the
        quantised type's rows for a re-quantisation."""
        uc_budget_step(self.params, self.mass[t0:t0 + n], n, self.state)
        self.state_host.copy_(self.state, non_blocking=True)
        self.state_ready.record()
        first = self.compact is None
        ahead = first or self.falling
        if ahead:
            self._score(q, W)
            self._evict()
            if self.packed is not None:
                self._decode()
        while not self.state_ready.query():  # the decision is tiny: poll for it
            pass
        st = uc_budget_state.from_buffer_copy(self.state_host.numpy().tobytes())
        n_cur = self.n_ev if first else self.compact.n_rows
        if st.k < n_cur:
            if not ahead:
                self._score(q, W)
                self._evict()
            self.set = 1 - self.set
            self.compact = self.kept[self.set]
            self.compact.n_rows = st.k
            self.plan = None
        elif first:  # nothing evicted: the original rows stay
            self.compact = self.dense[self.ev]
        if st.cfg != st.cfg_prev or self.packed is None:
            self._quantize((st.cfg, st.bits, st.group), decoded=ahead)
            self.plan = None
        if self.plan is None:  # the new layout's execution plan
            self._make_plan()
        self.falling = st.rho > self.w.rho_min
        rec = {"rho": st.rho, "B": st.B, "m": {self.ev: st.m[0], self.qt: st.m[1]},
               "b": {self.ev: st.b[0], self.qt: st.b[1]}, "k": st.k, "cfg": st.cfg,
               "bits": st.bits, "group": st.group}
        self.decisions[t] = rec
        return rec

    def _make_plan(self):
        self.plan = AttendPlan(self.shape, self.segments(), None, self.q_torch_dt, self.w.M,
                               self.sm, ws=self.ws_att)

    # ---- one timestep --------------------------------------------------------
    def attend(self, t: int, q: torch.Tensor, o: torch.Tensor):
        """Timestep t's attention over the current cache (on the layout's
        execution plan) and its type masses."""
        w = self.w
        if self.plan is None:
            self._make_plan()
        self.plan.attend(q, o, self.lse, self.seg_lse)
        uc_segment_mass(self.shape, w.M, self.nseg, self.lse, self.seg_lse, self.mass[t])

    def step(self, t: int, q: torch.Tensor, o: torch.Tensor):
        """Timestep t with query block q [1, Hq, M, D]; returns the boundary
        decision taken after it, if any."""
        self.attend(t, q, o)
        return self.after_step(t, q)

    def after_step(self, t: int, q: torch.Tensor):
        """The budget bookkeeping after timestep t's attention and type masses
        (a decision at a chunk boundary)."""
        w = self.w
        if t == 0:
            return self._boundary(0, 0, 1, q, w.M)
        C = w.chunk_steps
        if t % C == 0 and t < w.steps - 1:
            return self._boundary(t, t - C + 1, C, q, w.obs_window)
        return None


def calibrate_policies(w, inp: Dict, examples: int, q_obs: Optional[torch.Tensor] = None,
                       W: Optional[int] = None, top: float = 0.1, threshold: float = 0.5,
                       device="cuda"):
    """Calibration-based policy assignment (Sec. 3.2; App. B, "Calibration
    Setting"): for every segment type, the fraction of its attention mass
    that its top `top` share of tokens captures, per (example, KV head), from
    the importance scores of the observation queries over the whole context;
    averaged over the first `examples` batch elements (the calibration
    examples) and their KV heads.  A type at `threshold` or above is assigned
    eviction, otherwise quantisation.  Returns {segment name: (concentration,
    policy)} and the per-(b, h_kv) fractions [examples * Hkv, n_segments]."""
    B, Hkv, D = w.B, w.Hkv, w.D
    assert 0 < examples <= B
    shape = make_shape(B, w.Hq, Hkv, D)
    full = [dense_segment(inp["seg_k"][i], inp["seg_v"][i]) for i in range(len(w.segments))]
    q_obs = inp["q_obs"] if q_obs is None else q_obs
    W = w.W if W is None else W
    scores = [torch.empty(B, Hkv, s.n, device=device) for s in w.segments]
    uc_score_importance(shape, full, q_obs, W, sm_scale(D), scores)
    n = len(w.segments)
    frac = torch.empty(B * Hkv, n, device=device)
    for i, s in enumerate(w.segments):
        k = int(math.ceil(top * s.n))
        col = torch.empty(B * Hkv, device=device)
        uc_topk_mass(scores[i].view(B * Hkv, s.n), k, col)
        frac[:, i] = col
    conc = torch.empty(n, dtype=torch.float64, device=device)
    evict = torch.empty(n, dtype=torch.int32, device=device)
    uc_calibrate_policy(frac[: examples * Hkv].contiguous(), threshold, conc, evict)
    c, e = conc.cpu().numpy(), evict.cpu().numpy()
    out = {s.name: (float(c[i]), "evict" if e[i] else "quant") for i, s in enumerate(w.segments)}
    return out, frac[: examples * Hkv].cpu().numpy()
