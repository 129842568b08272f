"""Oracle pipeline for one KV head of a workload -- TEST INFRASTRUCTURE ONLY.

Chains the oracle's steps in the paper's order for a single (b, h_kv) and
its query heads: importance scores over the uncompressed context (Sec. 3.3),
budget -> rows kept / code width (Sec. 3.4), top-k eviction (App. E,
"Batched GQA token selection"), quantization (App. E storage), then masked,
fake-quantized attention over the full logical sequence (App. E reference
formulation).  Everything here is computed by ``oracle`` functions; the
inputs come from the shared seeded generator.
"""
from __future__ import annotations

import math
from typing import Dict, List, Optional

import numpy as np

import workloads as gen

from . import (ELEM, assign_bits, attend, dense_bytes, dequant, evict_rows, packed_bytes,
               quant_config, quantize, retention_next, score64, select, type_budget, widen)


def sm_scale(D: int) -> float:
    return float(np.float32(1.0 / math.sqrt(D)))


def plan(w) -> List[Dict]:
    """Rows kept per eviction segment and code width per quantised segment,
    from the storage budget of one (b, h_kv)."""
    D = w.D
    orig = sum(dense_bytes(s.n, D, w.q_dtype) for s in w.segments)
    budget = orig / w.budget_ratio if w.budget_ratio else None
    fixed = 0
    out = []
    for s in w.segments:
        if s.policy == "keep":
            out.append({"kind": "keep"})
            fixed += dense_bytes(s.n, D, s.dtype)
        elif s.policy == "quant":
            out.append({"kind": "quant", "bits": s.bits, "group": s.group})
            if s.bits:
                fixed += packed_bytes(s.n, D, s.group, s.bits, s.dtype)
        else:
            out.append({"kind": "evict"})
    for s, p in zip(w.segments, out):
        if p["kind"] == "evict":
            p["k"] = (int(math.floor(s.keep_ratio * s.n)) if s.keep_ratio is not None
                      else evict_rows(budget, fixed, s.n, D, s.dtype))
    return out


def head_inputs(w, b: int, h: int, steps: int = 0) -> Dict:
    """Generator bytes for KV head (b, h) and its query heads."""
    G = w.group_size
    bh = b * w.Hkv + h
    bq0 = b * w.Hq + h * G
    inp = {"seg_k": [], "seg_v": []}
    for i in range(len(w.segments)):
        inp["seg_k"].append(gen.segment_kv(w, i, "k", bh0=bh, nbh=1)[0])
        inp["seg_v"].append(gen.segment_kv(w, i, "v", bh0=bh, nbh=1)[0])
    inp["q_obs"] = gen.queries(w, gen.T_QOBS, w.W, bh0=bq0, nbh=G)
    if steps:
        inp["q_dec"] = gen.queries(w, gen.T_QDEC, steps, bh0=bq0, nbh=G)      # [G, steps, D]
        inp["k_dec"] = gen.decode_kv(w, "k", 0, steps, bh0=bh, nbh=1)[0]     # [steps, D]
        inp["v_dec"] = gen.decode_kv(w, "v", 0, steps, bh0=bh, nbh=1)[0]
    return inp


def compress_head(w, inp: Dict, pols: List[Dict], bits_override: Optional[int] = None) -> Dict:
    """Scores, mass, kept rows and quantised storage of one KV head."""
    D, G = w.D, w.group_size
    segs = w.segments
    K = np.concatenate([widen(inp["seg_k"][i], s.dtype) for i, s in enumerate(segs)], axis=0)
    seg_id = np.concatenate([np.full(s.n, i, np.int32) for i, s in enumerate(segs)])
    q = widen(inp["q_obs"], w.q_dtype)[None]                # [1, G, W, D]
    sc64, ms64 = score64(q, K[None, None], seg_id, len(segs), sm_scale(D))
    sc = sc64[0, 0].astype(np.float32)
    out = {"score64": sc64[0, 0], "score": sc, "mass": ms64[0, 0].astype(np.float32),
           "keep": {}, "packed": {}, "khat": [], "vhat": [], "present": []}
    start = 0
    for i, (s, p) in enumerate(zip(segs, pols)):
        n = s.n
        k_i, v_i = inp["seg_k"][i], inp["seg_v"][i]
        pres = np.ones(n, np.uint8)
        if p["kind"] == "evict":
            keep = select(sc[start:start + n][None], p["k"], 0)[0]
            out["keep"][i] = keep
            pres[:] = 0
            pres[keep] = 1
            kh, vh = widen(k_i, s.dtype), widen(v_i, s.dtype)
        elif p["kind"] == "quant":
            b_ = p["bits"] if p["bits"] else bits_override
            pk = quantize(k_i[None], v_i[None], s.dtype, p["group"], [b_])
            out["packed"][i] = pk
            kh, vh = dequant(pk, n, D, p["group"], s.dtype)
            kh, vh = kh[0], vh[0]
        else:
            kh, vh = widen(k_i, s.dtype), widen(v_i, s.dtype)
        out["khat"].append(kh)
        out["vhat"].append(vh)
        out["present"].append(pres)
        start += n
    return out


def attend_head(w, comp: Dict, q: np.ndarray, q_dtype: str, tail_k=None, tail_v=None,
                tail_dtype: str = "bf16"):
    """Masked shared-softmax attention of q [G, M, D] (stored dtype) over the
    head's logical sequence (+ optional protected tail rows [t, D])."""
    ks, vs, pr = list(comp["khat"]), list(comp["vhat"]), list(comp["present"])
    seg_id = [np.full(k.shape[0], i, np.int32) for i, k in enumerate(ks)]
    n_segs = len(ks)
    if tail_k is not None:
        ks.append(widen(tail_k, tail_dtype))
        vs.append(widen(tail_v, tail_dtype))
        pr.append(np.ones(tail_k.shape[0], np.uint8))
        seg_id.append(np.full(tail_k.shape[0], n_segs, np.int32))
        n_segs += 1
    K = np.concatenate(ks)[None, None]
    V = np.concatenate(vs)[None, None]
    P = np.concatenate(pr)[None, None]
    o, lse, sl, smass = attend(widen(q, q_dtype)[None], K, V, P, np.concatenate(seg_id), n_segs,
                               sm_scale(w.D))
    return o[0], lse[0], sl[0], smass[0]


def denoise_chain(w, b: int, steps: List[int], rows: Optional[np.ndarray] = None,
                  bits_given: Optional[Dict[int, List[int]]] = None) -> Dict:
    """Oracle chain of a denoising workload with drifting latent keys and
    queries and per-head latent code widths (text-to-image), for batch
    element b and its Hkv KV heads.

    Timestep t: the latent keys and the query block take the random-walk
    step (t >= 1); the latent is attended dense until widths exist (t = 0,
    the first full-KV step), afterwards fake-quantised with the widths in
    force; at every rescore_every-th step the per-head latent mass of that
    step's attention (Eq. 1 bracket at head granularity) sets the widths for
    the following steps: all heads at 2 bits, raised to 4 bits in descending
    mass order within the batch element's storage budget.

    steps: timesteps whose attention is returned (rows: optional query rows
    of every query head, default all).  The masses of a rescoring step always
    cover all M query rows.  bits_given[t]: widths decided at step t to use
    instead of the oracle's own decision (then that step's masses are not
    computed).
    Returns {"bits": {t: widths}, "mass": {t: [Hkv] latent masses},
    "att": {t: (o, lse, seg_lse) per KV head}, "packed": {t: quantised latent
    per KV head (steps with widths in force)}}."""
    G, Hq, Hkv, D, M = w.group_size, w.Hq, w.Hkv, w.D, w.M
    lat = next(i for i, s in enumerate(w.segments) if s.policy == "quant")
    ls = w.segments[lat]
    N, Gq = ls.n, ls.group
    bh0 = b * Hkv
    seg_k = [None] * len(w.segments)
    seg_v = []
    for i, s in enumerate(w.segments):
        seg_v.append(gen.segment_kv(w, i, "v", bh0=bh0, nbh=Hkv))
        if i != lat:
            seg_k[i] = gen.segment_kv(w, i, "k", bh0=bh0, nbh=Hkv)
    lk, mk = gen.segment_kv(w, lat, "k", bh0=bh0, nbh=Hkv, master=True)
    dk = gen.Drift(w, gen.T_DRIFT_K, mk, ls.dtype, start=bh0 * N * D)
    q, mq = gen.queries(w, gen.T_QPRE, M, bh0=b * Hq, nbh=Hq, step=0, master=True)
    dq = gen.Drift(w, gen.T_DRIFT_Q, mq, w.q_dtype, start=b * Hq * M * D)
    orig = sum(dense_bytes(s.n, D, w.q_dtype) for s in w.segments)
    fixed = sum(dense_bytes(s.n, D, s.dtype) for i, s in enumerate(w.segments) if i != lat)
    budget_b, fixed_b = Hkv * orig / w.budget_ratio, Hkv * fixed
    seg_id = np.concatenate([np.full(s.n, i, np.int32) for i, s in enumerate(w.segments)])
    nseg = len(w.segments)
    sm = sm_scale(D)
    bits = None
    out = {"bits": {}, "mass": {}, "att": {}, "packed": {}}
    last = max(steps)
    for t in range(last + 1):
        if t > 0:
            lk = dk.step()
            q = dq.step()
        rescore = t % w.rescore_every == 0
        if not (t in steps or (rescore and (bits_given is None or t not in bits_given))):
            if rescore:
                bits = list(bits_given[t])
            continue
        need_mass = rescore and (bits_given is None or t not in bits_given)
        att, heads = [], []
        for h in range(Hkv):
            ks, vs = [], []
            for i, s in enumerate(w.segments):
                if i != lat:
                    ks.append(widen(seg_k[i][h], s.dtype))
                    vs.append(widen(seg_v[i][h], s.dtype))
                elif bits is None:
                    ks.append(widen(lk[h], s.dtype))
                    vs.append(widen(seg_v[i][h], s.dtype))
                else:
                    pk = quantize(lk[h][None], seg_v[i][h][None], s.dtype, Gq, [bits[h]])
                    if t in steps:
                        out["packed"].setdefault(t, []).append(pk)
                    kh, vh = dequant(pk, N, D, Gq, s.dtype)
                    ks.append(kh[0])
                    vs.append(vh[0])
            heads.append((np.concatenate(ks), np.concatenate(vs)))
            if t not in steps:
                continue
            K, V = heads[h][0][None, None], heads[h][1][None, None]
            qh = widen(q[h * G:(h + 1) * G], w.q_dtype)          # [G, M, D]
            if rows is not None:
                qh = qh[:, rows]
            o, lse, sl, _ = attend(qh[None], K, V, None, seg_id, nseg, sm)
            att.append((o[0], lse[0], sl[0]))
        if t in steps:
            out["att"][t] = att
        if rescore:
            if need_mass:
                # Eq. 1 bracket per KV head: probability on the latent rows,
                # summed over the head's G query heads and all M query rows
                # (one scorer call over every head of the batch element)
                Kall = np.stack([k for k, _ in heads])[None]    # [1, Hkv, N, D]
                _, ms = score64(widen(q, w.q_dtype)[None], Kall, seg_id, nseg, sm)
                mass = ms[0, :, lat]
                out["mass"][t] = np.asarray(mass, np.float64)
                bits = [int(x) for x in assign_bits(mass, N, D, Gq, ls.dtype, budget_b, fixed_b)]
            else:
                bits = list(bits_given[t])
            out["bits"][t] = list(bits)
    return out


def stored(x: np.ndarray, dtype: str) -> np.ndarray:
    """Values that are exactly representable in dtype -> their stored form
    (bf16 and fp16 as uint16 bits, fp32 as float32); checked by widening back."""
    x32 = np.ascontiguousarray(x, np.float64).astype(np.float32)
    if dtype == "bf16":
        out = (x32.view(np.uint32) >> 16).astype(np.uint16)
    elif dtype == "f16":
        out = x32.astype(np.float16).view(np.uint16)
    else:
        out = x32
    if not np.array_equal(widen(out, dtype), x):
        raise ValueError("values are not exactly representable in " + dtype)
    return out


def budget_chain(w, b: int, steps: List[int], rows: Optional[np.ndarray] = None,
                 given: Optional[Dict[int, Dict]] = None, first_masses: bool = False) -> Dict:
    """Oracle chain of the dynamic budget (Sec. 3.3 Eq. 1-3, Sec. 3.4) for one
    request (batch element b, its Hkv KV heads and Hq query heads) of a
    prefill workload with fresh queries per timestep.

    Candidate types are the eviction- and quantization-managed segments
    (kept segments are fixed).  Per request: S_a = Hkv x the dense bytes of
    type a's rows.
    t = 0, the full-KV step: attention over the uncompressed cache gives
      m^(0)_a = Mean over (query head, query row) of the probability on type
      a's rows (Eq. 1 with one step), M^(0) = sum over candidates; scores for
      eviction = column sums of the softmax over the whole context of the
      step's queries (all M rows of the G query heads of each KV head).
      rho^(1) = rho_init, B^(1) = rho^(1) sum_a S_a, b^(1) = Eq. 2 with
      b^(0) = S.
    Chunk c >= 1 = timesteps (c-1)C+1 .. cC.  Each step attends the cache as
      compressed so far and adds its Mean(h, q) type masses to the chunk
      average m^(c) (Eq. 1); after the chunk's last step (if a step follows):
      rho^(c+1) = Eq. 3, B^(c+1) = rho^(c+1) sum_a S_a, b^(c+1) = Eq. 2.
    Translation (Sec. 3.4), applied from the next step on:
      evicting type: k = min(k_prev, floor(b_a / Hkv / (2 D sizeof + 4)));
        fewer rows are chosen among the rows still kept by scores from the
        last obs_window query rows of each query head at the chunk's last
        step, the softmax running over the whole current cache (kept rows,
        dequantised rows); eviction is irreversible.
      quantised type: the most faithful (bits, group) at or after the current
        one whose Hkv segments fit b_a; a change re-quantises the current
        dequantised values (irreversible).

    steps: timesteps whose attention is returned.  rows: query rows to attend
    at those steps (then no masses are computed and every boundary's
    decisions must be given; with first_masses the full-KV step's masses and
    scores are still computed over all query rows, so boundary 0 records the
    oracle's own decision).  given[t]: decisions of boundary t to apply
    instead of the oracle's own: "k", "cfg" and optionally "keep" (kept
    positions per head); the oracle's own decision from the same state is
    still recorded (decisions[t]["own"]) when the masses are known.
    Returns {"decisions": {t: {...}}, "att": {t: (o, lse, seg_lse)},
    "keep": {t: kept positions per head}, "packed": {t: packed storage},
    "mass": {t: per-type Mean masses of step t}}."""
    G, Hq, Hkv, D, M = w.group_size, w.Hq, w.Hkv, w.D, w.M
    segs = w.segments
    nseg = len(segs)
    ev = next(i for i, s in enumerate(segs) if s.policy == "evict")
    qt = next(i for i, s in enumerate(segs) if s.policy == "quant")
    cand = [ev, qt]
    dt = segs[ev].dtype
    sm = sm_scale(D)
    ng = int(math.log2(D // 32)) + 1
    bh0 = b * Hkv
    seg_k = [gen.segment_kv(w, i, "k", bh0=bh0, nbh=Hkv) for i in range(nseg)]
    seg_v = [gen.segment_kv(w, i, "v", bh0=bh0, nbh=Hkv) for i in range(nseg)]
    S = {a: Hkv * dense_bytes(segs[a].n, D, segs[a].dtype) for a in cand}
    S_total = float(sum(S.values()))
    seg_id = np.concatenate([np.full(s.n, i, np.int32) for i, s in enumerate(segs)])
    ev0 = sum(s.n for s in segs[:ev])          # first logical row of the evicting type
    n_ev, n_qt = segs[ev].n, segs[qt].n
    state = {"keep": None, "cfg": None, "packed": None,
             "qk": widen(seg_k[qt], dt), "qv": widen(seg_v[qt], dt)}
    out = {"decisions": {}, "att": {}, "keep": {}, "packed": {}, "mass": {}}

    def logical():
        """K, V [Hkv, N, D] of the full logical sequence and the present mask."""
        ks = [state["qk"] if i == qt else widen(seg_k[i], s.dtype) for i, s in enumerate(segs)]
        vs = [state["qv"] if i == qt else widen(seg_v[i], s.dtype) for i, s in enumerate(segs)]
        present = np.ones((Hkv, seg_id.shape[0]), np.uint8)
        if state["keep"] is not None:
            present[:, ev0:ev0 + n_ev] = 0
            for h in range(Hkv):
                present[h, ev0 + state["keep"][h]] = 1
        return np.concatenate(ks, axis=1), np.concatenate(vs, axis=1), present

    def rescore(q_obs):
        """Scores of the evicting type's present rows, per head, from the
        softmax of q_obs over the present rows of the whole cache."""
        K, _, present = logical()
        if state["keep"] is None:  # every row present: one scorer call for all heads
            s64, _ = score64(widen(q_obs, w.q_dtype)[None], K[None], seg_id, nseg, sm)
            return [s64[0, h][seg_id == ev] for h in range(Hkv)]
        sc = []
        for h in range(Hkv):
            idx = np.nonzero(present[h])[0]
            s64, _ = score64(widen(q_obs[h * G:(h + 1) * G], w.q_dtype)[None],
                             K[h, idx][None, None], seg_id[idx], nseg, sm)
            sc.append(s64[0, 0][seg_id[idx] == ev])
        return sc

    def decide(t, m, b_prev, rho, q_obs, pre=None):
        """Boundary t: the oracle's own decision (when masses are known) and
        the decision applied (the given one, if any, else its own)."""
        g = given.get(t) if given else None
        k_prev = n_ev if state["keep"] is None else state["keep"][0].shape[0]
        rows_ev = ([np.arange(n_ev, dtype=np.int32)] * Hkv if state["keep"] is None
                   else state["keep"])
        rec = {"rho": rho, "B": rho * S_total}
        own = None
        bud = None
        if m is not None:
            bud = type_budget([m[a] for a in cand], [b_prev[a] for a in cand], rec["B"])
            bud = {a: float(x) for a, x in zip(cand, bud)}
            own = {"k": min(k_prev, evict_rows(bud[ev] / Hkv, 0.0, n_ev, D, dt)),
                   "cfg": quant_config(bud[qt], n_qt, D, dt, Hkv,
                                       0 if state["cfg"] is None else state["cfg"][0])[0]}
            rec.update(m={a: m[a] for a in cand}, b=bud)
        k_new = int(g["k"]) if g is not None else own["k"]
        cfg_new = int(g["cfg"]) if g is not None else own["cfg"]
        reselect = state["keep"] is None or k_new < k_prev
        if own is not None and (state["keep"] is None or own["k"] < k_prev):
            sc = pre if (pre is not None and state["keep"] is None) else rescore(q_obs)
            rec["scores"] = sc
            own["keep"] = [rows_ev[h][select(sc[h].astype(np.float32)[None], own["k"])[0]]
                           for h in range(Hkv)]
        if reselect:
            if g is not None and "keep" in g:
                state["keep"] = [np.asarray(x, np.int32) for x in g["keep"]]
            elif own is not None and own["k"] == k_new and "keep" in own:
                state["keep"] = own["keep"]
            else:
                sc = rescore(q_obs)
                rec["scores"] = sc
                state["keep"] = [rows_ev[h][select(sc[h].astype(np.float32)[None], k_new)[0]]
                                 for h in range(Hkv)]
        if state["cfg"] is None or cfg_new != state["cfg"][0]:
            bits, group = 8 >> (cfg_new // ng), 32 << (cfg_new % ng)
            pk = quantize(stored(state["qk"], dt), stored(state["qv"], dt), dt, group,
                          [bits] * Hkv)
            state["qk"], state["qv"] = dequant(pk, n_qt, D, group, dt)
            state["packed"], state["cfg"] = pk, (cfg_new, bits, group)
        rec.update(k=k_new, cfg=state["cfg"][0], bits=state["cfg"][1], group=state["cfg"][2],
                   own=own)
        out["decisions"][t] = rec
        out["keep"][t] = [x.copy() for x in state["keep"]]
        out["packed"][t] = state["packed"]
        return bud

    C = w.chunk_steps
    rho = w.rho_init
    b_prev = dict(S)
    acc = {a: 0.0 for a in range(nseg)}
    n_acc = 0
    M0 = None
    full = rows is None
    for t in range(w.steps):
        boundary = t == 0 or (t % C == 0 and t < w.steps - 1)
        if not (full or t in steps or boundary):
            continue
        q = gen.queries(w, gen.T_QPRE, M, bh0=b * Hq, nbh=Hq, step=t)  # [Hq, M, D]
        m_t = None
        pre = None
        if t == 0 and not full and first_masses:
            # the full-KV step over all M query rows: Eq. 1 masses and the
            # eviction scores from one scorer call over every head
            K, _, _ = logical()
            s64, ms = score64(widen(q, w.q_dtype)[None], K[None], seg_id, nseg, sm)
            m_t = {a: float(ms[0, :, a].sum()) / (Hq * M) for a in range(nseg)}
            out["mass"][0] = m_t
            pre = [s64[0, h][seg_id == ev] for h in range(Hkv)]
        if full or t in steps:
            K, V, present = logical()
            qa = q if full else q[:, rows]
            o, lse, sl, smass = attend(widen(qa, w.q_dtype)[None], K[None], V[None],
                                       present[None], seg_id, nseg, sm)
            if full:  # Eq. 1 bracket, Mean over the query heads and rows of this step
                m_t = {a: float(smass[0, :, :, a].sum()) / (Hq * M) for a in range(nseg)}
                out["mass"][t] = m_t
            if t in steps:
                out["att"][t] = (o[0], lse[0], sl[0])
        if t == 0:
            M0 = sum(m_t[a] for a in cand) if m_t is not None else None
            b_prev = decide(0, m_t, b_prev, rho, q, pre)
            continue
        if full:
            for a in range(nseg):
                acc[a] += m_t[a]
            n_acc += 1
        if boundary:
            if full:
                m_c = {a: acc[a] / n_acc for a in range(nseg)}
                rho = retention_next(rho, w.rho_init, w.rho_min, sum(m_c[a] for a in cand), M0)
            else:
                m_c = None
            b_prev = decide(t, m_c, b_prev, rho, q[:, M - w.obs_window:])
            acc = {a: 0.0 for a in range(nseg)}
            n_acc = 0
    return out


def realized_compression(w, decisions: Dict[int, Dict]) -> float:
    """Average KV compression a dynamic-budget run achieves (App. B,
    "Compression Ratio": the realized ratio recorded against the target):
    1 - the mean, over the timesteps that attend the compressed cache
    (t = 1 .. steps-1), of stored / original bytes of the cached segments.
    The state of timestep t is the decision of the last boundary before it.
    Cached segments are the kept, eviction- and quantisation-managed ones;
    protected segments (the current step's own tokens) are no part of the
    cache.  Bytes per (b, h_kv): kept rows dense, kept evicted rows plus an
    int32 index each, packed codes with float scales and minima and the
    residual tail."""
    D = w.D
    cached = [s for s in w.segments if s.policy != "protect"]
    orig = sum(dense_bytes(s.n, D, s.dtype) for s in cached)
    bounds = sorted(decisions)
    tot = 0.0
    for t in range(1, w.steps):
        d = decisions[max(b for b in bounds if b < t)]
        stored = 0
        for s in cached:
            if s.policy == "keep":
                stored += dense_bytes(s.n, D, s.dtype)
            elif s.policy == "evict":
                stored += d["k"] * (2 * D * ELEM[s.dtype] + 4)
            else:
                stored += packed_bytes(s.n, D, d["group"], d["bits"], s.dtype)
        tot += stored / orig
    return 1.0 - tot / (w.steps - 1)


def calibrate_rho_min(w, target: float, requests: Optional[List[int]] = None,
                      iters: int = 12) -> Dict:
    """App. B, "Calibration Setting": the minimum retention ratio rho_min that
    makes the average realized compression of the dynamic run (requests'
    mean) match the target.  The realized compression does not increase
    with rho_min (a higher floor keeps at least as many bytes at every
    boundary), so it is found by bisection on [0, rho_init]: a probe whose
    compression exceeds the target raises the lower end.  Returns the last
    probe and every probe's (rho_min, compression)."""
    import workloads as gen
    requests = [0] if requests is None else requests

    def f(x):
        wx = gen.scaled(w, rho_min=x)
        return sum(realized_compression(wx, budget_chain(wx, b, [])["decisions"])
                   for b in requests) / len(requests)

    lo, hi = 0.0, w.rho_init
    probes = []
    x = hi
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
