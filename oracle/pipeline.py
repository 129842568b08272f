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

from . import (assign_bits, attend, dense_bytes, dequant, evict_rows, packed_bytes, quantize,
               score64, select, widen)


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
    of every query head, default all).  bits_given[t]: widths decided at step
    t to use instead of the oracle's own decision (for runs where only sampled
    rows can be attended and the full masses are not computed).
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
        att, mass = [], []
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
            K = np.concatenate(ks)[None, None]
            V = np.concatenate(vs)[None, None]
            qh = widen(q[h * G:(h + 1) * G], w.q_dtype)          # [G, M, D]
            if need_mass or rows is None:
                o, lse, sl, smass = attend(qh[None], K, V, None, seg_id, nseg, sm)
                mass.append(float(smass[0, :, :, lat].sum()))  # over the G heads and M rows
                if rows is not None:
                    o, lse, sl = o[:, :, rows], lse[:, :, rows], sl[:, :, rows]
            else:
                o, lse, sl, _ = attend(qh[:, rows][None], K, V, None, seg_id, nseg, sm)
            att.append((o[0], lse[0], sl[0]))
        if t in steps:
            out["att"][t] = att
        if rescore:
            if need_mass:
                out["mass"][t] = np.asarray(mass, np.float64)
                bits = [int(x) for x in assign_bits(mass, N, D, Gq, ls.dtype, budget_b, fixed_b)]
            else:
                bits = list(bits_given[t])
            out["bits"][t] = list(bits)
    return out
