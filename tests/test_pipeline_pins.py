"""Pins of the oracle's per-workload pipeline (``oracle/pipeline.py``):
``plan`` (storage budget -> rows kept / code width per segment, Sec. 3.4 with
the byte accounting of Sec. 3.3 and App. E) and ``denoise_chain`` (the
text-to-image chain: drifting latent keys and queries, per-head int2/int4
widths from the latent attention mass of a rescoring step, Sec. 3.3 Eq. 1
bracket at head granularity).

``plan`` is checked against the hand-derived values of
``tests/golden/budget_closed_forms.json`` and, on shapes of its own, against a
brute-force search over the row count that sums the byte sizes of the arrays
the stored segment really consists of.  ``denoise_chain`` runs on a tiny
drifting workload whose widths change at every rescoring step; every mass,
width and output is re-derived here with numpy (explicit softmax, the greedy
rule written out, quantisation by the separately pinned oracle quantizer), so
a dropped term, a width applied one step early, keys quantised only at the
rescoring steps or a mass summed over the wrong query heads fails a test.
"""
import json
import math
import os

import numpy as np
import pytest

GOLD = os.path.join(os.path.dirname(__file__), "golden")
ELEM = {"f32": 4, "f16": 2, "bf16": 2}
NP = {"f32": np.float32, "f16": np.float16, "bf16": np.uint16}


# ---------------------------------------------------------------- plan

def _stored_bytes(w, pols, ref):
    """Stored bytes of one (b, h_kv) after the plan, as the nbytes of the
    arrays that hold it: dense rows, kept rows plus int32 indices, and the
    quantizer's real outputs (codes, float scales/minima, residual tail)."""
    tot = 0
    for s, p in zip(w.segments, pols):
        row = np.zeros((1, w.D), NP[s.dtype]).nbytes
        if p["kind"] == "keep":
            tot += 2 * s.n * row
        elif p["kind"] == "evict":
            tot += 2 * p["k"] * row + np.zeros(p["k"], np.int32).nbytes
        else:
            x = np.zeros((1, s.n, w.D), NP[s.dtype])
            pk = ref.quantize(x, x, s.dtype, p["group"], [p["bits"]])
            tot += sum(pk[n].nbytes for n in ("codes_k", "codes_v", "scale_k", "min_k",
                                                "scale_v", "min_v", "tail_k", "tail_v"))
    return tot


def test_plan_closed_forms(ref, gen):
    import oracle.pipeline as op
    with open(os.path.join(GOLD, "budget_closed_forms.json")) as f:
        gold = json.load(f)["accounting"]
    for w in (gen.TINY_UNDERSTANDING, gen.UNDERSTANDING_7B, gen.IMAGE_EDITING,
              gen.TEXT_TO_IMAGE, gen.LONG_CONTEXT_64K):
        g = gold[w.name]
        pols = op.plan(w)
        assert [p["kind"] for p in pols] == [
            "evict" if s.policy == "evict" else s.policy for s in w.segments], w.name
        ks = [p["k"] for p in pols if p["kind"] == "evict"]
        if "k" in g:
            assert ks == [g["k"]], w.name
            assert _stored_bytes(w, pols, ref) == g["stored"], w.name
        else:
            # text-to-image: the latent width is per head, decided by mass
            # (pinned below on the chain); the plan leaves it open
            assert ks == [] and pols[1] == {"kind": "quant", "bits": None, "group": 64}
        for s, p in zip(w.segments, pols):
            if p["kind"] == "quant" and s.bits:
                assert (p["bits"], p["group"]) == (s.bits, s.group), w.name


def _brute_k(w, pols, ref, i):
    """Largest k whose stored bytes fit the budget, by trying every k."""
    orig = sum(2 * s.n * np.zeros((1, w.D), NP[w.q_dtype]).nbytes for s in w.segments)
    budget = orig / w.budget_ratio
    best = 0
    for k in range(w.segments[i].n + 1):
        trial = [dict(p) for p in pols]
        trial[i]["k"] = k
        if _stored_bytes(w, trial, ref) <= budget:
            best = k
    return best


@pytest.mark.parametrize("case", range(6))
def test_plan_budget_brute_force(ref, gen, case):
    """Budget-derived row counts on shapes of their own: the plan keeps the
    largest k for which every stored byte (other segments, kept rows, indices,
    scales and minima) fits orig / ratio, counting orig at the I/O type."""
    import oracle.pipeline as op
    rng = np.random.default_rng(100 + case)
    S = gen.SegSpec
    D = int(rng.choice([64, 128]))
    dt = str(rng.choice(["bf16", "f32"]))
    n_keep, n_ev, n_q = (int(x) for x in rng.integers(8, 200, 3))
    g = int(rng.choice([32, 64]))
    n_q = max(n_q, g)
    segs = [S("text", n_keep, "keep", "f16" if dt == "f32" else dt),
            S("vit", n_ev, "evict", dt),
            S("vae", n_q, "quant", dt, bits=int(rng.choice([2, 4, 8])), group=g)]
    order = rng.permutation(3)
    segs = tuple(segs[j] for j in order)
    ratio = float(rng.uniform(1.5, 6.0))
    w = gen.Workload(name="plan_case", recipe_id=9, B=1, Hq=2, Hkv=1, D=D, q_dtype=dt,
                     segments=segs, W=1, mode="decode", steps=1, M=1, budget_ratio=ratio)
    pols = op.plan(w)
    i = next(j for j, s in enumerate(segs) if s.policy == "evict")
    assert pols[i]["k"] == _brute_k(w, pols, ref, i), (case, pols)


# ---------------------------------------------------------------- denoise_chain

def _tiny_denoise(gen):
    """Three KV heads of two query heads each, a kept text segment and a
    128-row latent quantised per head at 2 or 4 bits (group 32), a budget
    ratio that admits exactly two 4-bit heads, drift sigma 0.05 and
    rescoring every 5 timesteps."""
    S = gen.SegSpec
    return gen.Workload(
        name="tiny_denoise", recipe_id=4, B=1, Hq=6, Hkv=3, D=64, q_dtype="bf16",
        segments=(S("text", 32, "keep", "bf16"),
                  S("latent", 128, "quant", "bf16", bits=None, group=32)),
        W=8, mode="prefill", steps=12, M=8, budget_ratio=2.1, n_outlier=2,
        outlier_scale=8.0, drift_sigma=0.05, rescore_every=5)


STEPS = [0, 1, 4, 5, 6, 10, 11]


@pytest.fixture(scope="module")
def dchain(gen):
    import oracle.pipeline as op
    w = _tiny_denoise(gen)
    return w, op.denoise_chain(w, 0, STEPS)


def _drifted(w, gen, T):
    """Latent keys [Hkv, N, D] and queries [Hq, M, D] (stored bf16) of every
    timestep 0..T, from the shared generator's random walk."""
    lat = 1
    N, D = w.segments[lat].n, w.D
    lk, mk = gen.segment_kv(w, lat, "k", bh0=0, nbh=w.Hkv, master=True)
    q, mq = gen.queries(w, gen.T_QPRE, w.M, bh0=0, nbh=w.Hq, step=0, master=True)
    dk = gen.Drift(w, gen.T_DRIFT_K, mk, "bf16", start=0)
    dq = gen.Drift(w, gen.T_DRIFT_Q, mq, "bf16", start=0)
    ks, qs = [lk], [q]
    for _ in range(T):
        ks.append(dk.step())
        qs.append(dq.step())
    assert ks[0].shape == (w.Hkv, N, D)
    return ks, qs


def _in_force(bits, t):
    """Widths decided at the last rescoring step strictly before t."""
    prev = [s for s in sorted(bits) if s < t]
    return None if not prev else bits[prev[-1]]


def _softmax_stats(q, K, V, seg_id, nseg, sm):
    """Explicit fp64 softmax over all rows: o, lse, per-segment lse, per-segment
    probability sums, for q [M, D]."""
    s = (q @ K.T) * sm
    m = s.max(axis=1, keepdims=True)
    e = np.exp(s - m)
    Z = e.sum(axis=1, keepdims=True)
    P = e / Z
    o = P @ V
    lse = (m + np.log(Z))[:, 0]
    seg = np.stack([m[:, 0] + np.log(e[:, seg_id == a].sum(axis=1)) for a in range(nseg)], 1)
    mass = np.stack([P[:, seg_id == a].sum(axis=1) for a in range(nseg)], 1)
    return o, lse, seg, mass


def _logical(w, ref, gen, lk_t, bits):
    """Per KV head, the K, V rows attention sees: text as stored, the latent
    dense (no widths yet) or quantised at its head's width and dequantised."""
    lat, D = 1, w.D
    N, G = w.segments[lat].n, w.segments[lat].group
    tk = ref.widen(gen.segment_kv(w, 0, "k", bh0=0, nbh=w.Hkv), "bf16")
    tv = ref.widen(gen.segment_kv(w, 0, "v", bh0=0, nbh=w.Hkv), "bf16")
    lv = gen.segment_kv(w, lat, "v", bh0=0, nbh=w.Hkv)
    out = []
    for h in range(w.Hkv):
        if bits is None:
            kh, vh = ref.widen(lk_t[h], "bf16"), ref.widen(lv[h], "bf16")
        else:
            pk = ref.quantize(lk_t[h][None], lv[h][None], "bf16", G, [bits[h]])
            kh, vh = ref.dequant(pk, N, D, G, "bf16")
            kh, vh = kh[0], vh[0]
        out.append((np.concatenate([tk[h], kh]), np.concatenate([tv[h], vh])))
    return out


def test_denoise_widths_change(dchain):
    """The fixture is meaningful: the widths differ between consecutive
    rescoring steps (so applying them a step early changes the outputs)."""
    w, r = dchain
    assert sorted(r["bits"]) == [0, 5, 10]
    assert r["bits"][0] != r["bits"][5] and r["bits"][5] != r["bits"][10]


def test_denoise_masses_brute_force(ref, gen, dchain):
    """Eq. 1 bracket at head granularity: the latent mass of KV head h at a
    rescoring step is the probability on the latent rows summed over that
    head's own query heads h*G .. h*G+G-1 and the M query rows, with the
    softmax over the whole cache as attended at that step."""
    import oracle.pipeline as op
    w, r = dchain
    G, D, M = w.group_size, w.D, w.M
    ks, qs = _drifted(w, gen, 10)
    seg_id = np.concatenate([np.zeros(32, np.int32), np.ones(128, np.int32)])
    for t in (0, 5, 10):
        heads = _logical(w, ref, gen, ks[t], _in_force(r["bits"], t))
        q = ref.widen(qs[t], "bf16")
        for h in range(w.Hkv):
            K, V = heads[h]
            mass = sum(_softmax_stats(q[hq], K, V, seg_id, 2, op.sm_scale(D))[3][:, 1].sum()
                       for hq in range(h * G, (h + 1) * G))
            assert abs(r["mass"][t][h] - mass) <= 1e-12 * M * G, (t, h)
        # the masses decide: no two heads tie within the comparison band
        m = np.sort(r["mass"][t])
        assert np.all(np.diff(m) > 1e-6 * m[-1]), t


def test_denoise_widths_greedy_by_hand(ref, gen, dchain):
    """Per-head widths of the batch element: every head at 2 bits, heads raised
    to 4 bits in descending latent-mass order while the stored bytes (the
    kept text plus each head's packed latent, as the nbytes of the quantizer's
    arrays) stay within Hkv x orig / ratio."""
    w, r = dchain
    D, N, G = w.D, w.segments[1].n, w.segments[1].group
    x = np.zeros((1, N, D), np.uint16)

    def head_bytes(b):
        pk = ref.quantize(x, x, "bf16", G, [b])
        return sum(pk[n].nbytes for n in ("codes_k", "codes_v", "scale_k", "min_k",
                                            "scale_v", "min_v", "tail_k", "tail_v"))

    orig = w.Hkv * sum(2 * s.n * D * 2 for s in w.segments)
    budget = orig / w.budget_ratio
    fixed = w.Hkv * 2 * 32 * D * 2
    for t, bits in r["bits"].items():
        mass = r["mass"][t]
        order = sorted(range(w.Hkv), key=lambda h: (-mass[h], h))
        want = [2] * w.Hkv
        for h in order:
            trial = list(want)
            trial[h] = 4
            if fixed + sum(head_bytes(b) for b in trial) <= budget:
                want = trial
            else:
                break
        assert bits == want, (t, bits, want)
        assert sorted(bits) == [2, 4, 4], t  # the ratio admits exactly two upgrades


def test_denoise_attention_brute_force(ref, gen, dchain):
    """Every returned timestep attends the latent keys drifted to that step,
    re-quantised with the widths of the last rescoring step before it (dense
    at t = 0), and the stored codes are those of that quantisation."""
    import oracle.pipeline as op
    w, r = dchain
    G, D = w.group_size, w.D
    N, Gq = w.segments[1].n, w.segments[1].group
    ks, qs = _drifted(w, gen, max(STEPS))
    lv = gen.segment_kv(w, 1, "v", bh0=0, nbh=w.Hkv)
    seg_id = np.concatenate([np.zeros(32, np.int32), np.ones(128, np.int32)])
    for t in STEPS:
        bits = _in_force(r["bits"], t)
        heads = _logical(w, ref, gen, ks[t], bits)
        q = ref.widen(qs[t], "bf16")
        for h in range(w.Hkv):
            K, V = heads[h]
            o_ref, lse_ref, sl_ref = r["att"][t][h]
            for g in range(G):
                o, lse, sl, _ = _softmax_stats(q[h * G + g], K, V, seg_id, 2, op.sm_scale(D))
                assert np.allclose(o_ref[g], o, rtol=1e-12, atol=1e-13), (t, h, g)
                assert np.allclose(lse_ref[g], lse, rtol=1e-13, atol=1e-13), (t, h, g)
                assert np.allclose(sl_ref[g], sl, rtol=1e-13, atol=1e-13), (t, h, g)
            if bits is not None:
                pk = ref.quantize(ks[t][h][None], lv[h][None], "bf16", Gq, [bits[h]])
                got = r["packed"][t][h]
                for name in ("codes_k", "codes_v", "scale_k", "min_k", "scale_v", "min_v"):
                    assert np.array_equal(got[name], pk[name]), (t, h, name)
    # the keys really drift: consecutive steps' latent keys differ
    assert not np.array_equal(ks[4], ks[5])


def test_denoise_sampled_rows_and_given_widths(ref, gen, dchain):
    """The modes the full-size GPU runs use: attention on sampled query rows
    equals the full chain's rows, and widths given from outside replace the
    chain's own decisions from that step on."""
    import oracle.pipeline as op
    w, r = dchain
    rows = np.array([0, 3, 7])
    rs = op.denoise_chain(w, 0, [6, 11], rows=rows, bits_given=r["bits"])
    for t in (6, 11):
        for h in range(w.Hkv):
            for a, b in zip(rs["att"][t][h], r["att"][t][h]):
                assert np.array_equal(a, b[:, rows]), (t, h)
    forced = {0: [2, 4, 4], 5: [4, 4, 2], 10: [4, 2, 4]}
    rf = op.denoise_chain(w, 0, [6], bits_given=forced)
    assert rf["mass"] == {}  # no masses are computed when every width is given
    ks, qs = _drifted(w, gen, 6)
    heads = _logical(w, ref, gen, ks[6], forced[5])
    q = ref.widen(qs[6], "bf16")
    seg_id = np.concatenate([np.zeros(32, np.int32), np.ones(128, np.int32)])
    for h in range(w.Hkv):
        o, _, _, _ = _softmax_stats(q[h * w.group_size], *heads[h], seg_id, 2,
                                    op.sm_scale(w.D))
        assert np.allclose(rf["att"][6][h][0][0], o, rtol=1e-12, atol=1e-13), h


def test_text_to_image_budget_admits_three_upgrades(ref, gen):
    """Full text-to-image shapes: the greedy rule under the 2.5x budget gives
    three 4-bit heads and one 2-bit head per batch element whatever the mass
    order (golden closed form), the 2-bit head being the least massive."""
    with open(os.path.join(GOLD, "budget_closed_forms.json")) as f:
        g = json.load(f)["accounting"]["text_to_image"]
    w = gen.TEXT_TO_IMAGE
    D, N = w.D, 4096
    orig = w.Hkv * sum(2 * s.n * D * 2 for s in w.segments)
    fixed = w.Hkv * 2 * 768 * D * 2
    rng = np.random.default_rng(7)
    for _ in range(5):
        mass = rng.uniform(0.5, 2.0, w.Hkv)
        bits = [int(b) for b in ref.assign_bits(list(mass), N, D, 64, "bf16",
                                                orig / w.budget_ratio, fixed)]
        assert bits.count(4) == g["n_int4"] and bits.count(2) == g["n_int2"]
        assert bits[int(np.argmin(mass))] == 2


def test_denoise_masses_without_attention(dchain):
    """Rescoring steps that return no attention still compute their masses
    over all query rows (the path the full-size runs take): the widths and
    masses equal those of the chain that also attends those steps."""
    import oracle.pipeline as op
    w, r = dchain
    rs = op.denoise_chain(w, 0, [11], rows=np.array([1, 6]))
    assert rs["bits"] == r["bits"]
    for t in r["mass"]:
        assert np.array_equal(rs["mass"][t], r["mass"][t]), t
    assert sorted(rs["att"]) == [11]
