"""Pins of the oracle's dynamic budget (Sec. 3.3 Eq. 1-3, Sec. 3.4
translation) against hand-derived values and brute force.

The chain runs on a tiny editing-shaped workload; every decision it takes is
re-derived here from the definitions with numpy (softmax sums for Eq. 1,
Eq. 3 and the byte rules by hand, top-k by sorting, attention by an explicit
masked softmax), so a dropped term, a wrong index, a mask on the wrong rows or
a budget applied to the wrong type fails one of them.
"""
import json
import math
import os

import numpy as np
import pytest

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def test_quant_config_closed_forms(ref):
    with open(os.path.join(GOLD, "budget_closed_forms.json")) as f:
        gold = json.load(f)["quant_config"]
    for c in gold["cases"]:
        got = ref.quant_config(c["budget"], c["N"], c["D"], "bf16", c["heads"], c["first"])
        assert got == (c["index"], c["bits"], c["group"]), c
    # monotone: a larger budget never picks a less faithful configuration
    last = None
    for budget in np.linspace(0, 6e6, 301):
        i = ref.quant_config(float(budget), 4096, 128, "bf16", 4)[0]
        assert last is None or i <= last
        last = i
    with pytest.raises(ValueError):
        ref.quant_config(1e6, 4096, 96, "bf16", 4)  # D not a power of two


def _tiny(gen):
    S = gen.SegSpec
    return gen.Workload(
        name="tiny_dynamic", recipe_id=3, B=1, Hq=4, Hkv=2, D=64, q_dtype="bf16",
        segments=(S("text", 32, "keep", "bf16"), S("vit", 256, "evict", "bf16"),
                  S("vae", 256, "quant", "bf16", bits=None, group=None)),
        W=16, mode="prefill", steps=11, M=16, n_outlier=2, outlier_scale=8.0,
        chunk_steps=5, rho_init=0.30, rho_min=0.15, obs_window=4)


def _softmax_rows(q, K, sm):
    s = (q @ K.T) * sm
    s -= s.max(axis=-1, keepdims=True)
    e = np.exp(s)
    return e / e.sum(axis=-1, keepdims=True)


def _topk(score, k):
    order = sorted(range(len(score)), key=lambda j: (-np.float32(score[j]), j))
    return np.sort(np.asarray(order[:k], np.int64))


@pytest.fixture(scope="module")
def chain(ref, gen):
    import oracle.pipeline as op
    w = _tiny(gen)
    return w, op.budget_chain(w, 0, [0, 3, 6, 10])


def test_chain_masses_and_schedule(ref, gen, chain):
    w, r = chain
    cand = [1, 2]
    # Eq. 1 bracket per step: the type masses of a step are a distribution
    for t, m in r["mass"].items():
        assert abs(sum(m.values()) - 1.0) < 1e-12, t
    d0, d5 = r["decisions"][0], r["decisions"][5]
    assert sorted(r["decisions"]) == [0, 5]  # boundaries: the full-KV step and t = 5 (t = 10 is last)
    # Eq. 1 chunk average over steps 1..5, Eq. 3 by hand
    m_c = {a: sum(r["mass"][t][a] for t in range(1, 6)) / 5 for a in cand}
    M0 = sum(r["mass"][0][a] for a in cand)
    rho5 = min(w.rho_init, max(w.rho_min, w.rho_init * sum(m_c.values()) / M0))
    assert d0["rho"] == w.rho_init and abs(d5["rho"] - rho5) < 1e-15
    for a in cand:
        assert abs(d5["m"][a] - m_c[a]) < 1e-15 and abs(d0["m"][a] - r["mass"][0][a]) < 1e-15
    # Eq. 2: total within B, never above the previous allocation
    S = {a: w.Hkv * 2 * w.segments[a].n * w.D * 2 for a in cand}
    for d, prev in ((d0, S), (d5, d0["b"])):
        assert sum(d["b"].values()) <= d["B"] * (1 + 1e-12)
        assert all(d["b"][a] <= prev[a] * (1 + 1e-12) for a in cand)
        assert abs(d["B"] - d["rho"] * sum(S.values())) < 1e-6


def test_chain_translation_by_hand(ref, gen, chain):
    w, r = chain
    D, Hkv = w.D, w.Hkv
    n = 256
    per_row = 2 * D * 2 + 4
    cfgs = [(b, g) for b in (8, 4, 2) for g in (32, 64)]

    def bytes_of(bits, g):
        return 2 * n * D * bits // 8 + (n // g) * D * 8 + n * (D // g) * 8

    k_prev, c_prev = n, 0
    for t in (0, 5):
        d = r["decisions"][t]
        k = min(k_prev, min(n, int(math.floor(d["b"][1] / Hkv / per_row))))
        assert d["k"] == k and all(x.shape == (k,) for x in r["keep"][t])
        fit = [i for i in range(c_prev, len(cfgs)) if Hkv * bytes_of(*cfgs[i]) <= d["b"][2]]
        c = fit[0] if fit else len(cfgs) - 1
        assert d["cfg"] == c and (d["bits"], d["group"]) == cfgs[c]
        pk = r["packed"][t]
        assert list(pk["bits"]) == [cfgs[c][0]] * Hkv and pk["scale_k"].shape[1] == n // cfgs[c][1]
        k_prev, c_prev = k, c


def test_chain_selection_and_attention_brute_force(ref, gen, chain):
    w, r = chain
    import oracle.pipeline as op
    G, Hq, Hkv, D, M = w.group_size, w.Hq, w.Hkv, w.D, w.M
    sm = op.sm_scale(D)
    n_text, n_ev, n_q = 32, 256, 256
    ks = [ref.widen(gen.segment_kv(w, i, "k", bh0=0, nbh=Hkv), "bf16") for i in range(3)]
    vs = [ref.widen(gen.segment_kv(w, i, "v", bh0=0, nbh=Hkv), "bf16") for i in range(3)]

    def q_of(t):
        return ref.widen(gen.queries(w, gen.T_QPRE, M, bh0=0, nbh=Hq, step=t), "bf16")

    # t = 0: scores over the whole uncompressed context from all M rows of the
    # step's G query heads; the kept ViT rows are the top k of them
    q0 = q_of(0)
    for h in range(Hkv):
        K = np.concatenate([ks[0][h], ks[1][h], ks[2][h]])
        P = _softmax_rows(q0[h * G:(h + 1) * G].reshape(-1, D), K, sm)
        score = P.sum(axis=0)[n_text:n_text + n_ev]
        assert np.array_equal(r["keep"][0][h], _topk(score, r["decisions"][0]["k"])), h
    # t = 5: the new kept set is the top k of the rows kept before, scored by
    # the last obs_window rows of each query head over the current cache
    kh0, vh0 = ref.dequant(r["packed"][0], n_q, D, r["decisions"][0]["group"], "bf16")
    q5 = q_of(5)[:, M - w.obs_window:]
    for h in range(Hkv):
        kept = r["keep"][0][h]
        K = np.concatenate([ks[0][h], ks[1][h][kept], kh0[h]])
        P = _softmax_rows(q5[h * G:(h + 1) * G].reshape(-1, D), K, sm)
        score = P.sum(axis=0)[n_text:n_text + kept.shape[0]]
        sel = _topk(score, r["decisions"][5]["k"])
        assert np.array_equal(r["keep"][5][h], kept[sel]), h
        assert np.all(np.isin(r["keep"][5][h], kept))  # irreversible: nested
    # attention at t = 3 (state of boundary 0) and t = 6 (state of boundary 5)
    for t, tb in ((3, 0), (6, 5)):
        kh, vh = ref.dequant(r["packed"][tb], n_q, D, r["decisions"][tb]["group"], "bf16")
        q = q_of(t)
        o_ref = r["att"][t][0]
        for hq in range(Hq):
            h = hq // G
            kept = r["keep"][tb][h]
            K = np.concatenate([ks[0][h], ks[1][h][kept], kh[h]])
            V = np.concatenate([vs[0][h], vs[1][h][kept], vh[h]])
            P = _softmax_rows(q[hq], K, sm)
            assert np.allclose(o_ref[hq], P @ V, rtol=1e-12, atol=1e-13), (t, hq)
    # re-quantisation at a configuration change starts from the dequantised values
    if r["decisions"][5]["cfg"] != r["decisions"][0]["cfg"]:
        pk = ref.quantize(op.stored(kh0, "bf16"), op.stored(vh0, "bf16"), "bf16",
                          r["decisions"][5]["group"], [r["decisions"][5]["bits"]] * Hkv)
        for name in ("codes_k", "codes_v", "scale_k", "min_k", "scale_v", "min_v"):
            assert np.array_equal(pk[name], r["packed"][5][name]), name


def test_stored_round_trip(ref):
    import oracle.pipeline as op
    x = ref.widen(np.arange(0, 65536, 97, dtype=np.uint16), "bf16")
    x = x[np.isfinite(x)]
    assert np.array_equal(ref.widen(op.stored(x, "bf16"), "bf16"), x)
    with pytest.raises(ValueError):
        op.stored(np.array([1.0 + 2.0 ** -12]), "bf16")


def test_chain_forced_requantisation(ref, gen, chain):
    """A boundary decision that narrows the quantised type (given, as for a
    run whose decisions come from elsewhere): the new storage is the old
    dequantised values quantised with the new (bits, group), and the next
    step attends exactly those values."""
    import oracle.pipeline as op
    w, r0 = chain
    D, Hkv, G, M = w.D, w.Hkv, w.group_size, w.M
    c5 = r0["decisions"][5]["cfg"] + 1          # one step less faithful
    r = op.budget_chain(w, 0, [6], given={5: {"k": r0["decisions"][5]["k"], "cfg": c5}})
    d = r["decisions"][5]
    assert d["cfg"] == c5 and (d["bits"], d["group"]) == (8 >> (c5 // 2), 32 << (c5 % 2))
    kh0, vh0 = ref.dequant(r["packed"][0], 256, D, r["decisions"][0]["group"], "bf16")
    pk = ref.quantize(op.stored(kh0, "bf16"), op.stored(vh0, "bf16"), "bf16", d["group"],
                      [d["bits"]] * Hkv)
    for name in ("codes_k", "codes_v", "scale_k", "min_k", "scale_v", "min_v"):
        assert np.array_equal(pk[name], r["packed"][5][name]), name
    kh, vh = ref.dequant(pk, 256, D, d["group"], "bf16")
    q = ref.widen(gen.queries(w, gen.T_QPRE, M, bh0=0, nbh=w.Hq, step=6), "bf16")
    ks = [ref.widen(gen.segment_kv(w, i, "k", bh0=0, nbh=Hkv), "bf16") for i in range(2)]
    vs = [ref.widen(gen.segment_kv(w, i, "v", bh0=0, nbh=Hkv), "bf16") for i in range(2)]
    for hq in range(w.Hq):
        h = hq // G
        kept = r["keep"][5][h]
        K = np.concatenate([ks[0][h], ks[1][h][kept], kh[h]])
        V = np.concatenate([vs[0][h], vs[1][h][kept], vh[h]])
        P = _softmax_rows(q[hq], K, op.sm_scale(D))
        assert np.allclose(r["att"][6][0][hq], P @ V, rtol=1e-12, atol=1e-13), hq


def test_topk_mass_closed_forms_and_brute_force(ref):
    """Sec. 3.2 / App. B concentration statistic."""
    assert np.allclose(ref.topk_mass(np.ones((3, 50), np.float32), 5), 0.1, rtol=0, atol=1e-15)
    s = np.full((1, 100), 1e-3, np.float32)
    s[0, 37] = 10.0
    exp = (10.0 + 9 * np.float64(np.float32(1e-3))) / (10.0 + 99 * np.float64(np.float32(1e-3)))
    assert abs(ref.topk_mass(s, 10)[0] - exp) < 1e-12
    rng = np.random.default_rng(3)
    x = rng.integers(0, 5, (4, 333)).astype(np.float32)  # ties on purpose
    for k in (0, 1, 34, 333):
        got = ref.topk_mass(x, k)
        for r in range(4):
            srt = np.sort(x[r].astype(np.float64))[::-1]
            want = srt[:k].sum() / srt.sum() if srt.sum() > 0 else 0.0
            assert abs(got[r] - want) < 1e-12, (k, r)
    assert np.all(ref.topk_mass(np.zeros((2, 10), np.float32), 3) == 0.0)
    with pytest.raises(ValueError):
        ref.topk_mass(x, 334)


def test_chain_first_masses_with_sampled_rows(ref, gen, chain):
    """The sampled-row mode with first_masses (used at full size): the
    full-KV step's masses, the oracle's own first decision and its kept rows
    equal those of the chain that attends every row."""
    import oracle.pipeline as op
    w, r = chain
    given = {t: {"k": d["k"], "cfg": d["cfg"], "keep": r["keep"][t]}
             for t, d in r["decisions"].items()}
    rs = op.budget_chain(w, 0, [3], rows=np.array([0, 5, 9]), given=given, first_masses=True)
    for a in range(3):
        assert abs(rs["mass"][0][a] - r["mass"][0][a]) < 1e-14, a
    own, d0 = rs["decisions"][0]["own"], r["decisions"][0]
    assert (own["k"], own["cfg"]) == (d0["k"], d0["cfg"])
    for h in range(w.Hkv):
        assert np.array_equal(own["keep"][h], r["keep"][0][h]), h
    assert rs["decisions"][5]["own"] is None  # later boundaries: given only
