"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each test checks the oracle against something other than itself: library
routines (numpy/scipy/torch conversions and softmax), closed forms, invariants
and brute force on tiny inputs, chosen so that a dropped term, a wrong sign or
index or a transposed operand fails at least one of them.
"""
import json
import math
import os

import numpy as np
import pytest
import scipy.special as sps
import torch

GOLD = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------- dtypes

def test_widen_matches_library_conversions(ref):
    rng = np.random.default_rng(1)
    x = (rng.standard_normal(20000) * np.exp(rng.uniform(-30, 30, 20000))).astype(np.float32)
    with np.errstate(over="ignore"):
        h = x.astype(np.float16)  # numpy: binary32 -> binary16 round-to-nearest-even
    assert np.array_equal(ref.widen(h, "f16"), h.astype(np.float64), equal_nan=True)
    b = torch.from_numpy(x).to(torch.bfloat16)
    bits = b.view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ref.widen(bits, "bf16"), b.to(torch.float64).numpy(), equal_nan=True)
    assert np.array_equal(ref.widen(x, "f32"), x.astype(np.float64))


def test_round_value_matches_library_conversions(ref):
    rng = np.random.default_rng(2)
    x = (rng.standard_normal(50000) * np.exp(rng.uniform(-25, 14, 50000))).astype(np.float32)
    # include exact halfway cases and subnormal fp16 inputs
    x = np.concatenate([x, np.float32([65504, 65519.99, 65520, 6e-8, 3e-8, 2.98e-8,
                                       1 + 2 ** -11, 1 + 3 * 2 ** -11, 1 + 2 ** -8,
                                       1 + 3 * 2 ** -8, -0.0, 0.0])])
    with np.errstate(over="ignore"):
        want16 = x.astype(np.float16).astype(np.float64)
    assert np.array_equal(ref.round_value(x, "f16"), want16)
    want_bf = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(ref.round_value(x, "bf16"), want_bf)
    assert np.array_equal(ref.round_value(x, "f32"), x.astype(np.float64))


# ---------------------------------------------------------------- quantizer

def _unpack(codes, off, rows, D, b):
    """Brute-force unpack of one head's codes per the layout (LSB first)."""
    out = np.zeros((rows, D), np.int64)
    rb = D * b // 8
    for r in range(rows):
        for c in range(D):
            byte = codes[off + r * rb + (c * b) // 8]
            out[r, c] = (int(byte) >> ((c % (8 // b)) * b)) & ((1 << b) - 1)
    return out


@pytest.mark.parametrize("b", [2, 4, 8])
def test_quant_ramp_gives_code_index(ref, b):
    """A ramp x_i = mn + i*s over a key channel (and a value group) maps code i
    with scale s and minimum mn (Sec. App. E storage; asymmetric min/max)."""
    G, D = 16, 16
    levels = (1 << b) - 1
    s = 0.25
    mn = -1.0
    idx = np.arange(G) % (levels + 1)
    idx[-1] = levels  # make the maximum reach the top code
    k = np.zeros((1, G, D), np.float32)
    for c in range(D):
        k[0, :, c] = mn + idx * s
    v = np.tile((mn + np.resize(idx, D) * s).astype(np.float32), (1, G, 1))
    v[0, :, D - 1] = mn + levels * s
    v[0, :, 0] = mn
    pk = ref.quantize(k, v, "f32", G, [b])
    ck = _unpack(pk["codes_k"], 0, G, D, b)
    assert np.array_equal(ck, np.tile(idx[:, None], (1, D)))
    assert np.all(pk["scale_k"] == np.float32(s)) and np.all(pk["min_k"] == np.float32(mn))
    cv = _unpack(pk["codes_v"], 0, G, D, b)
    assert np.all(cv.min(axis=1) == 0) and np.all(cv.max(axis=1) == levels)


def test_quant_constant_group(ref):
    k = np.full((1, 32, 32), 1.5, np.float32)
    v = np.full((1, 32, 32), -2.25, np.float32)
    pk = ref.quantize(k, v, "f32", 32, [4])
    assert not pk["codes_k"].any() and not pk["codes_v"].any()
    assert np.all(pk["scale_k"] == 0) and np.all(pk["min_k"] == 1.5)
    kh, vh = ref.dequant(pk, 32, 32, 32, "f32")
    assert np.all(kh == 1.5) and np.all(vh == -2.25)


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("b", [2, 4, 8])
def test_quant_error_bound_and_code_range(ref, gen, dtype, b):
    """|x - fmaf(code, s, mn)| <= s/2 (+ a few ulp); min -> 0, max -> 2^b-1;
    the dequantised value is that fmaf rounded to the segment dtype."""
    G, N, D, BH = 32, 100, 64, 3
    x64 = gen.normal(gen.stream(7, b, 1), 0, BH * N * D).reshape(BH, N, D) * 3
    y64 = gen.normal(gen.stream(7, b, 2), 0, BH * N * D).reshape(BH, N, D)
    k = gen.round_to(x64, dtype)
    v = gen.round_to(y64, dtype)
    pk = ref.quantize(k, v, dtype, G, [b] * BH)
    kw, vw = ref.widen(k, dtype), ref.widen(v, dtype)
    n_full = G * (N // G)
    for bh in range(BH):
        off = int(pk["code_off"][bh])
        ck = _unpack(pk["codes_k"], off, n_full, D, b)
        cv = _unpack(pk["codes_v"], off, n_full, D, b)
        assert ck.min() >= 0 and ck.max() <= (1 << b) - 1
        sk = np.repeat(pk["scale_k"][bh], G, axis=0)
        mk = np.repeat(pk["min_k"][bh], G, axis=0)
        xk = kw[bh, :n_full]
        # group minima / maxima are exact, and map to codes 0 / 2^b-1
        gk = xk.reshape(n_full // G, G, D)
        assert np.array_equal(pk["min_k"][bh], gk.min(axis=1).astype(np.float32))
        assert np.all(ck.reshape(n_full // G, G, D)[gk == gk.min(axis=1, keepdims=True)] == 0)
        assert np.all(ck.reshape(n_full // G, G, D)[gk == gk.max(axis=1, keepdims=True)] == (1 << b) - 1)
        fm = np.float32(ck) * sk.astype(np.float64) + mk  # exact in double
        fmaf = fm.astype(np.float32)  # one rounding = fmaf
        # (x - mn) / s is rounded in binary32 before rint, so the bound carries
        # a few ulp of the group's magnitude max(|x|, |mn|, |mx|)
        mag = np.repeat(np.abs(gk).max(axis=1), G, axis=0)
        ulp = np.spacing(mag.astype(np.float32)).astype(np.float64)
        assert np.all(np.abs(xk - fmaf) <= sk / 2 + 2 * ulp)
        sv = np.repeat(pk["scale_v"][bh], G, axis=1)
        mv = np.repeat(pk["min_v"][bh], G, axis=1)
        fmv = (np.float32(cv) * sv.astype(np.float64) + mv).astype(np.float32)
        xv = vw[bh, :n_full]
        magv = np.repeat(np.abs(xv).reshape(n_full, D // G, G).max(axis=2), G, axis=1)
        ulpv = np.spacing(magv.astype(np.float32)).astype(np.float64)
        assert np.all(np.abs(xv - fmv) <= sv / 2 + 2 * ulpv)
        kh, vh = ref.dequant(pk, N, D, G, dtype)
        assert np.array_equal(kh[bh, :n_full], ref.round_value(fmaf, dtype))
        assert np.array_equal(vh[bh, :n_full], ref.round_value(fmv, dtype))
        # residual tail: stored bytes, unchanged
        assert np.array_equal(pk["tail_k"][bh], k[bh, n_full:])
        assert np.array_equal(kh[bh, n_full:], kw[bh, n_full:])
        assert np.array_equal(vh[bh, n_full:], vw[bh, n_full:])


def test_quant_codes_brute_force(ref, gen):
    """Codes re-derived element by element with numpy binary32 arithmetic and
    packed per the stated layout."""
    G, N, D, b = 8, 19, 16, 4
    k = gen.round_to(gen.normal(99, 0, N * D).reshape(1, N, D) * 2, "bf16")
    v = gen.round_to(gen.normal(98, 0, N * D).reshape(1, N, D), "bf16")
    pk = ref.quantize(k, v, "bf16", G, [b])
    kw = ref.widen(k, "bf16").astype(np.float32)[0]
    vw = ref.widen(v, "bf16").astype(np.float32)[0]
    n_full = 16
    qmax = np.float32(15)
    want_k = np.zeros((n_full, D), np.int64)
    for g in range(n_full // G):
        blk = kw[g * G:(g + 1) * G]
        mn, mx = blk.min(axis=0), blk.max(axis=0)
        s = (mx - mn) / qmax
        for r in range(G):
            for c in range(D):
                want_k[g * G + r, c] = 0 if not s[c] > 0 else min(max(int(np.rint((blk[r, c] - mn[c]) / s[c])), 0), 15)
        assert np.array_equal(pk["scale_k"][0, g], s)
    assert np.array_equal(_unpack(pk["codes_k"], 0, n_full, D, b), want_k)
    want_v = np.zeros((n_full, D), np.int64)
    for r in range(n_full):
        for g in range(D // G):
            blk = vw[r, g * G:(g + 1) * G]
            mn, mx = blk.min(), blk.max()
            s = (mx - mn) / qmax
            for c in range(G):
                want_v[r, g * G + c] = min(max(int(np.rint((blk[c] - mn) / s)), 0), 15) if s > 0 else 0
    assert np.array_equal(_unpack(pk["codes_v"], 0, n_full, D, b), want_v)
    # packed byte layout: channel pairs share a byte, low nibble first
    assert pk["codes_k"][0] == (want_k[0, 0] | (want_k[0, 1] << 4))


# ---------------------------------------------------------------- scoring

def _tiny_qk(gen, B=1, Hq=4, Hkv=2, W=3, N=37, D=16, seed=5):
    q = gen.normal(gen.stream(seed, 1), 0, B * Hq * W * D).reshape(B, Hq, W, D)
    k = gen.normal(gen.stream(seed, 2), 0, B * Hkv * N * D).reshape(B, Hkv, N, D) * 1.5
    return q, k


def test_score_brute_force_and_invariants(ref, gen):
    B, Hq, Hkv, W, N, D = 2, 4, 2, 3, 37, 16
    q, k = _tiny_qk(gen, B, Hq, Hkv, W, N, D)
    seg = np.array([0] * 10 + [1] * 20 + [2] * 7, np.int32)
    sm = 1 / math.sqrt(D)
    sc, ms = ref.score64(q, k, seg, 3, sm)
    G = Hq // Hkv
    want = np.zeros((B, Hkv, N))
    for b in range(B):
        for h in range(Hkv):
            for g in range(G):
                logits = q[b, h * G + g] @ k[b, h].T * sm  # [W, N]
                want[b, h] += sps.softmax(logits, axis=1).sum(axis=0)
    assert np.allclose(sc, want, rtol=1e-13, atol=1e-15)
    assert np.allclose(sc.sum(axis=2), G * W, rtol=1e-12)
    for a in range(3):
        assert np.allclose(ms[..., a], sc[..., seg == a].sum(axis=2), rtol=1e-12)
    assert np.allclose(ms.sum(axis=2), G * W, rtol=1e-12)


def test_score_zero_query_uniform_and_dominant_row(ref, gen):
    B, Hq, Hkv, W, N, D = 1, 4, 1, 2, 50, 16
    q, k = _tiny_qk(gen, B, Hq, Hkv, W, N, D)
    seg = np.zeros(N, np.int32)
    sc, _ = ref.score64(np.zeros_like(q), k, seg, 1, 0.25)
    assert np.allclose(sc, Hq * W / N, rtol=1e-13)
    # a key aligned with every query direction and scaled up takes all mass
    k2 = k.copy()
    k2[0, 0, 17] = 0
    q2 = np.zeros_like(q)
    q2[..., 3] = 1.0
    k2[0, 0, 17, 3] = 400.0
    sc2, _ = ref.score64(q2, k2, seg, 1, 0.25)
    assert abs(sc2[0, 0, 17] - Hq * W) < 1e-9


# ---------------------------------------------------------------- selection

def _brute_select(s, k, n_recent):
    N = s.shape[0]
    cand = np.arange(N - n_recent)
    order = np.lexsort((cand, -s[cand].astype(np.float64)))  # score desc, index asc
    kept = np.concatenate([cand[order[: k - n_recent]], np.arange(N - n_recent, N)])
    return np.sort(kept)


def test_select_brute_force_ties_and_edges(ref):
    rng = np.random.default_rng(3)
    BH, N = 5, 300
    s = rng.integers(0, 20, (BH, N)).astype(np.float32) / 7  # many exact ties
    for k, nr in [(0, 0), (1, 0), (57, 0), (57, 5), (300, 0), (300, 300), (10, 10)]:
        got = ref.select(s, k, nr)
        for bh in range(BH):
            assert np.array_equal(got[bh], _brute_select(s[bh], k, nr)), (k, nr)
            assert np.all(np.diff(got[bh]) > 0)
            kept = np.zeros(N, bool)
            kept[got[bh]] = True
            cand = np.arange(N) < N - nr
            if k - nr > 0 and (~kept & cand).any():
                assert s[bh][kept & cand].min() >= s[bh][~kept & cand].max()
            assert kept[N - nr:].all()
    # exact ties resolve to the lower index
    t = np.zeros((1, 10), np.float32)
    assert np.array_equal(ref.select(t, 3, 0)[0], [0, 1, 2])
    with pytest.raises(ValueError):
        ref.select(t, 11, 0)
    with pytest.raises(ValueError):
        ref.select(t, 3, 4)


# ---------------------------------------------------------------- attention

def _tiny_attn(gen, B=2, Hq=4, Hkv=2, M=3, N=29, D=16, seed=11):
    q = gen.normal(gen.stream(seed, 1), 0, B * Hq * M * D).reshape(B, Hq, M, D)
    k = gen.normal(gen.stream(seed, 2), 0, B * Hkv * N * D).reshape(B, Hkv, N, D)
    v = gen.normal(gen.stream(seed, 3), 0, B * Hkv * N * D).reshape(B, Hkv, N, D)
    return q, k, v


def test_attend_brute_force(ref, gen):
    B, Hq, Hkv, M, N, D = 2, 4, 2, 3, 29, 16
    q, k, v = _tiny_attn(gen, B, Hq, Hkv, M, N, D)
    seg = np.array([0] * 9 + [1] * 15 + [2] * 5, np.int32)
    sm = 1 / math.sqrt(D)
    o, lse, sl, smass = ref.attend(q, k, v, None, seg, 3, sm)
    G = Hq // Hkv
    for b in range(B):
        for h in range(Hq):
            S = q[b, h] @ k[b, h // G].T * sm
            P = sps.softmax(S, axis=1)
            assert np.allclose(o[b, h], P @ v[b, h // G], rtol=1e-12, atol=1e-14)
            assert np.allclose(lse[b, h], sps.logsumexp(S, axis=1), rtol=1e-13)
            for a in range(3):
                assert np.allclose(sl[b, h, :, a], sps.logsumexp(S[:, seg == a], axis=1), rtol=1e-13)
                assert np.allclose(smass[b, h, :, a], P[:, seg == a].sum(axis=1), rtol=1e-12)


def test_attend_closed_forms(ref, gen):
    q, k, v = _tiny_attn(gen)
    seg = np.zeros(k.shape[2], np.int32)
    o, _, _, _ = ref.attend(np.zeros_like(q), k, v, None, seg, 1, 0.3)
    G = q.shape[1] // k.shape[1]
    for h in range(q.shape[1]):
        assert np.allclose(o[:, h], v[:, h // G].mean(axis=1)[:, None, :], rtol=1e-13)
    o1, lse1, _, _ = ref.attend(q, k[:, :, :1], v[:, :, :1], None, seg[:1], 1, 0.3)
    for h in range(q.shape[1]):
        assert np.allclose(o1[:, h], v[:, h // G, :1], rtol=0, atol=1e-15)


def test_attend_chunk_merge_order_and_mask(ref, gen):
    B, Hq, Hkv, M, N, D = 1, 4, 2, 2, 40, 16
    q, k, v = _tiny_attn(gen, B, Hq, Hkv, M, N, D, seed=12)
    seg = np.array([0] * 12 + [1] * 20 + [2] * 8, np.int32)
    sm = 0.25
    o, lse, sl, _ = ref.attend(q, k, v, None, seg, 3, sm)
    # chunks attended separately and merged by log-sum-exp equal one pass
    parts = [(0, 7), (7, 25), (25, 40)]
    outs = [ref.attend(q, k[:, :, a:b], v[:, :, a:b], None, seg[a:b], 3, sm) for a, b in parts]
    L = np.stack([p[1] for p in outs])
    mx = L.max(axis=0)
    w = np.exp(L - mx)
    merged = sum(w[i][..., None] * outs[i][0] for i in range(3)) / w.sum(axis=0)[..., None]
    assert np.allclose(merged, o, rtol=1e-12, atol=1e-14)
    assert np.allclose(mx + np.log(w.sum(axis=0)), lse, rtol=1e-13)
    # segment order does not matter
    perm = np.concatenate([np.arange(32, 40), np.arange(0, 12), np.arange(12, 32)])
    o2, lse2, sl2, _ = ref.attend(q, k[:, :, perm], v[:, :, perm], None, seg[perm], 3, sm)
    assert np.allclose(o2, o, rtol=1e-12, atol=1e-14) and np.allclose(sl2, sl, rtol=1e-13)
    # masked full sequence == physically compacted sequence (App. E identity)
    rng = np.random.default_rng(4)
    present = (rng.random((B, Hkv, N)) < 0.4).astype(np.uint8)
    present[..., 0] = 1
    om, lm, slm, _ = ref.attend(q, k, v, present, seg, 3, sm)
    G = Hq // Hkv
    for h in range(Hkv):
        sel = present[0, h].astype(bool)
        oc, lc, slc, _ = ref.attend(q[:, h * G:(h + 1) * G], k[:, h:h + 1, sel], v[:, h:h + 1, sel],
                                    None, seg[sel], 3, sm)
        assert np.allclose(om[:, h * G:(h + 1) * G], oc, rtol=1e-12, atol=1e-14)
        assert np.allclose(lm[:, h * G:(h + 1) * G], lc, rtol=1e-13)
        assert np.array_equal(np.isinf(slm[:, h * G:(h + 1) * G]), np.isinf(slc))


# ---------------------------------------------------------------- budgets

@pytest.fixture(scope="module")
def gold():
    with open(os.path.join(GOLD, "budget_closed_forms.json")) as f:
        return json.load(f)


def test_accounting_closed_forms(ref, gold):
    acc = gold["accounting"]
    D = 64
    c1 = acc["tiny_understanding"]
    assert int(math.floor(0.2 * 256)) == c1["k"]
    stored = ref.dense_bytes(64, D, "f16") + ref.evicted_bytes(51, D, "f32") + ref.packed_bytes(256, D, 32, 4, "f32")
    assert stored == c1["stored"] and ref.dense_bytes(576, D, "f32") == c1["original"]
    D = 128
    c2 = acc["understanding_7b"]
    orig = ref.dense_bytes(512 + 4096, D, "bf16")
    k = ref.evict_rows(orig / 5.0, ref.dense_bytes(512, D, "bf16"), 4096, D, "bf16")
    assert (orig, k) == (c2["original"], c2["k"])
    assert ref.dense_bytes(512, D, "bf16") + ref.evicted_bytes(k, D, "bf16") == c2["stored"]
    c3 = acc["image_editing"]
    stored = ref.dense_bytes(1024, D, "bf16") + ref.evicted_bytes(1024, D, "bf16") + ref.packed_bytes(4096, D, 64, 4, "bf16")
    assert stored == c3["stored"] and ref.dense_bytes(9216, D, "bf16") == c3["original"]
    c5 = acc["long_context_64k"]
    orig = ref.dense_bytes(65536, D, "bf16")
    fixed = ref.packed_bytes(4096, D, 64, 4, "bf16")
    k = ref.evict_rows(orig / 5.0, fixed, 61440, D, "bf16")
    assert (orig, k, fixed + ref.evicted_bytes(k, D, "bf16")) == (c5["original"], c5["k"], c5["stored"])
    c4 = acc["text_to_image"]
    orig = 4 * ref.dense_bytes(768 + 4096, D, "bf16")
    fixed = 4 * ref.dense_bytes(768, D, "bf16")
    bits = ref.assign_bits([0.3, 0.1, 0.4, 0.2], 4096, D, 64, "bf16", orig / 2.5, fixed)
    assert list(bits) == [4, 2, 4, 4]  # the lowest-mass head stays at 2 bits
    assert (bits == 4).sum() == c4["n_int4"] and (bits == 2).sum() == c4["n_int2"]
    stored = fixed + sum(ref.packed_bytes(4096, D, 64, int(b), "bf16") for b in bits)
    assert stored == c4["stored"] and orig == c4["original"]
    # equal mass: lower head index upgrades first
    assert list(ref.assign_bits([1, 1, 1, 1], 4096, D, 64, "bf16", orig / 2.5, fixed)) == [4, 4, 4, 2]
    for c in acc.values():
        if isinstance(c, dict) and "ratio" in c:
            assert abs(c["original"] / c["stored"] - c["ratio"]) < 1e-6  # ratios printed to 6 places


def test_type_budget_and_retention(ref, gold):
    for c in gold["type_budget"]["cases"]:
        got = ref.type_budget(c["mass"], c["b_prev"], c["B"])
        assert np.allclose(got, c["b_next"], rtol=1e-12, atol=1e-12), c
        assert got.sum() <= c["B"] * (1 + 1e-12)
        assert np.all(got <= np.asarray(c["b_prev"]) * (1 + 1e-12))
    for c in gold["retention"]["cases"]:
        assert abs(ref.retention_next(c["rho"], c["rho_init"], c["rho_min"], c["M_c"], c["M_0"]) - c["next"]) < 1e-12
    assert math.isnan(ref.retention_next(0.3, 0.2, 0.3, 1.0, 1.0))  # rho_min > rho_init
    # schedule is non-increasing and stays within [rho_min, rho_init]
    rho = 0.5
    rng = np.random.default_rng(5)
    for _ in range(50):
        nxt = ref.retention_next(rho, 0.5, 0.1, float(rng.uniform(0, 2)), 1.0)
        assert 0.1 <= nxt <= rho
        rho = nxt


# ---------------------------------------------------------------- generator

def test_generator_pins(gen):
    x = gen.normal(1234, 10, 4000)
    assert np.allclose(x, gen.normal_np(1234, 10, 4000), rtol=1e-14, atol=1e-15)
    big = gen.normal(77, 0, 400000)
    assert abs(big.mean()) < 0.01 and abs(big.std() - 1) < 0.01
    assert abs(np.mean(big ** 4) - 3) < 0.05  # Gaussian kurtosis
    w = gen.UNDERSTANDING_7B
    whole = gen.segment_kv(w, 1, "k", bh0=0, nbh=2, row0=0, n=64)
    piece = gen.segment_kv(w, 1, "k", bh0=1, nbh=1, row0=16, n=8)
    assert np.array_equal(whole[1, 16:24], piece[0])
    ch = gen.outlier_channels(w, 0)
    kw = whole[0].view(np.uint16).astype(np.uint32) << 16
    kf = kw.view(np.float32)
    std = kf.std(axis=0)
    assert set(np.argsort(std)[-2:]) == set(ch.tolist()) and len(ch) == 2


def test_generator_drift(gen):
    """Random-walk drift: a slice of a tensor drifts exactly as inside the
    whole, each step adds sigma * N(0,1) to the fp64 master, and the stored
    copy is the master rounded to the storage dtype."""
    w = gen.scaled(gen.TEXT_TO_IMAGE, M=8)
    k, m = gen.segment_kv(w, 1, "k", bh0=0, nbh=3, row0=0, n=64, master=True)
    whole = gen.Drift(w, gen.T_DRIFT_K, m.copy(), "bf16")
    part = gen.Drift(w, gen.T_DRIFT_K, m[2].copy(), "bf16", start=2 * 64 * w.D)
    prev = m.copy()
    for _ in range(3):
        a, b = whole.step(), part.step()
        assert np.array_equal(a[2], b)
        step = (whole.master - prev) / w.drift_sigma
        assert abs(step.mean()) < 0.02 and abs(step.std() - 1) < 0.02
        prev = whole.master.copy()
    rounded = torch.from_numpy(whole.master).to(torch.bfloat16).view(torch.int16).numpy()
    assert np.array_equal(a.view(np.int16), rounded)
