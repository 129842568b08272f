"""Seeded randomized-shape GPU parity of attention and scoring over mixed
segments: 50 cases drawn over batch, query/KV heads (group sizes 1-16), head
dim, element type, segment kinds and counts (dense with spare capacity,
packed with 2/4/8-bit codes, groups 8-128, per-head widths, residual tails),
row counts (empty segments and ragged tails included) and query rows per
step.  Each case asserts the kernel it reaches (the eligibility rules the
header documents) and matches the oracle: attention within 2e-3 max-abs /
1e-3 relative L2 with lse and per-segment lse, scores and masses within the
double-accumulation tolerance."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import oracle as ref  # noqa: E402
import paper_2609_32831_amd as uc  # noqa: E402
from gpu_util import TORCH, check_attention, dev, packed_from_oracle, rand_rows, sm_scale  # noqa: E402

N_CASES = 50


def _draw(seed):
    rng = np.random.default_rng(1000 + seed)
    D = int(rng.choice([128, 128, 128, 64]))
    dt = str(rng.choice(["bf16"] * 6 + ["f16", "f32"]))
    Hkv = int(rng.choice([1, 2, 4, 8]))
    G = int(rng.choice([1, 2, 4, 7, 8, 16]))
    B = int(rng.integers(1, 4))
    M = int(rng.choice([1, 1, 2, 3, 9, 37, 64, 130]))
    n_segs = int(rng.integers(1, 5))
    segs = []
    for _ in range(n_segs):
        n = int(rng.choice([0, int(rng.integers(1, 40)), int(rng.integers(40, 2500))]))
        if rng.random() < 0.45:
            g = int(rng.choice([g for g in (8, 16, 32, 64, 128) if g <= D]))
            bits = int(rng.choice([2, 4, 4, 8]))
            segs.append(("packed", n, g, bits, bool(rng.random() < 0.3)))
        else:
            segs.append(("dense", n, int(rng.integers(0, 9))))  # spare rows of capacity
    if sum(s[1] for s in segs) == 0:
        segs[0] = ("dense", 77, 3)
    # keep the oracle's share small: rows x query rows x heads
    while B * Hkv * G * M * sum(s[1] for s in segs) * D > 6e8 and M > 1:
        M = max(1, M // 2)
    return dict(D=D, dt=dt, Hkv=Hkv, G=G, B=B, M=M, segs=segs, seed=seed)


def _expected_attend_kernel(c):
    bf = c["dt"] == "bf16" and c["D"] == 128
    if not bf:
        return "attend_valu"
    if c["G"] * c["M"] > 16:
        return "prefill_mfma"
    for s in c["segs"]:
        if s[0] == "packed":
            bits = 4 if s[4] else s[3]  # per-head widths are 2 or 4
            if s[2] < 32 or bits > 4:
                return "attend_valu"
    return "decode_mfma"


def _expected_score_kernel(c):
    if c["dt"] != "bf16" or c["D"] != 128:
        return "score_valu"
    if any(s[0] == "packed" and s[2] < 32 for s in c["segs"]):
        return "score_valu"
    return "score_mfma"


def _build(c):
    B, Hkv, D, dt = c["B"], c["Hkv"], c["D"], c["dt"]
    BH = B * Hkv
    segs, kh, vh, seg_id = [], [], [], []
    for i, s in enumerate(c["segs"]):
        n = s[1]
        base = 100 * c["seed"] + 10 * i
        if s[0] == "dense":
            cap = n + s[2]
            k = rand_rows(base + 1, BH, max(cap, 1), D, dt, outliers=(3,))
            v = rand_rows(base + 2, BH, max(cap, 1), D, dt)
            segs.append(uc.dense_segment(dev(k, dt).reshape(B, Hkv, -1, D),
                                         dev(v, dt).reshape(B, Hkv, -1, D), n_rows=n))
            kh.append(ref.widen(k[:, :n], dt))
            vh.append(ref.widen(v[:, :n], dt))
        else:
            _, _, g, bits, per_head = s
            k = rand_rows(base + 1, BH, n, D, dt, 2.0, outliers=(3,))
            v = rand_rows(base + 2, BH, n, D, dt)
            hb = [bits] * BH if not per_head else [4 if (j % 3) else 2 for j in range(BH)]
            pk = ref.quantize(k, v, dt, g, hb)
            segs.append(packed_from_oracle(B, Hkv, n, D, g, dt, pk, per_head=per_head))
            a, b = ref.dequant(pk, n, D, g, dt)
            kh.append(a)
            vh.append(b)
        seg_id += [i] * n
    K = np.concatenate(kh, axis=1).reshape(B, Hkv, -1, D)
    V = np.concatenate(vh, axis=1).reshape(B, Hkv, -1, D)
    return segs, K, V, np.asarray(seg_id, np.int32)


@pytest.mark.parametrize("seed", range(N_CASES))
def test_random_shapes(seed):
    c = _draw(seed)
    B, Hkv, G, M, D, dt = c["B"], c["Hkv"], c["G"], c["M"], c["D"], c["dt"]
    Hq = Hkv * G
    print(f"CASE random seed={seed} B={B} Hq={Hq} Hkv={Hkv} D={D} dt={dt} M={M} "
          f"segs={c['segs']}", flush=True)
    segs, K, V, seg_id = _build(c)
    nseg = len(segs)
    q = rand_rows(7 + seed, B * Hq, M, D, dt).reshape(B, Hq, M, D)
    sm = sm_scale(D)
    shape = uc.make_shape(B, Hq, Hkv, D)
    qd = dev(q, dt)
    # attention
    o_ref, lse_ref, sl_ref, _ = ref.attend(ref.widen(q, dt), K, V, None, seg_id, nseg, sm)
    o = torch.empty(B, Hq, M, D, device="cuda")
    lse = torch.empty(B, Hq, M, device="cuda")
    sl = torch.empty(B, Hq, M, nseg, device="cuda")
    uc.uc_attend_mixed(shape, segs, qd, M, sm, o, lse, sl)
    assert uc.uc_last_kernel() == _expected_attend_kernel(c), uc.uc_last_kernel()
    o2 = torch.empty_like(o)
    uc.uc_attend_mixed(shape, segs, qd, M, sm, o2)  # the single-softmax form
    torch.cuda.synchronize()
    check_attention(o.cpu().numpy(), o_ref, "o")
    check_attention(o2.cpu().numpy(), o_ref, "o without statistics")
    assert np.allclose(lse.cpu().numpy(), lse_ref, rtol=1e-5, atol=1e-4)
    slg = sl.cpu().numpy()
    fin = np.isfinite(sl_ref)
    assert np.array_equal(np.isfinite(slg), fin)
    assert np.allclose(slg[fin], sl_ref[fin], rtol=1e-5, atol=1e-4)
    # importance scores over the same cache with the step's rows as the
    # observation window
    sc_ref, ms_ref = ref.score64(ref.widen(q, dt), K, seg_id, nseg, sm)
    outs = [torch.empty(B, Hkv, max(s.n_rows, 1), device="cuda") for s in segs]
    mass = torch.empty(B, Hkv, nseg, device="cuda")
    uc.uc_score_importance(shape, segs, qd, M, sm, [o_ if s.n_rows else None
                                                    for o_, s in zip(outs, segs)], mass)
    assert uc.uc_last_kernel() == _expected_score_kernel(c), uc.uc_last_kernel()
    torch.cuda.synchronize()
    tot = G * M
    col = 0
    for s, o_ in zip(segs, outs):
        n = s.n_rows
        if n:
            got = o_.cpu().numpy().reshape(B, Hkv, n).astype(np.float64)
            want = sc_ref[:, :, col:col + n]
            assert np.all(np.abs(got - want) <= 2e-5 * want + 1e-7 * tot), np.max(
                np.abs(got - want) / np.maximum(want, 1e-12))
        col += n
    assert np.allclose(mass.cpu().numpy(), ms_ref, rtol=2e-5, atol=1e-6 * tot)
