"""Per-call GPU parity against the CPU oracle (stage-isolated: both sides get
identical input bytes).  Bars: codes, scales, minima, tails and kept indices
bit-exact; attention within 2e-3 max-abs and 1e-3 relative L2 in fp32."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # collected on CPU-only hosts, never run there
    pytest.skip("needs a GPU", allow_module_level=True)

import oracle as ref  # noqa: E402
import paper_2609_32831_amd as uc  # noqa: E402
import workloads as gen  # noqa: E402
from gpu_util import (TORCH, UCDT, check_attention, dev, host_bytes, mixed_case,  # noqa: E402
                      packed_from_oracle, rand_rows, sm_scale)

_mixed_case = mixed_case


def _print_case(**kw):
    print("CASE", " ".join(f"{k}={v}" for k, v in kw.items()), flush=True)


# ------------------------------------------------------------------ quantize

QCASES = [
    # dtype, B, Hkv, N, D, G, bits (int or per-head list)
    ("f32", 1, 1, 256, 64, 32, 4),
    ("bf16", 2, 4, 4096 + 37, 128, 64, 4),
    ("bf16", 2, 4, 1000, 128, 64, [4, 2, 4, 4, 2, 4, 4, 2]),
    ("f16", 1, 2, 500, 128, 32, 2),
    ("bf16", 1, 3, 77, 64, 8, 8),
    ("bf16", 1, 2, 100, 128, 128, 4),   # shorter than one group: all tail
    ("bf16", 1, 1, 64, 128, 64, 2),     # exactly one group, no tail
    # shapes of the vectorised kernels: key groups shorter than a pass (8 rows),
    # head dim 64 with 8-bit codes, per-head widths with whole-row groups
    ("bf16", 1, 2, 300, 128, 8, 4),
    ("f16", 2, 2, 640 + 63, 64, 64, 8),
    ("bf16", 1, 4, 1024 + 5, 128, 128, [8, 2, 4, 8]),
    ("bf16", 1, 1, 48, 128, 16, 2),
]


@pytest.mark.parametrize("case", QCASES, ids=[f"q{i}" for i in range(len(QCASES))])
def test_quantize_bit_exact(case):
    dtype, B, Hkv, N, D, G, bits = case
    _print_case(test="quantize", dtype=dtype, B=B, Hkv=Hkv, N=N, D=D, G=G, bits=bits)
    BH = B * Hkv
    per_head = isinstance(bits, list)
    hb = bits if per_head else [bits] * BH
    k = rand_rows(11, BH, N, D, dtype, 2.0, outliers=(3, 40))
    v = rand_rows(12, BH, N, D, dtype)
    pk = ref.quantize(k, v, dtype, G, hb)
    seg = uc.packed_segment(B, Hkv, N, D, G, TORCH[dtype], bits=hb[0],
                            head_bits=hb if per_head else None)
    shape = uc.make_shape(B, Hkv, Hkv, D)
    kd = dev(k, dtype).reshape(B, Hkv, N, D)
    vd = dev(v, dtype).reshape(B, Hkv, N, D)
    uc.uc_quantize_segment(shape, kd, vd, N, seg)
    torch.cuda.synchronize()
    n = pk["codes_k"].shape[0]
    assert np.array_equal(seg.t["codes_k"].cpu().numpy()[:n], pk["codes_k"])
    assert np.array_equal(seg.t["codes_v"].cpu().numpy()[:n], pk["codes_v"])
    for name in ("scale_k", "min_k", "scale_v", "min_v"):
        got = seg.t[name].cpu().numpy().reshape(pk[name].shape)
        assert np.array_equal(got.view(np.uint32), pk[name].view(np.uint32)), name
    if pk["tail_k"].shape[1]:
        assert np.array_equal(host_bytes(seg.t["tail_k"]).reshape(pk["tail_k"].shape), pk["tail_k"])
        assert np.array_equal(host_bytes(seg.t["tail_v"]).reshape(pk["tail_v"].shape), pk["tail_v"])


def test_quantize_constant_and_ramp_groups():
    """Groups whose values are constant (scale 0: codes 0, minimum = the
    value) and exact ramps 0..15 (scale 1, minimum 0: code = value), through
    the vectorised kernels (bf16, head dim 128, group 64, 4 bits), plus a
    residual tail; bit-exact against the oracle and against the closed forms."""
    _print_case(test="quantize_constant_ramp")
    B, Hkv, D, G, N = 1, 2, 128, 64, 128 + 5
    BH = B * Hkv
    r = np.arange(N, dtype=np.float64)[None, :, None]
    c = np.arange(D, dtype=np.float64)[None, None, :]
    k = np.where(r < G, np.broadcast_to(c / 8.0, (BH, N, D)), np.broadcast_to(r % 16, (BH, N, D)))
    v = np.where(c < G, np.broadcast_to(r / 4.0, (BH, N, D)), np.broadcast_to(c % 16, (BH, N, D)))
    k = gen.round_to(np.ascontiguousarray(k), "bf16")
    v = gen.round_to(np.ascontiguousarray(v), "bf16")
    pk = ref.quantize(k, v, "bf16", G, [4] * BH)
    seg = uc.packed_segment(B, Hkv, N, D, G, torch.bfloat16, bits=4)
    shape = uc.make_shape(B, Hkv, Hkv, D)
    uc.uc_quantize_segment(shape, dev(k, "bf16").reshape(B, Hkv, N, D),
                           dev(v, "bf16").reshape(B, Hkv, N, D), N, seg)
    torch.cuda.synchronize()
    n = pk["codes_k"].shape[0]
    ck = seg.t["codes_k"].cpu().numpy()[:n]
    cv = seg.t["codes_v"].cpu().numpy()[:n]
    assert np.array_equal(ck, pk["codes_k"]) and np.array_equal(cv, pk["codes_v"])
    for name in ("scale_k", "min_k", "scale_v", "min_v"):
        got = seg.t[name].cpu().numpy().reshape(pk[name].shape)
        assert np.array_equal(got.view(np.uint32), pk[name].view(np.uint32)), name
    sk = seg.t["scale_k"].cpu().numpy().reshape(BH, N // G, D)
    mk = seg.t["min_k"].cpu().numpy().reshape(BH, N // G, D)
    assert np.all(sk[:, 0] == 0.0) and np.array_equal(mk[:, 0], np.broadcast_to(np.arange(D) / 8.0, (BH, D)))
    assert np.all(sk[:, 1] == 1.0) and np.all(mk[:, 1] == 0.0)
    sv = seg.t["scale_v"].cpu().numpy().reshape(BH, N // G * G, D // G)
    assert np.all(sv[:, :, 0] == 0.0) and np.all(sv[:, :, 1] == 1.0)
    codes = ck.reshape(BH, N // G * G, D // 2)    # 4-bit codes, two channels per byte
    lo, hi = codes & 15, codes >> 4
    assert np.all(lo[:, :G] == 0) and np.all(hi[:, :G] == 0)          # constant key groups
    rows = np.arange(G, 2 * G) % 16
    assert np.all(lo[:, G:2 * G] == rows[None, :, None]) and np.all(hi[:, G:2 * G] == rows[None, :, None])
    vcodes = cv.reshape(BH, N // G * G, D // 2)
    want_v = np.arange(D)[G:] % 16
    assert np.all((vcodes[:, :, G // 2:] & 15) == want_v[0::2]) and np.all((vcodes[:, :, G // 2:] >> 4) == want_v[1::2])
    assert np.all(vcodes[:, :, : G // 2] == 0)


# ------------------------------------------------------------------ select

@pytest.mark.parametrize("N,k,nr", [(1, 1, 0), (100, 37, 0), (100, 37, 5), (4099, 1024, 0),
                                    (4099, 4099, 0), (61440, 11735, 0), (300, 10, 10),
                                    (1500, 0, 0)])
def test_select_bit_exact(N, k, nr):
    _print_case(test="select", N=N, k=k, n_recent=nr)
    BH, D = 6, 128
    rng = np.random.default_rng(N + k)
    s = rng.integers(0, 50, (BH, N)).astype(np.float32) / 13.0  # many exact ties
    s[0] = rng.random(N).astype(np.float32)
    s[1, : N // 2] = 0.0
    s[2] = 1.0                                                    # all equal: lowest indices
    s[3] = rng.choice(np.array([-1.5, -0.0, 0.0, 2.0], np.float32), N)  # signs, -0 ties +0
    want = ref.select(s, k, nr)
    sd = torch.from_numpy(s).cuda()
    keep = torch.full((BH, max(k, 1)), -7, dtype=torch.int32, device="cuda")
    kv = rand_rows(5, BH, N, D, "bf16")
    ksrc = dev(kv, "bf16")
    vsrc = dev(kv[:, ::-1].copy(), "bf16")
    kdst = torch.zeros(BH, max(k, 1), D, dtype=torch.bfloat16, device="cuda")
    vdst = torch.zeros_like(kdst)
    uc.uc_select_keep(sd, k, nr, keep, ksrc, vsrc, kdst, vdst)
    torch.cuda.synchronize()
    if k == 0:
        return
    got = keep.cpu().numpy()
    assert np.array_equal(got, want)
    kb = host_bytes(kdst)
    vb = host_bytes(vdst)
    for bh in range(BH):
        assert np.array_equal(kb[bh], kv[bh][want[bh]])
        assert np.array_equal(vb[bh], kv[bh, ::-1][want[bh]])


# ------------------------------------------------------------------ attention

ACASES = [
    # B, Hq, Hkv, D, dtype, q dtype, M, sizes
    (1, 4, 1, 64, "f32", "f32", 1, (64, 256, 51, 256, 0, 4)),
    (2, 28, 4, 128, "bf16", "bf16", 1, (512, 4096, 406, 4096 + 17, 5, 16)),
    (2, 28, 4, 128, "bf16", "bf16", 7, (100, 900, 300, 1000, 3, 8)),
    (1, 8, 2, 64, "f16", "f16", 3, (33, 200, 77, 130, 1, 2)),
    (1, 14, 2, 128, "bf16", "bf16", 1, (0, 700, 1, 63, 2, 2)),   # empty text, tail-only pack
]


@pytest.mark.parametrize("case", ACASES, ids=[f"a{i}" for i in range(len(ACASES))])
def test_attend_parity(case):
    B, Hq, Hkv, D, dtype, qdt, M, sizes = case
    _print_case(test="attend", B=B, Hq=Hq, Hkv=Hkv, D=D, dtype=dtype, M=M, sizes=sizes)
    segs, K, V, seg_id = _mixed_case(B, Hq, Hkv, D, dtype, sizes, seed=D + M)
    q = rand_rows(99, B * Hq, M, D, qdt).reshape(B, Hq, M, D)
    sm = sm_scale(D)
    o_ref, lse_ref, sl_ref, _ = ref.attend(ref.widen(q, qdt), K, V, None, seg_id, 4, sm)
    shape = uc.make_shape(B, Hq, Hkv, D)
    qd = dev(q, qdt)
    o = torch.empty(B, Hq, M, D, device="cuda")
    lse = torch.empty(B, Hq, M, device="cuda")
    sl = torch.empty(B, Hq, M, 4, device="cuda")
    uc.uc_attend_mixed(shape, segs, qd, M, sm, o, lse, sl)
    torch.cuda.synchronize()
    check_attention(o.cpu().numpy(), o_ref, "o")
    assert np.allclose(lse.cpu().numpy(), lse_ref, rtol=1e-5, atol=1e-4)
    slg = sl.cpu().numpy()
    fin = np.isfinite(sl_ref)
    assert np.array_equal(np.isfinite(slg), fin)
    assert np.allclose(slg[fin], sl_ref[fin], rtol=1e-5, atol=1e-4)


def test_attend_full_budget_equals_uncompressed():
    """A 100%-budget eviction segment (all rows kept) plus 16-bit rows is exact
    attention over the original sequence."""
    B, Hq, Hkv, D, N = 2, 28, 4, 128, 1000
    BH = B * Hkv
    k = rand_rows(1, BH, N, D, "bf16", outliers=(7,))
    v = rand_rows(2, BH, N, D, "bf16")
    q = rand_rows(3, B * Hq, 1, D, "bf16").reshape(B, Hq, 1, D)
    scores = torch.rand(BH, N, device="cuda")
    keep = torch.empty(BH, N, dtype=torch.int32, device="cuda")
    kd, vd = dev(k, "bf16"), dev(v, "bf16")
    kc, vc = torch.empty_like(kd), torch.empty_like(vd)
    uc.uc_select_keep(scores, N, 0, keep, kd, vd, kc, vc)
    shape = uc.make_shape(B, Hq, Hkv, D)
    o1 = torch.empty(B, Hq, 1, D, device="cuda")
    o2 = torch.empty_like(o1)
    uc.uc_attend_mixed(shape, [uc.dense_segment(kd.reshape(B, Hkv, N, D), vd.reshape(B, Hkv, N, D))],
                       dev(q, "bf16"), 1, sm_scale(D), o1)
    uc.uc_attend_mixed(shape, [uc.dense_segment(kc.reshape(B, Hkv, N, D), vc.reshape(B, Hkv, N, D))],
                       dev(q, "bf16"), 1, sm_scale(D), o2)
    torch.cuda.synchronize()
    assert np.array_equal(keep.cpu().numpy(), np.tile(np.arange(N, dtype=np.int32), (BH, 1)))
    assert torch.equal(o1, o2)
    o_ref = ref.attend(ref.widen(q, "bf16"), ref.widen(k, "bf16").reshape(B, Hkv, N, D),
                       ref.widen(v, "bf16").reshape(B, Hkv, N, D), None, np.zeros(N, np.int32), 1,
                       sm_scale(D))[0]
    check_attention(o1.cpu().numpy(), o_ref, "full budget")


# ------------------------------------------------------------------ scoring

@pytest.mark.parametrize("B,Hq,Hkv,D,dtype,W,sizes", [
    (1, 4, 1, 64, "f32", 16, (64, 256, 256)),
    (2, 28, 4, 128, "bf16", 32, (512, 4096, 0)),
    (1, 14, 2, 128, "bf16", 5, (100, 333, 70)),
    (1, 28, 4, 128, "bf16", 40, (300, 1500)),        # 280 query rows: two query blocks
    (1, 14, 2, 128, "bf16", 600, (1030, 2100, 1)),   # 4200 query rows, ragged chunks
])
def test_score_parity(B, Hq, Hkv, D, dtype, W, sizes):
    _print_case(test="score", B=B, Hq=Hq, Hkv=Hkv, D=D, dtype=dtype, W=W, sizes=sizes)
    BH = B * Hkv
    ks, vs, segs, seg_id = [], [], [], []
    for a, n in enumerate(sizes):
        k = rand_rows(20 + a, BH, n, D, dtype, outliers=(2, 9))
        v = rand_rows(30 + a, BH, n, D, dtype)
        ks.append(k); vs.append(v)
        segs.append(uc.dense_segment(dev(k, dtype).reshape(B, Hkv, n, D),
                                     dev(v, dtype).reshape(B, Hkv, n, D)))
        seg_id += [a] * n
    q = rand_rows(40, B * Hq, W, D, dtype).reshape(B, Hq, W, D)
    K = np.concatenate([ref.widen(k, dtype) for k in ks], axis=1).reshape(B, Hkv, -1, D)
    sc_ref, ms_ref = ref.score64(ref.widen(q, dtype), K, np.asarray(seg_id, np.int32), len(sizes),
                                 sm_scale(D))
    shape = uc.make_shape(B, Hq, Hkv, D)
    tot = Hq // Hkv * W
    # bf16 / head dim 128 takes the matrix-core kernels; the VALU path is
    # checked on the same inputs
    for path in (uc.UC_PATH_AUTO, uc.UC_PATH_VALU):
        prev = uc.uc_set_path(path)
        try:
            outs = [torch.empty(B, Hkv, n, device="cuda") for n in sizes]
            mass = torch.empty(B, Hkv, len(sizes), device="cuda")
            uc.uc_score_importance(shape, segs, dev(q, dtype), W, sm_scale(D), outs, mass)
            torch.cuda.synchronize()
        finally:
            uc.uc_set_path(prev)
        got = np.concatenate([o.cpu().numpy().reshape(B, Hkv, -1) for o in outs],
                             axis=2).astype(np.float64)
        rel = np.abs(got - sc_ref) / np.maximum(sc_ref, 1e-12)
        # per-row probability mass is resolved to ~1e-6 of the row total
        assert np.all(np.abs(got - sc_ref) <= 2e-5 * sc_ref + 1e-7 * tot), (path, rel.max())
        assert np.allclose(mass.cpu().numpy(), ms_ref, rtol=2e-5, atol=1e-6 * tot), path
        assert np.allclose(got.sum(axis=2), tot, rtol=1e-5), path


SPCASES = [
    # B, Hq, Hkv, W, G, bits, per_head, (text, packed rows); packed rows past
    # n_full form the tail
    (1, 28, 4, 32, 64, 4, False, (300, 4096 + 17)),
    (2, 14, 2, 40, 32, 2, True, (0, 2000 + 5)),     # int2/int4 per head, two query blocks
    (1, 28, 4, 5, 128, 8, False, (64, 1030)),
    (1, 14, 2, 8, 16, 4, False, (100, 333)),        # groups below 32: the VALU scorer
]


@pytest.mark.parametrize("case", SPCASES, ids=[f"sp{i}" for i in range(len(SPCASES))])
def test_score_parity_packed(case):
    """Scoring over a cache holding a packed segment: the matrix-core passes
    decode its code rows in registers (keys only) and read its tail rows as
    stored; scores and masses match the oracle over the dequantised keys."""
    B, Hq, Hkv, W, G, bits, per_head, (n_text, n_pack) = case
    D = 128
    _print_case(test="score_packed", B=B, Hq=Hq, Hkv=Hkv, W=W, G=G, bits=bits, sizes=(n_text, n_pack))
    BH = B * Hkv
    kt = rand_rows(61, BH, n_text, D, "bf16", outliers=(3,))
    vt = rand_rows(62, BH, n_text, D, "bf16")
    kp = rand_rows(63, BH, n_pack, D, "bf16", 2.0, outliers=(3, 77))
    vp = rand_rows(64, BH, n_pack, D, "bf16")
    hb = [bits] * BH if not per_head else [4 if (i % 3) else 2 for i in range(BH)]
    pk = ref.quantize(kp, vp, "bf16", G, hb)
    segs = [uc.dense_segment(dev(kt, "bf16").reshape(B, Hkv, n_text, D),
                             dev(vt, "bf16").reshape(B, Hkv, n_text, D)),
            packed_from_oracle(B, Hkv, n_pack, D, G, "bf16", pk, per_head=per_head)]
    khp, _ = ref.dequant(pk, n_pack, D, G, "bf16")
    K = np.concatenate([ref.widen(kt, "bf16"), khp], axis=1).reshape(B, Hkv, -1, D)
    seg_id = np.asarray([0] * n_text + [1] * n_pack, np.int32)
    q = rand_rows(65, B * Hq, W, D, "bf16").reshape(B, Hq, W, D)
    sc_ref, ms_ref = ref.score64(ref.widen(q, "bf16"), K, seg_id, 2, sm_scale(D))
    shape = uc.make_shape(B, Hq, Hkv, D)
    tot = Hq // Hkv * W
    want_kernel = "score_mfma" if G >= 32 else "score_valu"
    for path, kernel in ((uc.UC_PATH_AUTO, want_kernel), (uc.UC_PATH_VALU, "score_valu")):
        prev = uc.uc_set_path(path)
        try:
            outs = [torch.empty(B, Hkv, n, device="cuda") for n in (n_text, n_pack)]
            mass = torch.empty(B, Hkv, 2, device="cuda")
            uc.uc_score_importance(shape, segs, dev(q, "bf16"), W, sm_scale(D), outs, mass)
            assert uc.uc_last_kernel() == kernel, (path, uc.uc_last_kernel())
            torch.cuda.synchronize()
        finally:
            uc.uc_set_path(prev)
        got = np.concatenate([o.cpu().numpy().reshape(B, Hkv, -1) for o in outs],
                             axis=2).astype(np.float64)
        assert np.all(np.abs(got - sc_ref) <= 2e-5 * sc_ref + 1e-7 * tot), (kernel, np.max(
            np.abs(got - sc_ref) / np.maximum(sc_ref, 1e-12)))
        assert np.allclose(mass.cpu().numpy(), ms_ref, rtol=2e-5, atol=1e-6 * tot), kernel


def test_segment_mass_from_attention():
    B, Hq, Hkv, D, M = 2, 28, 4, 128, 9
    segs, K, V, seg_id = _mixed_case(B, Hq, Hkv, D, "bf16", (64, 400, 100, 256, 3, 8), seed=3)
    q = rand_rows(7, B * Hq, M, D, "bf16").reshape(B, Hq, M, D)
    _, _, _, smass = ref.attend(ref.widen(q, "bf16"), K, V, None, seg_id, 4, sm_scale(D))
    want = smass.reshape(B, Hkv, Hq // Hkv, M, 4).sum(axis=(2, 3))
    shape = uc.make_shape(B, Hq, Hkv, D)
    o = torch.empty(B, Hq, M, D, device="cuda")
    lse = torch.empty(B, Hq, M, device="cuda")
    sl = torch.empty(B, Hq, M, 4, device="cuda")
    uc.uc_attend_mixed(shape, segs, dev(q, "bf16"), M, sm_scale(D), o, lse, sl)
    mass = torch.empty(B, Hkv, 4, device="cuda")
    uc.uc_segment_mass(shape, M, 4, lse, sl, mass)
    torch.cuda.synchronize()
    assert np.allclose(mass.cpu().numpy(), want, rtol=1e-4, atol=1e-5)


def test_append_rows():
    B, Hkv, D, cap = 2, 4, 128, 8
    shape = uc.make_shape(B, 28, Hkv, D)
    k = torch.zeros(B, Hkv, cap, D, dtype=torch.bfloat16, device="cuda")
    v = torch.zeros_like(k)
    seg = uc.dense_segment(k, v, n_rows=0)
    for t in range(3):
        kn = torch.randn(B, Hkv, 1, D, device="cuda").to(torch.bfloat16)
        vn = torch.randn(B, Hkv, 1, D, device="cuda").to(torch.bfloat16)
        uc.uc_append_rows(shape, kn, vn, 1, seg, t)
        torch.cuda.synchronize()
        assert torch.equal(k[:, :, t], kn[:, :, 0]) and torch.equal(v[:, :, t], vn[:, :, 0])
    assert not k[:, :, 3:].any()


# ------------------------------------------------------------------ matrix-core decode

DCASES = [
    # B, Hq, Hkv, M, G, bits, per_head, sizes (text, vit_full, vit_keep, pack, tail, cap)
    # every case reaches the matrix-core decode kernel (bf16, D = 128, G*M <= 16,
    # packed groups >= 32, widths <= 4); the test asserts it
    (2, 28, 4, 1, 64, 4, False, (512, 4096, 406, 4096, 7, 16)),
    (2, 28, 4, 2, 32, 4, False, (77, 3000, 1111, 4096 + 33, 1, 4)),
    (1, 28, 4, 1, 32, 2, True, (300, 900, 333, 1000, 3, 8)),          # int2/int4 per head, G 32
    (1, 28, 4, 1, 128, 2, False, (31, 700, 129, 5000, 2, 2)),         # int2, G 128
    (1, 16, 1, 1, 32, 4, True, (1, 64, 33, 520, 1, 1)),              # 16 query heads per KV head
    (2, 14, 2, 1, 64, 4, False, (4096, 61440 // 8, 1467, 4096, 511, 512)),
    (2, 28, 4, 1, 64, 2, False, (300, 2000, 512, 1000, 17, 32)),
    (1, 28, 4, 2, 128, 4, False, (0, 100, 3, 130, 0, 4)),
    (2, 28, 4, 1, 64, 4, True, (128, 1000, 257, 2048 + 40, 5, 8)),   # int2/int4 per head
    (1, 28, 4, 1, 32, 4, False, (0, 0, 0, 31, 1, 1)),                # tail-only packed rows
    # 64 KV heads, so that a head's shares are several tiles long: the largest
    # dense segment is split around the others at every phase (compacted
    # rows here, the first segment in the next case), its last share ending
    # in a partial tile
    (8, 56, 8, 1, 64, 4, False, (200, 3000, 1500, 2048 + 10, 37, 64)),
    (8, 56, 8, 1, 32, 4, False, (2000, 300, 100, 1024, 3, 4)),
]

# decode cases outside the matrix-core kernel's range (groups below 32,
# 8-bit codes): the VALU kernel serves them, and the test asserts that
VCASES = [
    (1, 28, 4, 1, 16, 2, True, (300, 900, 333, 1000, 3, 8)),
    (1, 28, 4, 1, 128, 8, False, (31, 700, 129, 5000, 2, 2)),
    (1, 16, 1, 1, 8, 4, True, (1, 64, 33, 520, 1, 1)),
]


def _decode_case(case):
    B, Hq, Hkv, M, G, bits, per_head, sizes = case
    D = 128
    segs, K, V, seg_id = _mixed_case(B, Hq, Hkv, D, "bf16", sizes, seed=G + bits, G=G,
                                     bits=bits, per_head=per_head)
    q = rand_rows(77, B * Hq, M, D, "bf16").reshape(B, Hq, M, D)
    o_ref, lse_ref, sl_ref, _ = ref.attend(ref.widen(q, "bf16"), K, V, None, seg_id, 4,
                                           sm_scale(D))
    return segs, q, (o_ref, lse_ref, sl_ref)


@pytest.mark.parametrize("case", VCASES, ids=[f"v{i}" for i in range(len(VCASES))])
def test_decode_valu_parity(case):
    B, Hq, Hkv, M, G, bits, per_head, sizes = case
    _print_case(test="decode_valu", B=B, Hq=Hq, Hkv=Hkv, M=M, G=G, bits=bits, sizes=sizes)
    D = 128
    segs, q, (o_ref, lse_ref, sl_ref) = _decode_case(case)
    shape = uc.make_shape(B, Hq, Hkv, D)
    o = torch.empty(B, Hq, M, D, device="cuda")
    lse = torch.empty(B, Hq, M, device="cuda")
    sl = torch.empty(B, Hq, M, 4, device="cuda")
    uc.uc_attend_mixed(shape, segs, dev(q, "bf16"), M, sm_scale(D), o, lse, sl)
    assert uc.uc_last_kernel() == "attend_valu"
    torch.cuda.synchronize()
    check_attention(o.cpu().numpy(), o_ref, "valu")
    assert np.allclose(lse.cpu().numpy(), lse_ref, rtol=1e-5, atol=1e-4)
    fin = np.isfinite(sl_ref)
    slg = sl.cpu().numpy()
    assert np.array_equal(np.isfinite(slg), fin)
    assert np.allclose(slg[fin], sl_ref[fin], rtol=1e-5, atol=1e-4)


@pytest.mark.parametrize("case", DCASES, ids=[f"d{i}" for i in range(len(DCASES))])
def test_decode_mfma_parity(case):
    B, Hq, Hkv, M, G, bits, per_head, sizes = case
    _print_case(test="decode_mfma", B=B, Hq=Hq, Hkv=Hkv, M=M, G=G, bits=bits, sizes=sizes)
    D = 128
    segs, q, (o_ref, lse_ref, sl_ref) = _decode_case(case)
    sm = sm_scale(D)
    shape = uc.make_shape(B, Hq, Hkv, D)
    qd = dev(q, "bf16")
    outs = {}
    # matrix-core path with per-segment statistics (one record per segment),
    # matrix-core path with o only (one running state across segments), and
    # the VALU path
    for name, path, want_sl, kernel in (
            ("mfma", uc.UC_PATH_AUTO, True, "decode_mfma"),
            ("mfma_o", uc.UC_PATH_AUTO, False, "decode_mfma"),
            ("valu", uc.UC_PATH_VALU, True, "attend_valu")):
        prev = uc.uc_set_path(path)
        try:
            o = torch.empty(B, Hq, M, D, device="cuda")
            lse = torch.empty(B, Hq, M, device="cuda") if want_sl else None
            sl = torch.empty(B, Hq, M, 4, device="cuda") if want_sl else None
            uc.uc_attend_mixed(shape, segs, qd, M, sm, o, lse, sl)
            assert uc.uc_last_kernel() == kernel, (name, uc.uc_last_kernel())
            torch.cuda.synchronize()
            outs[name] = (o.cpu().numpy(), None if lse is None else lse.cpu().numpy(),
                          None if sl is None else sl.cpu().numpy())
        finally:
            uc.uc_set_path(prev)
    for name, (o, lse, sl) in outs.items():
        check_attention(o, o_ref, f"path {name}")
        if lse is None:
            continue
        assert np.allclose(lse, lse_ref, rtol=1e-5, atol=1e-4)
        fin = np.isfinite(sl_ref)
        assert np.array_equal(np.isfinite(sl), fin)
        assert np.allclose(sl[fin], sl_ref[fin], rtol=1e-5, atol=1e-4)
    # the two kernels agree far inside the bar
    assert np.abs(outs["mfma"][0] - outs["valu"][0]).max() < 5e-4
    assert np.abs(outs["mfma_o"][0] - outs["valu"][0]).max() < 5e-4


# ------------------------------------------------------------------ matrix-core prefill

PCASES = [
    # B, Hq, Hkv, M, G, bits, per_head, sizes (text, vit_full, vit_keep, pack, tail, cap)
    (1, 28, 4, 64, 64, 4, False, (100, 900, 300, 1000 + 17, 5, 8)),   # 448 rows per KV head
    (2, 14, 2, 37, 16, 2, True, (33, 200, 77, 130, 1, 2)),            # ragged block, group 16
    (1, 28, 4, 3, 128, 8, False, (0, 100, 3, 130, 0, 4)),             # 21 rows, 8-bit, empty text
    (1, 16, 1, 2, 32, 4, False, (1, 64, 33, 520, 1, 1)),              # 32 rows, 16 heads per KV
    (1, 28, 4, 40, 64, 4, False, (0, 0, 0, 31, 0, 1)),                # tail-only packed rows
    # 256 KV heads of one 252-row block: a grid of one workgroup per CU, so the
    # eight-wave layout with two tiles per stage runs; 15 tiles (the last
    # stage holds one), partial tiles in every view
    (64, 28, 4, 36, 64, 4, False, (70, 300, 111, 200 + 17, 3, 8)),
]


@pytest.mark.parametrize("case", PCASES, ids=[f"p{i}" for i in range(len(PCASES))])
def test_prefill_mfma_parity(case):
    B, Hq, Hkv, M, G, bits, per_head, sizes = case
    _print_case(test="prefill_mfma", B=B, Hq=Hq, Hkv=Hkv, M=M, G=G, bits=bits, sizes=sizes)
    D = 128
    segs, K, V, seg_id = _mixed_case(B, Hq, Hkv, D, "bf16", sizes, seed=3 * G + bits, G=G,
                                     bits=bits, per_head=per_head)
    q = rand_rows(55, B * Hq, M, D, "bf16").reshape(B, Hq, M, D)
    sm = sm_scale(D)
    o_ref, lse_ref, sl_ref, _ = ref.attend(ref.widen(q, "bf16"), K, V, None, seg_id, 4, sm)
    shape = uc.make_shape(B, Hq, Hkv, D)
    qd = dev(q, "bf16")
    outs = {}
    for name, path, kernel in (("mfma", uc.UC_PATH_AUTO, "prefill_mfma"),
                               ("valu", uc.UC_PATH_VALU, "attend_valu")):
        prev = uc.uc_set_path(path)
        try:
            o = torch.empty(B, Hq, M, D, device="cuda")
            lse = torch.empty(B, Hq, M, device="cuda")
            sl = torch.empty(B, Hq, M, 4, device="cuda")
            uc.uc_attend_mixed(shape, segs, qd, M, sm, o, lse, sl)
            assert uc.uc_last_kernel() == kernel, (name, uc.uc_last_kernel())
            torch.cuda.synchronize()
            outs[name] = (o.cpu().numpy(), lse.cpu().numpy(), sl.cpu().numpy())
        finally:
            uc.uc_set_path(prev)
    for name, (o, lse, sl) in outs.items():
        check_attention(o, o_ref, f"path {name}")
        assert np.allclose(lse, lse_ref, rtol=1e-5, atol=1e-4), name
        fin = np.isfinite(sl_ref)
        assert np.array_equal(np.isfinite(sl), fin), name
        assert np.allclose(sl[fin], sl_ref[fin], rtol=1e-5, atol=1e-4), name
    # fp16 probabilities (11 significant bits) on the matrix-core path
    assert np.abs(outs["mfma"][0] - outs["valu"][0]).max() < 1.5e-3



def test_prefill_value_outside_fp16_range():
    """A value row holding 70000 (beyond fp16's 65504) switches the prefill
    PV product from fp16 to bf16 hi + lo parts; the result still matches.  The
    row's key is zero so its probability is moderate and the output finite."""
    B, Hq, Hkv, D, M = 1, 28, 4, 128, 9
    segs, K, V, seg_id = _mixed_case(B, Hq, Hkv, D, "bf16", (64, 300, 100, 256, 3, 8), seed=11)
    kt, vt = segs[0].t["k"], segs[0].t["v"]          # dense text segment [B, Hkv, 64, D]
    kt[:, :, 5] = 0
    vt[:, :, 5, 3] = 70000.0
    torch.cuda.synchronize()
    K = K.copy()
    V = V.copy()
    K[:, :, 5] = 0.0
    V[:, :, 5, 3] = float(torch.tensor(70000.0, dtype=torch.bfloat16))
    q = rand_rows(12, B * Hq, M, D, "bf16").reshape(B, Hq, M, D)
    o_ref, lse_ref, _, _ = ref.attend(ref.widen(q, "bf16"), K, V, None, seg_id, 4, sm_scale(D))
    o = torch.empty(B, Hq, M, D, device="cuda")
    lse = torch.empty(B, Hq, M, device="cuda")
    uc.uc_attend_mixed(uc.make_shape(B, Hq, Hkv, D), segs, dev(q, "bf16"), M, sm_scale(D), o, lse)
    torch.cuda.synchronize()
    assert uc.uc_last_kernel() == "prefill_mfma"
    og = o.cpu().numpy()
    assert np.isfinite(og).all() and np.abs(og).max() > 10.0
    check_attention(og, o_ref, "value outside fp16 range")  # the usual bar
    assert np.allclose(lse.cpu().numpy(), lse_ref, rtol=1e-5, atol=1e-4)


# ------------------------------------------------------------------ timing hook

@pytest.mark.parametrize("M", [1, 40], ids=["decode", "prefill"])
def test_kernel_events_bracket_attention_kernel(M):
    """uc_set_kernel_events: the pair lies inside the call's own pair, the
    outputs are unchanged, and the setting lasts exactly one call."""
    B, Hq, Hkv, D = 1, 28, 4, 128
    _print_case(test="kernel_events", M=M)
    segs, K, V, seg_id = _mixed_case(B, Hq, Hkv, D, "bf16", (100, 900, 300, 1000 + 17, 5, 8),
                                     seed=3, G=64, bits=4, per_head=False)
    q = dev(rand_rows(5, B * Hq, M, D, "bf16").reshape(B, Hq, M, D), "bf16")
    shape = uc.make_shape(B, Hq, Hkv, D)
    sm = sm_scale(D)
    o0 = torch.empty(B, Hq, M, D, device="cuda")
    uc.uc_attend_mixed(shape, segs, q, M, sm, o0)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    for e in ev:
        e.record()
    torch.cuda.synchronize()
    o1 = torch.empty_like(o0)
    ev[0].record()
    uc.uc_set_kernel_events(ev[2], ev[3])
    uc.uc_attend_mixed(shape, segs, q, M, sm, o1)
    ev[1].record()
    torch.cuda.synchronize()
    call_ms, kern_ms = ev[0].elapsed_time(ev[1]), ev[2].elapsed_time(ev[3])
    assert 0.0 < kern_ms <= call_ms
    assert ev[0].elapsed_time(ev[2]) >= 0.0 and ev[3].elapsed_time(ev[1]) >= 0.0
    assert torch.equal(o0, o1)
    # the next call records nothing: the kernel pair keeps its timestamps
    uc.uc_attend_mixed(shape, segs, q, M, sm, o1)
    torch.cuda.synchronize()
    assert ev[2].elapsed_time(ev[3]) == kern_ms
    assert ev[0].elapsed_time(ev[2]) <= call_ms
