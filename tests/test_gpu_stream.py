"""GPU parity of the streaming residual tail (App. E storage: the N mod G
most recent rows of a quantised segment stay in its tail; full row groups are
quantised as they complete).  The oracle's definition is plain: after any
sequence of appends the segment equals the group-wise quantisation of all its
rows, so every array is compared bit for bit with ``oracle.quantize`` of the
rows so far, and attention over the growing segment is compared with the
oracle's masked, fake-quantised attention."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import oracle as ref  # noqa: E402
import paper_2609_32831_amd as uc  # noqa: E402
from gpu_util import TORCH, check_attention, dev, rand_rows, sm_scale  # noqa: E402

SCASES = [
    # B, Hq, Hkv, D, dtype, G, bits, N0, capacity, appended chunks
    (2, 28, 4, 128, "bf16", 64, 4, 100, 400, [1] * 70 + [50, 3, 1]),
    (1, 8, 2, 64, "f16", 32, 2, 0, 200, [1] * 40 + [33, 64, 1]),
    (1, 14, 2, 128, "bf16", 32, 8, 31, 300, [5, 64, 100, 1]),
    (1, 7, 1, 128, "bf16", 128, 4, 0, 256, [127, 1, 1, 127]),
]


def _case(**kw):
    print("CASE", " ".join(f"{k}={v}" for k, v in kw.items()), flush=True)


def _compare(seg, pk, B, Hkv, n, D, G, bits):
    """GPU packed segment (capacity layout) vs the oracle's quantisation of
    its n rows."""
    BH = B * Hkv
    n_full = G * (n // G)
    cap_full = seg.t["scale_v"].shape[2]
    rb = D * bits // 8
    ck = seg.t["codes_k"].cpu().numpy()
    cv = seg.t["codes_v"].cpu().numpy()
    for bh in range(BH):
        o = int(pk["code_off"][bh])
        g0 = bh * cap_full * rb
        assert np.array_equal(ck[g0:g0 + n_full * rb], pk["codes_k"][o:o + n_full * rb]), bh
        assert np.array_equal(cv[g0:g0 + n_full * rb], pk["codes_v"][o:o + n_full * rb]), bh
    for name, rows in (("scale_k", n_full // G), ("min_k", n_full // G), ("scale_v", n_full),
                       ("min_v", n_full)):
        g = seg.t[name].reshape(BH, -1, seg.t[name].shape[-1])[:, :rows].cpu().numpy()
        assert np.array_equal(g.view(np.uint32), pk[name].view(np.uint32)), name
    tl = n - n_full
    for name in ("tail_k", "tail_v"):
        g = seg.t[name].reshape(BH, -1, D)[:, :tl].contiguous()
        bits_t = torch.int32 if g.dtype == torch.float32 else torch.int16
        g = g.view(bits_t).cpu().numpy()
        r = np.ascontiguousarray(pk[name].reshape(BH, tl, D))
        assert np.array_equal(g, r.view(g.dtype)), name  # bit patterns


@pytest.mark.parametrize("case", SCASES, ids=[f"s{i}" for i in range(len(SCASES))])
def test_stream_append_equals_batch_quantisation(case):
    B, Hq, Hkv, D, dt, G, bits, N0, cap, chunks = case
    _case(test="stream_append", B=B, Hkv=Hkv, D=D, dtype=dt, G=G, bits=bits, N0=N0, cap=cap)
    BH = B * Hkv
    n_total = N0 + sum(chunks)
    assert n_total <= cap
    K = rand_rows(11, BH, n_total, D, dt, 2.0, outliers=(3,))
    V = rand_rows(12, BH, n_total, D, dt)
    Kd = dev(K, dt).reshape(B, Hkv, n_total, D)
    Vd = dev(V, dt).reshape(B, Hkv, n_total, D)
    shape = uc.make_shape(B, Hq, Hkv, D)
    seg = uc.packed_segment(B, Hkv, N0, D, G, TORCH[dt], bits=bits, capacity=cap)
    if N0:
        uc.uc_quantize_segment(shape, Kd[:, :, :N0].contiguous(), Vd[:, :, :N0].contiguous(), N0,
                               seg)
    n = N0
    checks = {N0 + sum(chunks[:i + 1]) for i in range(len(chunks)) if i % 17 == 0 or
              i >= len(chunks) - 3}
    for c in chunks:
        uc.uc_stream_append(shape, seg, Kd[:, :, n:n + c].contiguous(),
                            Vd[:, :, n:n + c].contiguous(), c)
        n += c
        assert seg.n_rows == n
        if n in checks:
            torch.cuda.synchronize()
            pk = ref.quantize(K[:, :n], V[:, :n], dt, G, [bits] * BH)
            _compare(seg, pk, B, Hkv, n, D, G, bits)
    # attention over a dense segment and the grown packed segment, through
    # every path (decode, prefill and the VALU kernels)
    kt = rand_rows(13, BH, 50, D, dt)
    vt = rand_rows(14, BH, 50, D, dt)
    dense = uc.dense_segment(dev(kt, dt).reshape(B, Hkv, 50, D), dev(vt, dt).reshape(B, Hkv, 50, D))
    pk = ref.quantize(K[:, :n], V[:, :n], dt, G, [bits] * BH)
    kh, vh = ref.dequant(pk, n, D, G, dt)
    Kl = np.concatenate([ref.widen(kt, dt), kh], axis=1).reshape(B, Hkv, -1, D)
    Vl = np.concatenate([ref.widen(vt, dt), vh], axis=1).reshape(B, Hkv, -1, D)
    seg_id = np.concatenate([np.zeros(50, np.int32), np.ones(n, np.int32)])
    sm = sm_scale(D)
    for M in (1, 40):
        q = rand_rows(15 + M, B * Hq, M, D, dt).reshape(B, Hq, M, D)
        o_ref, lse_ref, _, _ = ref.attend(ref.widen(q, dt), Kl, Vl, None, seg_id, 2, sm)
        for path in (uc.UC_PATH_AUTO, uc.UC_PATH_VALU):
            prev = uc.uc_set_path(path)
            try:
                o = torch.empty(B, Hq, M, D, device="cuda")
                lse = torch.empty(B, Hq, M, device="cuda")
                uc.uc_attend_mixed(shape, [dense, seg], dev(q, dt), M, sm, o, lse)
                torch.cuda.synchronize()
            finally:
                uc.uc_set_path(prev)
            check_attention(o.cpu().numpy(), o_ref, f"M={M} path={path}")
            assert np.allclose(lse.cpu().numpy(), lse_ref, rtol=1e-5, atol=1e-4)
