"""GPU parity of attention through an execution plan of a frozen layout
(uc_plan_create / uc_plan_attend; App. E, "Cached metadata and execution
plans", and packed KV dequantised into a reusable workspace): every call
equals uc_attend_mixed on the same segments bit for bit -- outputs, lse and
per-segment lse -- on the multi-query matrix-core path (whose workspace
preparation the later calls reuse), the decode path and the VALU path; after
a segment is rewritten, uc_plan_invalidate makes the next call see the new
contents.  Each case also matches the oracle."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import oracle as ref  # noqa: E402
import paper_2609_32831_amd as uc  # noqa: E402
from gpu_util import check_attention, dev, packed_from_oracle, rand_rows, sm_scale  # noqa: E402

D = 128


def _segments(B, Hkv, seed):
    """A dense segment, a packed int4 segment with a residual tail and a
    dense segment with spare capacity; their logical K/V for the oracle."""
    BH = B * Hkv
    segs, kh, vh, sid = [], [], [], []
    k = rand_rows(seed, BH, 300, D, "bf16", outliers=(5,))
    v = rand_rows(seed + 1, BH, 300, D, "bf16")
    segs.append(uc.dense_segment(dev(k, "bf16").reshape(B, Hkv, 300, D),
                                 dev(v, "bf16").reshape(B, Hkv, 300, D)))
    kh.append(ref.widen(k, "bf16"))
    vh.append(ref.widen(v, "bf16"))
    n = 200
    k = rand_rows(seed + 2, BH, n, D, "bf16", 2.0, outliers=(5,))
    v = rand_rows(seed + 3, BH, n, D, "bf16")
    pk = ref.quantize(k, v, "bf16", 64, [4] * BH)
    segs.append(packed_from_oracle(B, Hkv, n, D, 64, "bf16", pk))
    a, b = ref.dequant(pk, n, D, 64, "bf16")
    kh.append(a)
    vh.append(b)
    k = rand_rows(seed + 4, BH, 40, D, "bf16")
    v = rand_rows(seed + 5, BH, 40, D, "bf16")
    segs.append(uc.dense_segment(dev(k, "bf16").reshape(B, Hkv, 40, D),
                                 dev(v, "bf16").reshape(B, Hkv, 40, D), n_rows=33))
    kh.append(ref.widen(k[:, :33], "bf16"))
    vh.append(ref.widen(v[:, :33], "bf16"))
    for i, x in enumerate(kh):
        sid.append(np.full(x.shape[1], i, np.int32))
    return segs, kh, vh, sid


def _oracle(q, B, Hkv, kh, vh, sid, sm):
    K = np.concatenate(kh, axis=1).reshape(B, Hkv, -1, D)
    V = np.concatenate(vh, axis=1).reshape(B, Hkv, -1, D)
    return ref.attend(ref.widen(q, "bf16"), K, V, None, np.concatenate(sid), len(kh), sm)


@pytest.mark.parametrize("M,path,kernel", [(64, "auto", "prefill_mfma"),
                                           (1, "auto", "decode_mfma"),
                                           (64, "valu", "attend_valu")])
def test_plan_attend_matches_attend_mixed(M, path, kernel):
    B, Hq, Hkv = 2, 28, 4
    print(f"CASE plan_attend M={M} path={path}", flush=True)
    shape = uc.make_shape(B, Hq, Hkv, D)
    sm = sm_scale(D)
    segs, kh, vh, sid = _segments(B, Hkv, seed=11)
    ns = len(segs)
    prev = uc.uc_set_path(uc.UC_PATH_VALU if path == "valu" else uc.UC_PATH_AUTO)
    try:
        plan = uc.AttendPlan(shape, segs, None, torch.bfloat16, M, sm)
        ws2 = torch.empty(uc.uc_attend_workspace_size(shape, segs, uc.UC_BF16, M),
                          dtype=torch.uint8, device="cuda")
        for call in range(3):
            q = rand_rows(50 + call, B * Hq, M, D, "bf16").reshape(B, Hq, M, D)
            qd = dev(q, "bf16")
            o, o2 = (torch.empty(B, Hq, M, D, device="cuda") for _ in range(2))
            lse, lse2 = (torch.empty(B, Hq, M, device="cuda") for _ in range(2))
            sl, sl2 = (torch.empty(B, Hq, M, ns, device="cuda") for _ in range(2))
            plan.attend(qd, o, lse, sl)
            assert uc.uc_last_kernel() == kernel
            uc.uc_attend_mixed(shape, segs, qd, M, sm, o2, lse2, sl2, ws=ws2)
            torch.cuda.synchronize()
            assert torch.equal(o, o2) and torch.equal(lse, lse2) and torch.equal(sl, sl2), call
            o_ref, lse_ref, _, _ = _oracle(q, B, Hkv, kh, vh, sid, sm)
            check_attention(o.cpu().numpy(), o_ref, f"call {call}")
            assert np.allclose(lse.cpu().numpy(), lse_ref, rtol=1e-5, atol=1e-4)
        # rewrite the packed segment's codes and the dense V rows in place; the
        # plan sees the new contents after uc_plan_invalidate
        BH = B * Hkv
        k = rand_rows(90, BH, 200, D, "bf16", 2.0)
        v = rand_rows(91, BH, 200, D, "bf16")
        pk = ref.quantize(k, v, "bf16", 64, [4] * BH)
        new = packed_from_oracle(B, Hkv, 200, D, 64, "bf16", pk)
        for name, t in new.t.items():
            if t is not None:
                segs[1].t[name].copy_(t)
        kh[1], vh[1] = ref.dequant(pk, 200, D, 64, "bf16")
        v0 = rand_rows(92, BH, 300, D, "bf16")
        segs[0].t["v"].copy_(dev(v0, "bf16").reshape(B, Hkv, 300, D))
        vh[0] = ref.widen(v0, "bf16")
        plan.invalidate()
        q = rand_rows(60, B * Hq, M, D, "bf16").reshape(B, Hq, M, D)
        o, o2 = (torch.empty(B, Hq, M, D, device="cuda") for _ in range(2))
        plan.attend(dev(q, "bf16"), o)
        uc.uc_attend_mixed(shape, segs, dev(q, "bf16"), M, sm, o2, ws=ws2)
        torch.cuda.synchronize()
        assert torch.equal(o, o2)
        o_ref, _, _, _ = _oracle(q, B, Hkv, kh, vh, sid, sm)
        check_attention(o.cpu().numpy(), o_ref, "after invalidate")
        plan.close()
    finally:
        uc.uc_set_path(prev)
