"""GPU parity of the fused decode step (Sec. 3.1: the new rows belong to the
protected segment; App. E: attention over the reassembled segments):
uc_attend_append equals uc_append_rows followed by uc_attend_mixed.  Checked
against the oracle's attention over the logical sequence after the append,
against the two-call sequence on the same inputs, and the protected segment's
rows bit for bit after every step."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import oracle as ref  # noqa: E402
import paper_2609_32831_amd as uc  # noqa: E402
from gpu_util import check_attention, dev, host_bytes, packed_from_oracle, rand_rows, sm_scale  # noqa: E402

D = 128


def _case(**kw):
    print("CASE", " ".join(f"{k}={v}" for k, v in kw.items()), flush=True)


def _build(B, Hkv, parts, cap, n0, seed):
    """Segments (dense / packed parts, then a dense tail of capacity cap with
    n0 live rows) and the logical K/V of the parts and of the tail's rows."""
    BH = B * Hkv
    segs, kh, vh, sid = [], [], [], []
    for j, p in enumerate(parts):
        s = seed * 10 + j
        if p[0] == "dense":
            n = p[1]
            k = rand_rows(s, BH, n, D, "bf16", outliers=(5,))
            v = rand_rows(s + 500, BH, n, D, "bf16")
            segs.append(uc.dense_segment(dev(k, "bf16").reshape(B, Hkv, n, D),
                                         dev(v, "bf16").reshape(B, Hkv, n, D)))
            kh.append(ref.widen(k, "bf16"))
            vh.append(ref.widen(v, "bf16"))
        else:
            n, G, bits = p[1], p[2], p[3]
            k = rand_rows(s, BH, n, D, "bf16", 2.0, outliers=(5,))
            v = rand_rows(s + 500, BH, n, D, "bf16")
            pk = ref.quantize(k, v, "bf16", G, [bits] * BH)
            segs.append(packed_from_oracle(B, Hkv, n, D, G, "bf16", pk))
            a, b = ref.dequant(pk, n, D, G, "bf16")
            kh.append(a)
            vh.append(b)
        sid.append(np.full(kh[-1].shape[1], j, np.int32))
    tk = rand_rows(seed * 10 + 9, BH, cap, D, "bf16")
    tv = rand_rows(seed * 10 + 8, BH, cap, D, "bf16")
    tail = uc.dense_segment(dev(tk, "bf16").reshape(B, Hkv, cap, D),
                            dev(tv, "bf16").reshape(B, Hkv, cap, D), n_rows=n0)
    segs.append(tail)
    return segs, kh, vh, sid, tk[:, :n0], tv[:, :n0]


def _oracle(q, B, Hkv, kh, vh, sid, tk, tv, n_segs, sm):
    K = np.concatenate(kh + [ref.widen(tk, "bf16")], axis=1).reshape(B, Hkv, -1, D)
    V = np.concatenate(vh + [ref.widen(tv, "bf16")], axis=1).reshape(B, Hkv, -1, D)
    seg_id = np.concatenate(sid + [np.full(tk.shape[1], n_segs - 1, np.int32)])
    return ref.attend(ref.widen(q, "bf16"), K, V, None, seg_id, n_segs, sm)


CASES = [
    # B, Hq, Hkv, M, parts, tail capacity, tail rows before, rows per step, steps
    (2, 28, 4, 1, [("dense", 300), ("packed", 200, 64, 4)], 40, 5, 1, 6),
    (1, 28, 4, 2, [("packed", 130, 32, 2), ("dense", 1000)], 64, 0, 3, 4),
    (3, 14, 2, 1, [("dense", 17)], 70, 31, 2, 5),   # tail rows cross a 32-row tile
    (1, 28, 4, 1, [], 8, 0, 1, 3),                   # the tail alone, from empty
]


@pytest.mark.parametrize("case", CASES, ids=[f"a{i}" for i in range(len(CASES))])
def test_attend_append_matches_two_calls_and_oracle(case):
    B, Hq, Hkv, M, parts, cap, n0, n_new, steps = case
    _case(test="attend_append", B=B, Hq=Hq, Hkv=Hkv, M=M, parts=parts, cap=cap, n0=n0,
          n_new=n_new, steps=steps)
    BH = B * Hkv
    shape = uc.make_shape(B, Hq, Hkv, D)
    sm = sm_scale(D)
    segs, kh, vh, sid, tk, tv = _build(B, Hkv, parts, cap, n0, seed=len(parts) + cap)
    # a second set of segments for the two-call sequence: same parts, own tail
    segs2, _, _, _, _, _ = _build(B, Hkv, parts, cap, n0, seed=len(parts) + cap)
    ns = len(segs)
    for step in range(steps):
        kn = rand_rows(700 + step, BH, n_new, D, "bf16")
        vn = rand_rows(800 + step, BH, n_new, D, "bf16")
        q = rand_rows(900 + step, B * Hq, M, D, "bf16").reshape(B, Hq, M, D)
        kd = dev(kn, "bf16").reshape(B, Hkv, n_new, D)
        vd = dev(vn, "bf16").reshape(B, Hkv, n_new, D)
        o = torch.empty(B, Hq, M, D, device="cuda")
        lse = torch.empty(B, Hq, M, device="cuda")
        pos = segs[-1].n_rows
        uc.uc_attend_append(shape, segs, ns - 1, kd, vd, n_new, dev(q, "bf16"), M, sm, o, lse)
        assert segs[-1].n_rows == pos + n_new
        o2 = torch.empty(B, Hq, M, D, device="cuda")
        uc.uc_append_rows(shape, kd, vd, n_new, segs2[-1], pos)
        segs2[-1].n_rows = pos + n_new
        uc.uc_attend_mixed(shape, segs2, dev(q, "bf16"), M, sm, o2)
        torch.cuda.synchronize()
        tk = np.concatenate([tk, kn], axis=1)
        tv = np.concatenate([tv, vn], axis=1)
        o_ref, lse_ref, _, _ = _oracle(q, B, Hkv, kh, vh, sid, tk, tv, ns, sm)
        check_attention(o.cpu().numpy(), o_ref, f"step {step}")
        assert np.allclose(lse.cpu().numpy(), lse_ref, rtol=1e-5, atol=1e-4), step
        # the same computation up to summation order
        assert np.abs(o.cpu().numpy() - o2.cpu().numpy()).max() < 5e-4, step
        # the protected segment holds every row appended so far, bit for bit
        n = pos + n_new
        got_k = host_bytes(segs[-1].t["k"]).reshape(BH, cap, D)[:, :n]
        got_v = host_bytes(segs[-1].t["v"]).reshape(BH, cap, D)[:, :n]
        assert np.array_equal(got_k, tk.view(np.uint16)), step
        assert np.array_equal(got_v, tv.view(np.uint16)), step
        # rows past the live ones are untouched
        init = rand_rows((len(parts) + cap) * 10 + 9, BH, cap, D, "bf16")
        rest = host_bytes(segs[-1].t["k"]).reshape(BH, cap, D)[:, n:]
        assert np.array_equal(rest, init[:, n:].view(np.uint16)), step


def test_attend_append_two_call_paths():
    """Per-segment outputs, the VALU path and a full segment list take the
    two-call route inside the library; results and stored rows agree."""
    B, Hq, Hkv, M = 1, 28, 4, 1
    _case(test="attend_append_fallbacks")
    BH = B * Hkv
    shape = uc.make_shape(B, Hq, Hkv, D)
    sm = sm_scale(D)
    for mode in ("seg_lse", "valu", "max_segments"):
        parts = [("dense", 100), ("packed", 128, 64, 4)]
        if mode == "max_segments":
            parts = [("dense", 20 + 7 * i) for i in range(uc.UC_MAX_SEGMENTS - 1)]
        segs, kh, vh, sid, tk, tv = _build(B, Hkv, parts, 16, 3, seed=41)
        ns = len(segs)
        kn = rand_rows(61, BH, 2, D, "bf16")
        vn = rand_rows(62, BH, 2, D, "bf16")
        q = rand_rows(63, B * Hq, M, D, "bf16").reshape(B, Hq, M, D)
        o = torch.empty(B, Hq, M, D, device="cuda")
        lse = torch.empty(B, Hq, M, device="cuda")
        sl = torch.empty(B, Hq, M, ns, device="cuda") if mode == "seg_lse" else None
        prev = uc.uc_set_path(uc.UC_PATH_VALU if mode == "valu" else uc.UC_PATH_AUTO)
        try:
            uc.uc_attend_append(shape, segs, ns - 1, dev(kn, "bf16").reshape(B, Hkv, 2, D),
                                dev(vn, "bf16").reshape(B, Hkv, 2, D), 2, dev(q, "bf16"), M, sm,
                                o, lse, sl)
            torch.cuda.synchronize()
        finally:
            uc.uc_set_path(prev)
        tk = np.concatenate([tk, kn], axis=1)
        tv = np.concatenate([tv, vn], axis=1)
        o_ref, lse_ref, sl_ref, _ = _oracle(q, B, Hkv, kh, vh, sid, tk, tv, ns, sm)
        check_attention(o.cpu().numpy(), o_ref, mode)
        assert np.allclose(lse.cpu().numpy(), lse_ref, rtol=1e-5, atol=1e-4), mode
        if sl is not None:
            got = sl.cpu().numpy()
            fin = np.isfinite(sl_ref)
            assert np.array_equal(np.isfinite(got), fin)
            assert np.allclose(got[fin], sl_ref[fin], rtol=1e-5, atol=1e-4)
        assert segs[-1].n_rows == 5
        got_k = host_bytes(segs[-1].t["k"]).reshape(BH, 16, D)[:, :5]
        assert np.array_equal(got_k, tk.view(np.uint16)), mode


def test_attend_append_kernel_events():
    """The timing hook brackets the fused launch inside the call's own pair,
    and its outputs are those of an untimed call."""
    B, Hq, Hkv = 1, 28, 4
    _case(test="attend_append_events")
    shape = uc.make_shape(B, Hq, Hkv, D)
    kn = dev(rand_rows(1, Hkv, 1, D, "bf16"), "bf16").reshape(B, Hkv, 1, D)
    q = dev(rand_rows(2, Hq, 1, D, "bf16"), "bf16").reshape(B, Hq, 1, D)
    outs = []
    for timed in (False, True):
        segs, _, _, _, _, _ = _build(B, Hkv, [("dense", 4096)], 8, 0, seed=5)
        o = torch.empty(B, Hq, 1, D, device="cuda")
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
        for e in ev:
            e.record()
        torch.cuda.synchronize()
        ev[0].record()
        if timed:
            uc.uc_set_kernel_events(ev[2], ev[3])
        uc.uc_attend_append(shape, segs, 1, kn, kn, 1, q, 1, sm_scale(D), o)
        ev[1].record()
        torch.cuda.synchronize()
        outs.append(o)
    call_ms, kern_ms = ev[0].elapsed_time(ev[1]), ev[2].elapsed_time(ev[3])
    assert 0.0 < kern_ms <= call_ms
    assert torch.equal(outs[0], outs[1])


@pytest.mark.parametrize("case", CASES[:3], ids=[f"p{i}" for i in range(3)])
@pytest.mark.parametrize("path", ["auto", "valu"])
def test_plan_steps_match_attend_append(case, path):
    """Decode steps through an execution plan (uc_plan_create /
    uc_plan_attend_append, App. E "Cached metadata and execution plans")
    equal the same steps through uc_attend_append bit for bit -- outputs,
    lse and the stored tail rows -- on the matrix-core path and on the VALU
    path (which runs the two-call route), and match the oracle."""
    B, Hq, Hkv, M, parts, cap, n0, n_new, steps = case
    _case(test="plan_steps", B=B, Hq=Hq, Hkv=Hkv, M=M, parts=parts, cap=cap, n0=n0,
          n_new=n_new, steps=steps, path=path)
    BH = B * Hkv
    shape = uc.make_shape(B, Hq, Hkv, D)
    sm = sm_scale(D)
    seed = len(parts) + cap
    segs, kh, vh, sid, tk, tv = _build(B, Hkv, parts, cap, n0, seed=seed)
    segs2, _, _, _, _, _ = _build(B, Hkv, parts, cap, n0, seed=seed)
    ns = len(segs)
    prev = uc.uc_set_path(uc.UC_PATH_VALU if path == "valu" else uc.UC_PATH_AUTO)
    try:
        plan = uc.AttendPlan(shape, segs, ns - 1, torch.bfloat16, M, sm)
        assert plan.tail_rows == n0
        ws2 = torch.empty(uc.uc_attend_workspace_size(
            shape, segs2[:-1] + [uc.dense_segment(segs2[-1].t["k"], segs2[-1].t["v"])],
            uc.UC_BF16, M), dtype=torch.uint8, device="cuda")
        for step in range(steps):
            kn = rand_rows(700 + step, BH, n_new, D, "bf16")
            vn = rand_rows(800 + step, BH, n_new, D, "bf16")
            q = rand_rows(900 + step, B * Hq, M, D, "bf16").reshape(B, Hq, M, D)
            kd = dev(kn, "bf16").reshape(B, Hkv, n_new, D)
            vd = dev(vn, "bf16").reshape(B, Hkv, n_new, D)
            qd = dev(q, "bf16")
            o, o2 = (torch.empty(B, Hq, M, D, device="cuda") for _ in range(2))
            lse, lse2 = (torch.empty(B, Hq, M, device="cuda") for _ in range(2))
            # the plan takes raw device addresses as well as tensors
            plan.attend_append(kd.data_ptr(), vd, n_new, qd, o, lse)
            uc.uc_attend_append(shape, segs2, ns - 1, kd, vd, n_new, qd, M, sm, o2, lse2, ws=ws2)
            torch.cuda.synchronize()
            assert plan.tail_rows == segs[-1].n_rows == segs2[-1].n_rows == n0 + (step + 1) * n_new
            assert torch.equal(o, o2) and torch.equal(lse, lse2), step
            n = segs[-1].n_rows
            assert torch.equal(segs[-1].t["k"][:, :, :n], segs2[-1].t["k"][:, :, :n]), step
            assert torch.equal(segs[-1].t["v"][:, :, :n], segs2[-1].t["v"][:, :, :n]), step
            tk = np.concatenate([tk, kn], axis=1)
            tv = np.concatenate([tv, vn], axis=1)
            o_ref, lse_ref, _, _ = _oracle(q, B, Hkv, kh, vh, sid, tk, tv, ns, sm)
            check_attention(o.cpu().numpy(), o_ref, f"step {step}")
        plan.close()
    finally:
        uc.uc_set_path(prev)
