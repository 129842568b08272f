"""Host-side checks of the C ABI that need no GPU: every declared symbol is
exported, argument validation rejects bad calls before any launch, and the
host-only accounting / budget helpers agree with the oracle."""
import ctypes
import math
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def uc():
    import paper_2609_32831_amd as m
    return m


def declared_functions():
    src = open(os.path.join(ROOT, "include", "unicache.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(uc_[a-z_]+)\s*\(", src)))


def test_every_declared_symbol_is_exported(uc):
    names = declared_functions()
    assert len(names) >= 18
    lib = ctypes.CDLL(uc.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n


def test_struct_layout_matches_header(uc):
    # offsets follow from the field order in unicache.h on LP64
    assert ctypes.sizeof(uc.uc_shape) == 16
    assert uc.uc_segment.k.offset == 16 and uc.uc_segment.group.offset == 40
    assert uc.uc_segment.codes_bytes.offset == 64
    assert uc.uc_segment.tail_v.offset == 128 and ctypes.sizeof(uc.uc_segment) == 136


FAKE = 0x100000  # aligned non-null address; validation never dereferences it


def _dense(uc, n, dt=2, k=FAKE, v=FAKE, stride=0):
    return uc.uc_segment(kind=uc.UC_SEG_DENSE, dtype=dt, n_rows=n, row_stride=stride, k=k, v=v)


def _packed(uc, n, G=64, bits=4, D=128, BH=1, **kw):
    nf = G * (n // G)
    d = dict(kind=uc.UC_SEG_PACKED, dtype=2, n_rows=n, group=G, bits=bits,
             codes_bytes=BH * nf * D * bits // 8, codes_k=FAKE, codes_v=FAKE, scale_k=FAKE,
             min_k=FAKE, scale_v=FAKE, min_v=FAKE, tail_k=FAKE, tail_v=FAKE)
    d.update(kw)
    return uc.uc_segment(**d)


def _attend(uc, shape, segs, M=1, q=FAKE, o=FAKE, ws=FAKE, ws_bytes=1 << 40, scale=0.1):
    arr = (uc.uc_segment * len(segs))(*segs)
    return uc.lib.uc_attend_mixed(ctypes.byref(shape), arr, len(segs), q, uc.UC_BF16, M,
                                  ctypes.c_float(scale), o, None, None, ws, ws_bytes, None)


def test_attend_validation(uc):
    good = uc.uc_shape(1, 4, 1, 128)
    E = uc.UC_E_INVALID
    assert _attend(uc, uc.uc_shape(1, 4, 1, 96), [_dense(uc, 8)]) == E  # D
    assert "D must be 64 or 128" in uc.uc_last_error()
    assert _attend(uc, uc.uc_shape(1, 6, 4, 128), [_dense(uc, 8)]) == E  # Hq % Hkv
    assert _attend(uc, uc.uc_shape(0, 4, 1, 128), [_dense(uc, 8)]) == E
    assert _attend(uc, good, [_dense(uc, 0)]) == E  # no rows at all
    assert _attend(uc, good, [_dense(uc, 8)], M=0) == E
    assert _attend(uc, good, [_dense(uc, 8)], q=None) == E
    assert _attend(uc, good, [_dense(uc, 8)], o=None) == E
    assert _attend(uc, good, [_dense(uc, 8, k=None)]) == E
    assert _attend(uc, good, [_dense(uc, 8, k=FAKE + 8)]) == E  # misaligned
    assert _attend(uc, good, [_dense(uc, 8, stride=4)]) == E  # stride < rows
    assert _attend(uc, good, [_dense(uc, 8, dt=7)]) == E
    assert _attend(uc, good, [_dense(uc, 8)], scale=0.0) == E
    assert _attend(uc, good, [_dense(uc, 8)] * 9) == E  # too many segments
    assert _attend(uc, good, [_packed(uc, 128, bits=3)]) == E
    assert _attend(uc, good, [_packed(uc, 128, G=48)]) == E
    assert _attend(uc, good, [_packed(uc, 128, G=256)]) == E
    assert _attend(uc, good, [_packed(uc, 128, codes_bytes=10)]) == E
    assert _attend(uc, good, [_packed(uc, 100, tail_k=None)]) == E  # tail rows, no tail
    assert _attend(uc, good, [_packed(uc, 128, scale_v=None)]) == E
    assert _attend(uc, good, [_packed(uc, 128, head_bits=FAKE)]) == E  # no code_off
    # with per-head widths, bits is their bound and must still be a valid width
    assert _attend(uc, good, [_packed(uc, 128, bits=5, head_bits=FAKE, code_off=FAKE)]) == E
    # a workspace that is too small is its own status
    assert _attend(uc, good, [_dense(uc, 8)], ws_bytes=16) == uc.UC_E_WORKSPACE
    assert uc.uc_status_string(uc.UC_E_WORKSPACE).startswith("UC_E_WORKSPACE")


def test_select_quantize_append_validation(uc):
    L, E = uc.lib, uc.UC_E_INVALID
    f = lambda *a: L.uc_select_keep(*a)
    assert f(FAKE, 4, 10, 11, 0, FAKE, None, None, None, None, 2, 128, None, 0, None) == E
    assert f(FAKE, 4, 10, 5, 6, FAKE, None, None, None, None, 2, 128, None, 0, None) == E
    assert f(FAKE, 4, 10, -1, 0, FAKE, None, None, None, None, 2, 128, None, 0, None) == E
    assert f(FAKE, 4, 10, 5, 0, None, None, None, None, None, 2, 128, None, 0, None) == E
    assert f(FAKE, 4, 10, 5, 0, FAKE, FAKE, None, FAKE, FAKE, 2, 128, None, 0, None) == E
    assert f(FAKE, 4, 10, 5, 0, FAKE, FAKE, FAKE, FAKE, FAKE, 2, 96, None, 0, None) == E
    # k = 0 is a valid no-op
    assert f(None, 4, 10, 0, 0, None, None, None, None, None, 2, 128, None, 0, None) == uc.UC_OK
    sh = uc.uc_shape(1, 4, 1, 128)
    out = _packed(uc, 128)
    assert L.uc_quantize_segment(ctypes.byref(sh), FAKE, FAKE, 2, 100, ctypes.byref(out), None) == E
    out_f = _packed(uc, 128, dtype=0)
    assert L.uc_quantize_segment(ctypes.byref(sh), FAKE, FAKE, 2, 128, ctypes.byref(out_f), None) == E
    assert L.uc_quantize_segment(ctypes.byref(sh), None, FAKE, 2, 128, ctypes.byref(out), None) == E
    dense = _dense(uc, 4, stride=8)
    assert L.uc_append_rows(ctypes.byref(sh), FAKE, FAKE, 5, ctypes.byref(dense), 4, None) == E
    assert L.uc_append_rows(ctypes.byref(sh), FAKE, FAKE, 1, ctypes.byref(out), 0, None) == E
    assert L.uc_segment_mass(ctypes.byref(sh), 0, 1, FAKE, FAKE, FAKE, None) == E


def test_score_columns_validation(uc):
    """uc_score_columns checks its row normalisers and workspace before any
    launch, and enqueues nothing when neither scores nor masses are asked for
    (so the last call runs without a GPU)."""
    L, E = uc.lib, uc.UC_E_INVALID
    sh = uc.uc_shape(1, 28, 4, 128)
    segs = (uc.uc_segment * 2)(_dense(uc, 100), _packed(uc, 256, BH=4))
    need = L.uc_score_workspace_size(ctypes.byref(sh), segs, 2, 32)
    assert need > 0
    outs = (ctypes.c_void_p * 2)(FAKE, None)

    def f(lse=FAKE, ld=64, W=32, out=outs, mass=None, ws_bytes=need, q_ld=32):
        return L.uc_score_columns(ctypes.byref(sh), segs, 2, FAKE, q_ld, uc.UC_BF16, W,
                                  ctypes.c_float(0.1), lse, ld, out, mass, FAKE, ws_bytes, None)
    assert f(lse=None) == E
    assert "row_lse" in uc.uc_last_error()
    assert f(ld=31) == E
    assert f(q_ld=31) == E
    assert f(W=0) == E
    assert f(ws_bytes=need - 1) == uc.UC_E_WORKSPACE
    assert f(out=None, mass=None) == uc.UC_OK  # nothing asked for: no work


def test_evict_step_validation(uc):
    """uc_evict_step rejects bad segments before any launch; an empty
    current segment is a valid no-op (no launch, so it runs without a GPU)."""
    L, E = uc.lib, uc.UC_E_INVALID
    sh = uc.uc_shape(1, 28, 4, 128)
    BUF = 1 << 30  # far from FAKE: no overlap

    def f(cur, out, scores=FAKE, k_dev=FAKE):
        return L.uc_evict_step(ctypes.byref(sh), scores, ctypes.byref(cur), k_dev,
                               ctypes.byref(out), None)
    cur = _dense(uc, 100, stride=128)
    out = _dense(uc, 0, k=BUF, v=BUF + (1 << 24), stride=128)
    out.idx = BUF + (1 << 25)
    assert f(cur, _dense(uc, 0, k=BUF, v=BUF + (1 << 24), stride=99)) == E  # stride < N
    assert "row_stride" in uc.uc_last_error()
    assert f(cur, _packed(uc, 128)) == E
    assert f(_packed(uc, 128), out) == E
    o2 = _dense(uc, 0, dt=1, k=BUF, v=BUF + (1 << 24), stride=128)
    o2.idx = BUF + (1 << 25)
    assert f(cur, o2) == E  # dtype
    assert f(cur, out, scores=None) == E
    assert f(cur, out, k_dev=None) == E
    o3 = _dense(uc, 0, k=BUF, v=BUF + (1 << 24), stride=128)
    assert f(cur, o3) == E  # out idx NULL
    o4 = _dense(uc, 0, k=FAKE, v=BUF + (1 << 24), stride=128)
    o4.idx = BUF + (1 << 25)
    assert f(cur, o4) == E  # out rows overlap cur rows
    assert "overlap" in uc.uc_last_error()
    assert f(_dense(uc, 0, stride=8), out) == uc.UC_OK  # no rows: nothing to do


def _attend_append(uc, shape, segs, tail, n_new, kn=FAKE, vn=FAKE, q=FAKE, M=1, ws_bytes=1 << 40):
    arr = (uc.uc_segment * len(segs))(*segs)
    return uc.lib.uc_attend_append(ctypes.byref(shape), arr, len(segs), tail, kn, vn, n_new, q,
                                   uc.UC_BF16, M, ctypes.c_float(0.1), FAKE, None, None, FAKE,
                                   ws_bytes, None)


def test_attend_append_validation(uc):
    sh = uc.uc_shape(1, 4, 1, 128)
    E = uc.UC_E_INVALID
    tail = _dense(uc, 7, stride=8)
    segs = [_dense(uc, 64), tail]
    assert _attend_append(uc, sh, segs, 2, 1) == E  # tail index out of range
    assert _attend_append(uc, sh, segs, -1, 1) == E
    assert _attend_append(uc, sh, [_dense(uc, 64), _packed(uc, 128)], 1, 1) == E  # not dense
    assert "not dense" in uc.uc_last_error()
    assert _attend_append(uc, sh, segs, 1, -1) == E
    assert _attend_append(uc, sh, segs, 1, 2) == E  # 7 + 2 rows > capacity 8
    assert "exceed row_stride" in uc.uc_last_error()
    assert _attend_append(uc, sh, [_dense(uc, 64), _dense(uc, 3)], 1, 1) == E  # no capacity
    assert _attend_append(uc, sh, segs, 1, 1, kn=None) == E
    assert _attend_append(uc, sh, segs, 1, 1, vn=FAKE + 4) == E  # misaligned
    assert _attend_append(uc, sh, segs, 1, 1, q=None) == E
    assert _attend_append(uc, sh, segs, 1, 1, M=0) == E
    assert _attend_append(uc, sh, segs, 1, 1, ws_bytes=16) == uc.UC_E_WORKSPACE
    # an empty tail with nothing else to attend is an error only without new rows
    assert _attend_append(uc, sh, [_dense(uc, 0, stride=4)], 0, 0) == E


def test_plan_validation(uc):
    """uc_plan_create validates as uc_attend_append does; a plan's step checks
    its own pointers, capacity and workspace before any launch, and a
    rejected step leaves the tail's row count alone."""
    sh = uc.uc_shape(1, 4, 1, 128)
    E = uc.UC_E_INVALID
    L = uc.lib

    def create(segs, tail, M=1, scale=0.1, q_dt=None):
        h = ctypes.c_void_p()
        arr = (uc.uc_segment * len(segs))(*segs)
        st = L.uc_plan_create(ctypes.byref(sh), arr, len(segs), tail,
                              uc.UC_BF16 if q_dt is None else q_dt, M, ctypes.c_float(scale),
                              ctypes.byref(h))
        return st, h

    segs = [_dense(uc, 64), _dense(uc, 7, stride=8)]
    assert create(segs, 2)[0] == E  # tail out of range
    assert create(segs, 0)[0] == E  # tail without a row capacity
    assert create([_dense(uc, 64), _packed(uc, 128)], 1)[0] == E  # tail not dense
    assert create(segs, 1, M=0)[0] == E
    assert create(segs, 1, scale=-1.0)[0] == E
    assert create(segs, 1, q_dt=99)[0] == E
    st, h = create([_dense(uc, 64, stride=64)] * uc.UC_MAX_SEGMENTS, 1)
    assert st == uc.UC_E_UNSUPPORTED and not h
    assert L.uc_plan_create(ctypes.byref(sh), (uc.uc_segment * 2)(*segs), 2, 1, uc.UC_BF16, 1,
                            ctypes.c_float(0.1), None) == E
    st, h = create(segs, 1)
    assert st == uc.UC_OK and h
    try:
        assert L.uc_plan_tail_rows(h) == 7
        need = L.uc_plan_workspace_size(h)
        assert need > 0
        # the workspace covers the tail at its capacity: the same as
        # uc_attend_workspace_size with 8 tail rows
        full = (uc.uc_segment * 2)(_dense(uc, 64), _dense(uc, 8, stride=8))
        assert need >= L.uc_attend_workspace_size(ctypes.byref(sh), full, 2, uc.UC_BF16, 1)

        def step(n_new, kn=FAKE, vn=FAKE, q=FAKE, o=FAKE, ws_bytes=1 << 40):
            return L.uc_plan_attend_append(h, kn, vn, n_new, q, o, None, FAKE, ws_bytes, None)

        assert step(2) == E  # 7 + 2 rows > capacity 8
        assert "exceed row_stride" in uc.uc_last_error()
        assert step(-1) == E
        assert step(1, kn=None) == E
        assert step(1, vn=FAKE + 4) == E  # misaligned
        assert step(1, q=None) == E
        assert step(1, o=None) == E
        assert step(1, ws_bytes=need - 1) == uc.UC_E_WORKSPACE
        assert L.uc_plan_tail_rows(h) == 7  # no rejected step moved the tail
        assert L.uc_plan_attend_append(None, FAKE, FAKE, 1, FAKE, FAKE, None, FAKE, 1 << 40,
                                       None) == E
    finally:
        assert L.uc_plan_destroy(h) == uc.UC_OK
    assert L.uc_plan_destroy(None) == uc.UC_OK
    assert L.uc_plan_tail_rows(None) == -1 and L.uc_plan_workspace_size(None) == 0
    assert L.uc_plan_invalidate(None) == E
    assert L.uc_plan_attend(None, FAKE, FAKE, None, None, FAKE, 1 << 40, None) == E
    # a plan without a tail: attention only
    st, h = create(segs, -1, M=64)
    assert st == uc.UC_OK and h
    try:
        assert L.uc_plan_tail_rows(h) == -1
        need = L.uc_plan_workspace_size(h)
        assert need >= L.uc_attend_workspace_size(ctypes.byref(sh), (uc.uc_segment * 2)(*segs),
                                                  2, uc.UC_BF16, 64)
        assert L.uc_plan_attend_append(h, FAKE, FAKE, 1, FAKE, FAKE, None, FAKE, 1 << 40,
                                       None) == E
        assert "no tail" in uc.uc_last_error()
        assert L.uc_plan_attend(h, None, FAKE, None, None, FAKE, 1 << 40, None) == E
        assert L.uc_plan_attend(h, FAKE, FAKE, None, None, FAKE, need - 1,
                                None) == uc.UC_E_WORKSPACE
        assert L.uc_plan_invalidate(h) == uc.UC_OK
    finally:
        L.uc_plan_destroy(h)
    assert create(segs, -2)[0] == E


def test_dynamic_budget_entry_validation(uc):
    sh = uc.uc_shape(1, 4, 2, 128)
    dense = _dense(uc, 64)
    # dequantisation needs a packed segment; compose needs non-overlapping out
    assert uc.lib.uc_dequantize_segment(ctypes.byref(sh), ctypes.byref(dense), 16, 16, None) == \
        uc.UC_E_INVALID
    assert uc.lib.uc_compose_index(4096, 8, 8192, -1, 4, 16384, None) == uc.UC_E_INVALID
    assert uc.lib.uc_compose_index(4096, 8, 8192, 2, 4, 4096 + 16, None) == uc.UC_E_INVALID
    assert uc.lib.uc_compose_index(4096, 8, 8192, 2, 0, 16384, None) == uc.UC_OK
    with pytest.raises(uc.UcError):
        uc.uc_quant_config(1e6, 4096, 96, uc.UC_BF16, 4)
    assert uc.lib.uc_quant_config(1e6, 4096, 128, uc.UC_BF16, 4, 9, None, None) == -1


def test_kernel_events_setting(uc):
    # null events are accepted and mean "record nothing"; the setting is
    # cleared by the next attention call even when that call fails validation
    uc.uc_set_kernel_events(None, None)
    uc.uc_set_kernel_events(None, None)


def test_workspace_size_helpers(uc):
    sh = uc.uc_shape(2, 8, 2, 128)
    segs = [_dense(uc, 300), _packed(uc, 200, BH=4)]
    arr = (uc.uc_segment * 2)(*segs)
    assert uc.lib.uc_attend_workspace_size(ctypes.byref(sh), arr, 2, uc.UC_BF16, 1) > 0
    assert uc.lib.uc_score_workspace_size(ctypes.byref(sh), arr, 2, 16) > 0
    # invalid description -> 0
    bad = uc.uc_shape(2, 8, 3, 128)
    assert uc.lib.uc_attend_workspace_size(ctypes.byref(bad), arr, 2, uc.UC_BF16, 1) == 0


def test_host_helpers_agree_with_oracle(uc, ref):
    rng = np.random.default_rng(0)
    for _ in range(200):
        rows = int(rng.integers(0, 70000))
        D = int(rng.choice([64, 128]))
        dt = int(rng.integers(0, 3))
        name = ["f32", "f16", "bf16"][dt]
        G = int(rng.choice([8, 16, 32, 64]))
        b = int(rng.choice([2, 4, 8]))
        assert uc.uc_dense_bytes(rows, D, dt) == ref.dense_bytes(rows, D, name)
        assert uc.uc_evicted_bytes(rows, D, dt) == ref.evicted_bytes(rows, D, name)
        assert uc.uc_packed_bytes(rows, D, G, b, dt) == ref.packed_bytes(rows, D, G, b, name)
        budget = float(rng.uniform(0, 4e7))
        fixed = float(rng.uniform(0, 2e7))
        assert uc.uc_evict_rows_for_budget(budget, fixed, rows, D, dt) == \
            ref.evict_rows(budget, fixed, rows, D, name)
        nh = int(rng.integers(1, 9))
        mass = rng.integers(0, 4, nh).astype(np.float32)  # ties on purpose
        bud = float(rng.uniform(0, 2e6))
        assert uc.uc_assign_bits(mass, 4096, 128, 64, 2, bud, 1e5) == \
            list(ref.assign_bits(mass.astype(np.float64), 4096, 128, 64, "bf16", bud, 1e5))
        nt = int(rng.integers(1, 6))
        m = np.where(rng.random(nt) < 0.2, 0.0, rng.random(nt))
        bp = rng.uniform(0, 10, nt)
        B = float(rng.uniform(0, 30))
        assert np.allclose(uc.uc_type_budget(m, bp, B), ref.type_budget(m, bp, B), rtol=1e-12)
        args = (float(rng.uniform(0.2, 1)), 0.6, 0.2, float(rng.uniform(0, 2)), 1.0)
        a = uc.uc_retention_next(*args)
        assert a == ref.retention_next(*args) or (math.isnan(a) and math.isnan(ref.retention_next(*args)))
        Dq = int(rng.choice([32, 64, 128]))
        first = int(rng.integers(0, 3 * (int(math.log2(Dq // 32)) + 1)))
        qb = float(rng.uniform(0, 8 * Dq * rows // 2 + 1e5))
        assert uc.uc_quant_config(qb, rows, Dq, dt, nh, first) == \
            ref.quant_config(qb, rows, Dq, name, nh, first)
    assert uc.uc_packed_bytes(100, 128, 48, 4, 2) == -1


def test_budget_structs_and_validation():
    """uc_budget_params / uc_budget_state mirror the header's layouts, and
    uc_budget_step / uc_calibrate_policy reject bad arguments on the host
    (nothing is launched)."""
    import paper_2609_32831_amd as uc
    P, S = uc.uc_budget_params, uc.uc_budget_state
    assert ctypes.sizeof(P) == 56 and P.rho_init.offset == 40 and P.rho_min.offset == 48
    assert ctypes.sizeof(S) == 88 and S.m.offset == 24 and S.b.offset == 40
    assert S.k.offset == 56 and S.n_boundaries.offset == 80
    L, E = uc.lib, uc.UC_E_INVALID
    FAKE = 4096
    good = P(28, 4, 128, 16, 3, 1, 2, 4096, 4096, uc.UC_BF16, 0.3, 0.15)
    assert L.uc_budget_step(ctypes.byref(good), None, 1, FAKE, None) == E
    assert L.uc_budget_step(ctypes.byref(good), FAKE, 0, FAKE, None) == E
    assert L.uc_budget_step(ctypes.byref(good), FAKE, 1, FAKE + 4, None) == E  # misaligned state
    for field, bad in (("qt", 1), ("ev", 3), ("rho_min", 0.4), ("rho_min", 0.0), ("Hq", 30),
                       ("D", 96), ("n_segs", 9), ("dtype", 7)):
        p = P.from_buffer_copy(good)
        setattr(p, field, bad)
        assert L.uc_budget_step(ctypes.byref(p), FAKE, 1, FAKE, None) == E, field
    assert "rho_min" in uc.uc_last_error() or uc.uc_last_error()
    assert L.uc_calibrate_policy(FAKE, 0, 2, 0.5, FAKE, FAKE, None) == E
    assert L.uc_calibrate_policy(FAKE, 4, 9, 0.5, FAKE, FAKE, None) == E
    assert L.uc_calibrate_policy(None, 4, 2, 0.5, FAKE, FAKE, None) == E
    assert L.uc_calibrate_policy(FAKE, 4, 2, float("nan"), FAKE, FAKE, None) == E


def test_read_probe_validation(uc):
    """uc_read_probe rejects NULL pointers, unknown patterns and sizes that are
    not whole 4 KB pieces per workgroup before anything is launched."""
    L, E = uc.lib, uc.UC_E_INVALID
    unit = uc.uc_read_probe_unit()
    assert unit % 4096 == 0 and unit >= 4096
    assert uc.uc_read_probe_sink_bytes() == unit // 4096 * 4 * 16
    assert L.uc_read_probe(None, unit, 0, FAKE, None) == E
    assert L.uc_read_probe(FAKE, unit, 0, None, None) == E
    assert L.uc_read_probe(FAKE, unit, 2, FAKE, None) == E
    assert L.uc_read_probe(FAKE, unit, -1, FAKE, None) == E
    assert L.uc_read_probe(FAKE, 0, 0, FAKE, None) == E
    assert L.uc_read_probe(FAKE, unit + 4096, 1, FAKE, None) == E
    assert "multiple" in uc.uc_last_error()
