"""The allocation-free attention entry point (uc_attend_mixed_noalloc) against
uc_attend_mixed with a caller workspace: same results on two calls in a row,
the second with a smaller input (the static scratch array keeps the first
call's contents), on the matrix-core decode kernel with per-segment
statistics, the VALU path, and a small prefill block; calls whose workspace
exceeds the static array are refused before any launch."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import oracle as ref  # noqa: E402
import paper_2609_32831_amd as uc  # noqa: E402
from gpu_util import check_attention, dev, rand_rows, sm_scale  # noqa: E402
from gpu_util import mixed_case as _mixed_case  # noqa: E402


def _run(segs, B, Hq, Hkv, M, q, noalloc, stats=True):
    D = 128
    shape = uc.make_shape(B, Hq, Hkv, D)
    o = torch.empty(B, Hq, M, D, device="cuda")
    lse = torch.empty(B, Hq, M, device="cuda") if stats else None
    sl = torch.empty(B, Hq, M, len(segs), device="cuda") if stats else None
    if noalloc:
        uc.uc_attend_mixed_noalloc(shape, segs, q, M, sm_scale(D), o, lse, sl)
    else:
        uc.uc_attend_mixed(shape, segs, q, M, sm_scale(D), o, lse, sl)
    kernel = uc.uc_last_kernel()
    torch.cuda.synchronize()
    return kernel, [x.cpu().numpy() for x in (o, lse, sl) if x is not None]


# B, Hq, Hkv, M, sizes; each pair runs the larger case first, then the smaller
CASES = [
    ((2, 28, 4, 1, (512, 4096, 1500, 4096 + 17, 5, 8)),
     (1, 28, 4, 1, (100, 900, 300, 256, 3, 4)), "decode_mfma"),
    ((1, 28, 4, 40, (100, 900, 300, 1000 + 17, 5, 8)),
     (1, 28, 4, 9, (64, 300, 100, 256, 3, 8)), "prefill_mfma"),
]


@pytest.mark.parametrize("big,small,kernel", CASES, ids=["decode", "prefill"])
def test_noalloc_matches_workspace_call(big, small, kernel):
    for B, Hq, Hkv, M, sizes in (big, small):
        print(f"CASE noalloc B={B} Hq={Hq} Hkv={Hkv} M={M} sizes={sizes}", flush=True)
        D = 128
        segs, K, V, seg_id = _mixed_case(B, Hq, Hkv, D, "bf16", sizes, seed=M + B)
        q = rand_rows(5 + M, B * Hq, M, D, "bf16").reshape(B, Hq, M, D)
        qd = dev(q, "bf16")
        shape = uc.make_shape(B, Hq, Hkv, D)
        need = uc.lib.uc_attend_workspace_size(shape, uc._seg_array(segs), len(segs), uc.UC_BF16, M)
        assert 0 < need <= uc.UC_SCRATCH_BYTES
        k1, got = _run(segs, B, Hq, Hkv, M, qd, True)
        k0, want = _run(segs, B, Hq, Hkv, M, qd, False)
        assert k1 == k0 == kernel, (k1, k0)
        for a, b in zip(got, want):  # same kernels, same order of sums
            assert np.array_equal(a, b, equal_nan=True)
        o_ref = ref.attend(ref.widen(q, "bf16"), K, V, None, seg_id, 4, sm_scale(D))[0]
        check_attention(got[0], o_ref, "noalloc")
        # without per-segment statistics (the decode kernel's single-state form)
        _, got_o = _run(segs, B, Hq, Hkv, M, qd, True, stats=False)
        _, want_o = _run(segs, B, Hq, Hkv, M, qd, False, stats=False)
        assert np.array_equal(got_o[0], want_o[0])


def test_noalloc_valu_path_and_limit():
    B, Hq, Hkv, M, D = 1, 28, 4, 3, 128
    segs, K, V, seg_id = _mixed_case(B, Hq, Hkv, D, "bf16", (33, 200, 77, 130, 1, 2), seed=4)
    qd = dev(rand_rows(6, B * Hq, M, D, "bf16").reshape(B, Hq, M, D), "bf16")
    prev = uc.uc_set_path(uc.UC_PATH_VALU)
    try:
        k1, got = _run(segs, B, Hq, Hkv, M, qd, True)
        k0, want = _run(segs, B, Hq, Hkv, M, qd, False)
    finally:
        uc.uc_set_path(prev)
    assert k1 == k0 == "attend_valu"
    for a, b in zip(got, want):
        assert np.array_equal(a, b, equal_nan=True)
    # a 4096-row prefill block over a packed segment needs more than the array
    B, M = 2, 4096
    segs, _, _, _ = _mixed_case(B, Hq, Hkv, D, "bf16", (64, 300, 100, 4096, 3, 8), seed=9)
    shape = uc.make_shape(B, Hq, Hkv, D)
    need = uc.lib.uc_attend_workspace_size(shape, uc._seg_array(segs), len(segs), uc.UC_BF16, M)
    assert need > uc.UC_SCRATCH_BYTES
    q = torch.zeros(B, Hq, M, D, dtype=torch.bfloat16, device="cuda")
    o = torch.full((B, Hq, M, D), 7.0, device="cuda")
    with pytest.raises(uc.UcError) as e:
        uc.uc_attend_mixed_noalloc(shape, segs, q, M, sm_scale(D), o)
    assert e.value.status == uc.UC_E_UNSUPPORTED and "static array" in str(e.value)
    torch.cuda.synchronize()
    assert bool((o == 7.0).all())  # refused before any launch: nothing written
