"""Importance scores from the row normalisers of an attention pass already
run (uc_score_columns; Sec. 3.3 Eq. 1 bracket, App. E "Efficient
attention-guided allocation") against the oracle's scores of the same
observation rows over the same cache, on both kernel paths."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # collected on CPU-only hosts, never run there
    pytest.skip("needs a GPU", allow_module_level=True)

import oracle as ref  # noqa: E402
import paper_2609_32831_amd as uc  # noqa: E402
from gpu_util import dev, mixed_case, rand_rows, sm_scale  # noqa: E402

CASES = [
    # B, Hq, Hkv, M, W, sizes (text, vit full, vit kept, packed, tail, tail cap), G, bits,
    # per-head widths
    (1, 28, 4, 300, 32, (1024, 4096, 1227, 4096 + 17, 1000, 1024), 128, 4, False),
    (2, 28, 4, 64, 64, (100, 900, 333, 1000, 3, 8), 32, 2, True),    # W = M: every row
    (1, 14, 2, 40, 7, (0, 200, 77, 130, 0, 4), 64, 4, False),        # no text, no tail rows
]


def _bar(got, want, tot):
    # as the two-pass scorer: each probability to ~2e-5 of itself or 1e-7 of
    # the row total (the normaliser comes from another kernel's fp32 sums)
    return np.abs(got - want) <= 2e-5 * want + 1e-7 * tot


@pytest.mark.parametrize("case", CASES)
def test_score_columns_from_attention_lse(case):
    B, Hq, Hkv, M, W, sizes, G, bits, per_head = case
    D = 128
    print("CASE score_columns", case, flush=True)
    segs, K, V, seg_id = mixed_case(B, Hq, Hkv, D, "bf16", sizes, seed=M + W, G=G, bits=bits,
                                    per_head=per_head)
    q = rand_rows(90 + W, B * Hq, M, D, "bf16").reshape(B, Hq, M, D)
    qd = dev(q, "bf16")
    q_obs = qd[:, :, M - W:].contiguous()
    sc_ref, ms_ref = ref.score64(ref.widen(q, "bf16")[:, :, M - W:], K, seg_id, 4, sm_scale(D))
    shape = uc.make_shape(B, Hq, Hkv, D)
    tot = Hq // Hkv * W
    o = torch.empty(B, Hq, M, D, device="cuda")
    lse = torch.empty(B, Hq, M, device="cuda")
    uc.uc_attend_mixed(shape, segs, qd, M, sm_scale(D), o, lse)
    n = [s.n_rows for s in segs]
    bounds = np.cumsum([0] + n)
    for path, kernel in ((uc.UC_PATH_AUTO, "score_mfma"), (uc.UC_PATH_VALU, "score_valu")):
        prev = uc.uc_set_path(path)
        try:
            # only the compacted segment's scores: the others stay untouched
            outs = [torch.full((B, Hkv, max(k, 1)), -7.0, device="cuda") for k in n]
            want = [None, outs[1], None, None]
            uc.uc_score_columns(shape, segs, q_obs, W, sm_scale(D), lse.view(-1)[M - W:], M, want)
            assert uc.uc_last_kernel() == kernel
            torch.cuda.synchronize()
            got1 = outs[1].cpu().numpy().astype(np.float64)
            assert np.all(_bar(got1, sc_ref[:, :, bounds[1]:bounds[2]], tot)), path
            for i in (0, 2, 3):
                assert torch.all(outs[i] == -7.0), (path, i)
            # every segment and the masses
            outs = [torch.empty(B, Hkv, k, device="cuda") for k in n]
            mass = torch.empty(B, Hkv, 4, device="cuda")
            uc.uc_score_columns(shape, segs, q_obs, W, sm_scale(D), lse.view(-1)[M - W:], M, outs,
                                mass)
            torch.cuda.synchronize()
        finally:
            uc.uc_set_path(prev)
        got = np.concatenate([t.cpu().numpy() for t in outs], axis=2).astype(np.float64)
        assert np.all(_bar(got, sc_ref, tot)), path
        assert np.allclose(mass.cpu().numpy(), ms_ref, rtol=2e-5, atol=1e-6 * tot), path
        assert np.allclose(got.sum(axis=2), tot, rtol=1e-5), path


def test_score_columns_given_exact_lse():
    """With the oracle's own normalisers (fp64 rounded to fp32) as row_lse the
    scores equal the oracle's: the call is the second pass alone."""
    B, Hq, Hkv, D, W = 2, 28, 4, 128, 32
    segs, K, V, seg_id = mixed_case(B, Hq, Hkv, D, "bf16", (64, 400, 100, 256, 3, 8), seed=5)
    q = rand_rows(17, B * Hq, W, D, "bf16").reshape(B, Hq, W, D)
    qw = ref.widen(q, "bf16")
    _, lse64, _, _ = ref.attend(qw, K, V, None, seg_id, 4, sm_scale(D))
    sc_ref, _ = ref.score64(qw, K, seg_id, 4, sm_scale(D))
    shape = uc.make_shape(B, Hq, Hkv, D)
    lse = torch.from_numpy(lse64.astype(np.float32)).cuda()
    outs = [torch.empty(B, Hkv, s.n_rows, device="cuda") for s in segs]
    uc.uc_score_columns(shape, segs, dev(q, "bf16"), W, sm_scale(D), lse, W, outs)
    assert uc.uc_last_kernel() == "score_mfma"
    torch.cuda.synchronize()
    got = np.concatenate([t.cpu().numpy() for t in outs], axis=2).astype(np.float64)
    assert np.all(_bar(got, sc_ref, Hq // Hkv * W))
