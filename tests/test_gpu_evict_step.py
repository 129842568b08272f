"""uc_evict_step (row count read on the device) against the oracle's
selection and the plain composition of logical indices (Sec. 3.4, App. E
"Batched GQA token selection"): kept indices and rows bit-exact."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # collected on CPU-only hosts, never run there
    pytest.skip("needs a GPU", allow_module_level=True)

import oracle as ref  # noqa: E402
import paper_2609_32831_amd as uc  # noqa: E402
from gpu_util import dev, host_bytes, rand_rows  # noqa: E402

D = 128


def _scores(seed, BH, N):
    rng = np.random.default_rng(seed)
    s = rng.random((BH, N)).astype(np.float32)
    # ties across the cut and signed zeros
    s[:, ::7] = s[:, 3:4]
    s[:, 1::11] = 0.0
    s[:, 2::13] = -0.0
    return s


@pytest.mark.parametrize("B,Hkv,N,cap,ks,with_idx", [
    (1, 4, 1227, 1300, [469, 469, 469, 469], True),
    (2, 4, 4096, 4096, [1227] * 8, False),          # first eviction: idx = local positions
    (1, 4, 469, 512, [178, 0, 468, 1], True),       # k differs per call below
])
def test_evict_step_matches_select(B, Hkv, N, cap, ks, with_idx):
    print(f"CASE evict_step B={B} Hkv={Hkv} N={N} cap={cap} k={ks[0]} idx={with_idx}", flush=True)
    BH = B * Hkv
    shape = uc.make_shape(B, 28, Hkv, D)
    kr = rand_rows(71, BH, cap, D, "bf16")
    vr = rand_rows(72, BH, cap, D, "bf16")
    rng = np.random.default_rng(N)
    lidx = np.sort(np.stack([rng.choice(4 * cap, cap, replace=False) for _ in range(BH)]), 1)
    lidx = lidx.astype(np.int32)
    cur = uc.dense_segment(dev(kr, "bf16").reshape(B, Hkv, cap, D),
                           dev(vr, "bf16").reshape(B, Hkv, cap, D), n_rows=N,
                           idx=torch.from_numpy(lidx).cuda() if with_idx else None)
    sc = _scores(N + cap, BH, N)
    sc_d = torch.from_numpy(sc).cuda()
    for k in sorted(set(ks)) + [N, N + 5]:
        ok_ = torch.full((B, Hkv, cap, D), 3.0, dtype=torch.bfloat16, device="cuda")
        ov_ = torch.full_like(ok_, -3.0)
        oi = torch.full((B, Hkv, cap), -9, dtype=torch.int32, device="cuda")
        out = uc.dense_segment(ok_, ov_, idx=oi)
        k_dev = torch.tensor([k], dtype=torch.int32, device="cuda")
        uc.uc_evict_step(shape, sc_d, cur, k_dev, out)
        torch.cuda.synchronize()
        if k >= N:  # nothing written
            assert torch.all(oi == -9) and torch.all(ok_ == 3.0) and torch.all(ov_ == -3.0), k
            continue
        keep = ref.select(sc, k)  # [BH, k] ascending local positions
        want_idx = np.take_along_axis(lidx, keep, 1) if with_idx else keep
        got_idx = oi.cpu().numpy().reshape(BH, cap)
        assert np.array_equal(got_idx[:, :k], want_idx), k
        assert np.all(got_idx[:, k:] == -9), k
        gk = host_bytes(ok_).reshape(BH, cap, D)
        gv = host_bytes(ov_).reshape(BH, cap, D)
        for bh in range(BH):
            assert np.array_equal(gk[bh, :k], kr[bh][keep[bh]]), (k, bh)
            assert np.array_equal(gv[bh, :k], vr[bh][keep[bh]]), (k, bh)
