"""GPU parity of the calibration statistic (Sec. 3.2; App. B, "Calibration
Setting"): the fraction of a type's attention mass on its top 10 % of tokens,
and the eviction / quantisation assignment it drives."""
import math

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import oracle as ref  # noqa: E402
import oracle.pipeline as op  # noqa: E402
import paper_2609_32831_amd as uc  # noqa: E402
import workloads as gen  # noqa: E402
from paper_2609_32831_amd.runner import calibrate_policies  # noqa: E402
from workloads.device import device_inputs  # noqa: E402


@pytest.mark.parametrize("N,k", [(1000, 0), (1000, 1), (4097, 410), (777, 777), (61440, 6144)])
def test_topk_mass_parity(N, k):
    print("CASE topk_mass", N, k, flush=True)
    rng = np.random.default_rng(N + k)
    BH = 37
    x = rng.random((BH, N)).astype(np.float32) ** 4
    x[:5] = np.floor(x[:5] * 8)  # ties
    out = torch.empty(BH, device="cuda")
    uc.uc_topk_mass(torch.from_numpy(x).cuda(), k, out)
    torch.cuda.synchronize()
    assert np.allclose(out.cpu().numpy(), ref.topk_mass(x, k), rtol=2e-6, atol=1e-7)


def test_calibration_long_context_64k():
    """Ten calibration examples of the 64k context: the heavy-tailed ViT keys
    concentrate their mass (eviction), the Gaussian text keys do not
    (quantisation) -- the policies the workload is configured with; per
    (example, head) fractions agree with the oracle on sampled heads."""
    w = gen.LONG_CONTEXT_64K
    inp = device_inputs(w, "cuda", steps=1)
    res, f = calibrate_policies(w, inp, examples=10)
    print("CASE calibration", {k: (round(c, 4), p) for k, (c, p) in res.items()}, flush=True)
    assert res["vit"][1] == "evict" and res["text"][1] == "quant"
    for s in w.segments:
        assert res[s.name][1] == ("evict" if s.policy == "evict" else "quant")
    n_t = w.segments[0].n
    for (b, h) in [(0, 1), (9, 3)]:
        hi = op.head_inputs(w, b, h)
        K = np.concatenate([ref.widen(hi["seg_k"][i], s.dtype) for i, s in enumerate(w.segments)])
        seg_id = np.concatenate([np.full(s.n, i, np.int32) for i, s in enumerate(w.segments)])
        sc, _ = ref.score64(ref.widen(hi["q_obs"], w.q_dtype)[None], K[None, None], seg_id, 2,
                            op.sm_scale(w.D))
        sc = sc[0, 0].astype(np.float32)
        for i, s in enumerate(w.segments):
            part = sc[seg_id == i][None]
            want = ref.topk_mass(part, int(math.ceil(0.1 * s.n)))[0]
            got = f[b * w.Hkv + h, i]
            assert abs(got - want) <= 1e-5 * want + 1e-6, (b, h, s.name, got, want)


def test_rho_min_calibration_against_oracle():
    """rho_min calibration (App. B) on the editing workload with 128-row query
    blocks: at two of the GPU bisection's probes the oracle's own chain gives
    the same realized compression."""
    from paper_2609_32831_amd.calibrate import calibrate_rho_min
    w = gen.scaled(gen.IMAGE_EDITING_DYNAMIC, M=128, W=128)
    inp = device_inputs(w, "cuda")
    res = calibrate_rho_min(w, inp, w.target_compression, requests=[0], iters=8)
    print("CASE rho_min calibration M=128", res["rho_min"], res["compression"], flush=True)
    for x, c in (res["probes"][0], res["probes"][-1]):
        wx = gen.scaled(w, rho_min=x)
        want = op.realized_compression(wx, op.budget_chain(wx, 0, [])["decisions"])
        assert abs(c - want) <= 1e-12, (x, c, want)


def test_rho_min_calibration_full_size():
    """Full size, both requests: the calibrated rho_min gives an average
    realized compression within 0.5 percentage points of the 80 % target."""
    from paper_2609_32831_amd.calibrate import calibrate_rho_min
    w = gen.IMAGE_EDITING_DYNAMIC
    inp = device_inputs(w, "cuda")
    res = calibrate_rho_min(w, inp, w.target_compression, requests=list(range(w.B)), iters=12)
    print("CASE rho_min calibration full", res, flush=True)
    assert abs(res["compression"] - w.target_compression) <= 0.005, res
