"""GPU parity of the device-side budget decision (uc_budget_step: Sec. 3.3
Eq. 1-3 and the Sec. 3.4 translation) and of the calibration rule
(uc_calibrate_policy: Sec. 3.2, App. B) against the oracle's rules applied on
the host to the same inputs, over chains of random chunk masses."""
import ctypes

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import oracle as ref  # noqa: E402
import paper_2609_32831_amd as uc  # noqa: E402


def _oracle_chain(masses, Hq, Hkv, D, M, ev, qt, n_ev, n_qt, rho_init, rho_min):
    """The decisions of a chain of boundaries from the oracle's functions:
    masses[c] is [n_steps, Hkv, n_segs] of boundary c (one step at c = 0)."""
    S = [Hkv * ref.dense_bytes(n, D, "bf16") for n in (n_ev, n_qt)]
    out = []
    rho, b_prev, k_prev, cfg_prev, M0 = rho_init, list(S), n_ev, 0, None
    for c, mc in enumerate(masses):
        m = [float(np.mean([mc[t, :, a].astype(np.float64).sum() / (Hq * M)
                            for t in range(mc.shape[0])])) for a in (ev, qt)]
        if c == 0:
            M0 = m[0] + m[1]
        else:
            rho = ref.retention_next(rho, rho_init, rho_min, m[0] + m[1], M0)
        B = rho * sum(S)
        b = [float(x) for x in ref.type_budget(m, b_prev, B)]
        k = min(k_prev, ref.evict_rows(b[0] / Hkv, 0.0, n_ev, D, "bf16"))
        cfg, bits, group = ref.quant_config(b[1], n_qt, D, "bf16", Hkv, cfg_prev)
        out.append(dict(rho=rho, B=B, m=m, b=b, k=k, cfg=cfg, bits=bits, group=group,
                        k_prev=k_prev, cfg_prev=cfg_prev if c else -1))
        b_prev, k_prev, cfg_prev = b, k, cfg
    return out


@pytest.mark.parametrize("seed", range(6))
def test_budget_step_chain(seed):
    rng = np.random.default_rng(seed)
    Hq, Hkv, D, M = 28, 4, 128, int(rng.choice([16, 4096]))
    n_segs, ev, qt = 3, 1, 2
    n_ev, n_qt = 4096, 4096
    rho_init, rho_min = 0.30, 0.15
    C = 5
    print(f"CASE budget_step seed={seed} M={M}", flush=True)
    masses = []
    for c in range(5):
        n = 1 if c == 0 else C
        # per-step type masses summing to G*M per KV head, drifting apart
        p = rng.dirichlet([1.0 + 4 * seed, 2.0, 2.0 + c], size=(n, Hkv))
        masses.append((p * (Hq // Hkv) * M).astype(np.float32))
    want = _oracle_chain(masses, Hq, Hkv, D, M, ev, qt, n_ev, n_qt, rho_init, rho_min)
    params = uc.uc_budget_params(Hq, Hkv, D, M, n_segs, ev, qt, n_ev, n_qt, uc.UC_BF16,
                                 rho_init, rho_min)
    state = uc.budget_state_tensor()
    for c, mc in enumerate(masses):
        md = torch.from_numpy(mc).cuda()
        uc.uc_budget_step(params, md, mc.shape[0], state)
        st = uc.budget_state_read(state)
        w = want[c]
        assert st.n_boundaries == c + 1
        assert abs(st.rho - w["rho"]) <= 1e-12 * w["rho"], (c, st.rho, w["rho"])
        assert abs(st.B - w["B"]) <= 1e-12 * w["B"], c
        for i in range(2):
            assert abs(st.m[i] - w["m"][i]) <= 1e-12 * max(w["m"][i], 1e-300), (c, i)
            assert abs(st.b[i] - w["b"][i]) <= 1e-9 * max(w["b"][i], 1.0), (c, i)
        assert (st.k, st.cfg, st.bits, st.group) == (w["k"], w["cfg"], w["bits"], w["group"]), c
        assert (st.k_prev, st.cfg_prev) == (w["k_prev"], w["cfg_prev"]), c


def test_budget_step_rejects_bad_arguments():
    params = uc.uc_budget_params(28, 4, 128, 16, 3, 1, 1, 4096, 4096, uc.UC_BF16, 0.3, 0.15)
    state = uc.budget_state_tensor()
    mass = torch.zeros(1, 4, 3, device="cuda")
    with pytest.raises(uc.UcError):  # ev == qt
        uc.uc_budget_step(params, mass, 1, state)
    params.qt, params.rho_min = 2, 0.5  # rho_min > rho_init
    with pytest.raises(uc.UcError):
        uc.uc_budget_step(params, mass, 1, state)
    torch.cuda.synchronize()
    assert uc.budget_state_read(state).n_boundaries == 0  # nothing was enqueued


def test_calibrate_policy_mean_and_rule():
    rng = np.random.default_rng(5)
    frac = rng.uniform(0.0, 1.0, (40, 3)).astype(np.float32)
    frac[:, 0] *= 0.4                        # a quantisation type
    frac[:, 1] = 0.6 + 0.4 * frac[:, 1]      # an eviction type
    frac[:, 2] = 0.5                         # exactly at the threshold: eviction
    conc = torch.empty(3, dtype=torch.float64, device="cuda")
    ev = torch.empty(3, dtype=torch.int32, device="cuda")
    uc.uc_calibrate_policy(torch.from_numpy(frac).cuda(), 0.5, conc, ev)
    want = frac.astype(np.float64).mean(axis=0)
    assert np.allclose(conc.cpu().numpy(), want, rtol=1e-15, atol=0)
    assert ev.cpu().numpy().tolist() == [0, 1, 1]
