"""Pins of the oracle's realized compression and rho_min calibration (App. B,
"Compression Ratio" and "Calibration Setting"; Sec. 3.3 Eq. 3) on a tiny
editing-shaped workload with a protected self segment that draws attention
away from the cached conditioning as the timesteps advance.

The realized compression is re-derived from the byte sizes of the arrays the
chain actually stores; monotonicity in rho_min and the bisection's result are
checked against brute force over a grid of rho_min values; rho_min = rho_init
has the closed form rho = rho_init at every boundary."""
import numpy as np
import pytest


def _tiny(gen):
    S = gen.SegSpec
    return gen.Workload(
        name="tiny_dynamic_self", recipe_id=3, B=1, Hq=4, Hkv=2, D=64, q_dtype="bf16",
        segments=(S("text", 32, "keep", "bf16"), S("vit", 256, "evict", "bf16"),
                  S("vae", 256, "quant", "bf16", bits=None, group=None),
                  S("self", 64, "protect", "bf16", self_align=6.0)),
        W=16, mode="prefill", steps=16, M=16, n_outlier=2, outlier_scale=8.0,
        chunk_steps=3, rho_init=0.30, rho_min=0.15, obs_window=4, self_pull=10.0, self_ramp=6)


def _compression_by_hand(w, r):
    """1 - mean over t >= 1 of (stored nbytes / original nbytes), from the
    kept index arrays and the packed arrays of the state in force at t."""
    D = w.D
    orig = sum(2 * s.n * D * 2 for s in w.segments if s.policy != "protect")
    text = 2 * w.segments[0].n * D * 2
    bounds = sorted(r["decisions"])
    fr = []
    for t in range(1, w.steps):
        tb = max(b for b in bounds if b < t)
        keep = r["keep"][tb][0]                          # one KV head's kept rows
        vit = 2 * keep.shape[0] * np.zeros((1, D), np.uint16).nbytes + keep.astype(np.int32).nbytes
        pk = r["packed"][tb]
        Hkv = pk["bits"].shape[0]
        vae = sum(pk[n].nbytes for n in ("codes_k", "codes_v", "scale_k", "min_k", "scale_v",
                                          "min_v", "tail_k", "tail_v")) / Hkv
        fr.append((text + vit + vae) / orig)
    return 1.0 - float(np.mean(fr))


@pytest.fixture(scope="module")
def grid(gen):
    import oracle.pipeline as op
    w = _tiny(gen)
    out = []
    for x in np.linspace(0.0, w.rho_init, 31)[1:]:
        wx = gen.scaled(w, rho_min=float(x))
        r = op.budget_chain(wx, 0, [])
        out.append((float(x), op.realized_compression(wx, r["decisions"]), r))
    return w, out


def test_realized_compression_by_hand(gen, grid):
    import oracle.pipeline as op
    w, g = grid
    for x, c, r in g[::6]:
        assert abs(c - _compression_by_hand(gen.scaled(w, rho_min=x), r)) < 1e-12, x


def test_realized_compression_monotone_in_rho_min(grid):
    w, g = grid
    cs = [c for _, c, _ in g]
    assert all(a >= b - 1e-15 for a, b in zip(cs, cs[1:]))   # higher floor: less compression
    assert cs[0] > cs[-1] + 0.05                                # the floor binds


def test_rho_min_equal_rho_init_closed_form(gen, grid):
    w, g = grid
    x, c, r = g[-1]
    assert x == pytest.approx(w.rho_init)
    assert all(d["rho"] == w.rho_init for d in r["decisions"].values())


def test_self_pull_moves_mass_to_the_protected_segment(grid):
    _, g = grid
    m = g[0][2]["mass"]
    self_mass = [m[t][3] for t in sorted(m)]
    assert self_mass[0] < 0.2 and self_mass[-1] > 0.8
    assert all(b >= a - 0.02 for a, b in zip(self_mass, self_mass[1:6]))


@pytest.mark.parametrize("target", [0.72, 0.75, 0.79])
def test_calibration_matches_brute_force(gen, grid, target):
    import oracle.pipeline as op
    w, g = grid
    res = op.calibrate_rho_min(w, target, iters=10)
    best_grid = min(abs(c - target) for _, c, _ in g)
    assert abs(res["compression"] - target) <= best_grid + 1e-12, (res, best_grid)
    assert abs(res["compression"] - target) <= 0.005
    # the reported compression is that of the returned rho_min
    wx = gen.scaled(w, rho_min=res["rho_min"])
    assert op.realized_compression(wx, op.budget_chain(wx, 0, [])["decisions"]) == res["compression"]
