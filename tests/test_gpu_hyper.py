"""GPU parity of the hyperparameter fit (Sec. 3.2, GP hyperparameter optimisation): the
HIP library through its C-ABI against the fp64 oracle on the same seeded inputs.

Both sides compute in fp64; they differ in summation order (and the Cholesky's
blocking), which the conditioning of K amplifies (cond(K) <= n s / floor). Measured
differences on C1..C5 are below 3e-14 (objective) and 1e-13 (gradient); the bars keep
a margin of 1e4 for worse-conditioned settings:
  * objective: |dv| <= 1e-10 max(|v|, 1);
  * gradient:  |dg| <= 1e-8 max(|g|_inf, 1) per entry (the trace formula carries K^-1);
  * L-BFGS: every sample objective to the bar above, the same kept starts (up to ties
    within that bar), the device's final objective equal to the oracle's objective at
    the device's final setting, and each final objective within 1e-6 of the oracle's
    final objective from the same start (both stop within the gradient tolerance of
    the same maximum; a start whose paths separate is checked for validity instead).
"""
import math

import numpy as np
import pytest

from oracle import gp_hyper as gh
from workloads import hyper_starts, make_workload

pytestmark = pytest.mark.gpu

PRIOR = (1.5, 1.0)
FLOOR = 1e-6
TOL_V = 1e-10
TOL_G = 1e-8


@pytest.fixture(autouse=True)
def _announce(request):
    print(f"\n[gpu] {request.node.nodeid}", flush=True)
    yield


def _gp():
    from paper_2212_11142_amd import gp
    return gp


def _dev(a, dtype=None):
    import torch
    a = np.ascontiguousarray(a if dtype is None else a.astype(dtype))
    return torch.from_numpy(a).cuda()


def _inputs(name, n=None):
    gp = _gp()
    w = make_workload(name, 256)
    X = [c[:n] for c in w.X] if n else w.X
    y = w.y[:n] if n else w.y
    feas = w.feasible[:n] if n else w.feasible
    space = gp.Space(w.space)
    return w, space, X, y, feas, (gp.to_device_columns(space, X), _dev(np.nan_to_num(y, nan=0.0)),
                                  _dev(feas))


def _check_values(got, ref, label):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    inf_g, inf_r = ~np.isfinite(got), ~np.isfinite(ref)
    assert np.array_equal(inf_g, inf_r), f"{label}: -inf pattern {inf_g} vs {inf_r}"
    ok = ~inf_r
    e = np.abs(got[ok] - ref[ok]) / np.maximum(np.abs(ref[ok]), 1.0)
    assert e.size == 0 or e.max() <= TOL_V, f"{label}: objective rel err {e.max():.2e}"
    return 0.0 if e.size == 0 else float(e.max())


@pytest.mark.parametrize("name,n", [("C1", None), ("C2", None), ("C3", None), ("C4", None),
                                    ("C5", 300)])
def test_log_posterior_parity(name, n):
    gp = _gp()
    w, space, X, y, feas, (Xd, yd, fd) = _inputs(name, n)
    d = len(w.space)
    theta = np.concatenate([hyper_starts(d, 5, 31), hyper_starts(d, 2, 32)])
    theta[5:, d + 1] = -3.0   # two settings with a noise variance well above the floor
    T, yf = gh.hyper_data(w.space, X, y, feas)
    for prior in (None, PRIOR):
        out = gp.log_posterior(space, Xd, yd, fd, _dev(theta), prior, FLOOR)
        v = out["value"].cpu().numpy()
        g = out["grad"].cpu().numpy()
        ref = [gh.log_posterior(T, yf, t, prior, FLOOR) for t in theta]
        ev = _check_values(v, [r[0] for r in ref], f"{name} prior={prior}")
        eg = 0.0
        for b, (rv, rg) in enumerate(ref):
            if rg is None:
                continue
            scale = max(np.abs(rg).max(), 1.0)
            e = np.abs(g[b] - rg).max() / scale
            eg = max(eg, e)
            assert e <= TOL_G, f"{name} setting {b}: gradient rel err {e:.2e}"
        print(f"{name} prior={prior}: value err {ev:.1e} grad err {eg:.1e}")


def test_log_posterior_full_c5():
    """C5 at its full n = 2048 (d = 12 with two permutations): two settings."""
    gp = _gp()
    w, space, X, y, feas, (Xd, yd, fd) = _inputs("C5")
    d = len(w.space)
    theta = hyper_starts(d, 2, 41)
    out = gp.log_posterior(space, Xd, yd, fd, _dev(theta), PRIOR, FLOOR)
    T, yf = gh.hyper_data(w.space, X, y, feas)
    for b in range(2):
        rv, rg = gh.log_posterior(T, yf, theta[b], PRIOR, FLOOR)
        _check_values(out["value"][b:b + 1].cpu().numpy(), [rv], f"C5 setting {b}")
        g = out["grad"][b].cpu().numpy()
        assert np.abs(g - rg).max() <= TOL_G * max(np.abs(rg).max(), 1.0)


def test_log_posterior_edges():
    """Settings at the edges of the arithmetic: an infinite lengthscale (parameter
    dropped; -inf with the prior), a zero lengthscale (not a kernel), an overflowing
    output scale (the factorisation overflows: not a kernel), a huge noise."""
    gp = _gp()
    w, space, X, y, feas, (Xd, yd, fd) = _inputs("C1")
    d = len(w.space)
    base = hyper_starts(d, 1, 3)[0]
    rows = []
    for q, v in [(0, 800.0), (0, -800.0), (d, 800.0), (d + 1, 800.0), (d + 1, -800.0)]:
        t = base.copy()
        t[q] = v
        rows.append(t)
    theta = np.array(rows)
    T, yf = gh.hyper_data(w.space, X, y, feas)
    for prior in (None, PRIOR):
        out = gp.log_posterior(space, Xd, yd, fd, _dev(theta), prior, FLOOR, want_grad=False)
        ref = [gh.log_posterior(T, yf, t, prior, FLOOR, want_grad=False)[0] for t in theta]
        _check_values(out["value"].cpu().numpy(), ref, f"edges prior={prior}")


def test_log_posterior_many_settings_and_feasible_subset():
    """More settings than one batch (3 batches of 64) and an infeasible subset that
    must be ignored."""
    gp = _gp()
    w, space, X, y, feas, (Xd, yd, fd) = _inputs("C3", 120)
    d = len(w.space)
    theta = hyper_starts(d, 150, 51)
    out = gp.log_posterior(space, Xd, yd, fd, _dev(theta), PRIOR, FLOOR, want_grad=False)
    T, yf = gh.hyper_data(w.space, X, y, feas)
    ref = [gh.log_posterior(T, yf, t, PRIOR, FLOOR, want_grad=False)[0] for t in theta]
    _check_values(out["value"].cpu().numpy(), ref, "C3 150 settings")
    assert 0 < feas.sum() < len(feas)


def _check_fit(w, X, y, feas, out, ref, T, yf, label):
    v0 = out["value0"].cpu().numpy()
    _check_values(v0, ref["obj0"], f"{label} samples")
    keep = out["keep"].cpu().numpy()
    # the kept starts: same indices, or equal objectives where they differ
    for r, (a, b) in enumerate(zip(keep, ref["keep"])):
        if a != b:
            assert abs(ref["obj0"][a] - ref["obj0"][b]) <= TOL_V * max(abs(ref["obj0"][b]), 1.0), \
                f"{label}: start {r} is sample {a}, oracle {b}"
    theta = out["theta"].cpu().numpy()
    val = out["value"].cpu().numpy()
    its = out["iters"].cpu().numpy()
    status = out["status"].cpu().numpy()
    for k in range(len(keep)):
        rv, rg = gh.log_posterior(T, yf, theta[k], PRIOR, FLOOR)
        _check_values([val[k]], [rv], f"{label} start {k}: objective at the device's setting")
        if not math.isfinite(rv):
            continue
        o = int(np.nonzero(ref["keep"] == keep[k])[0][0]) if keep[k] in ref["keep"] else -1
        if o >= 0:
            dv = abs(val[k] - ref["obj"][o]) / max(abs(ref["obj"][o]), 1.0)
            gmax = np.abs(rg).max()
            # same maximum, or (paths separated) a point the oracle also finds stationary
            assert dv <= 1e-6 or (status[k] in (1, 2) and gmax <= 1e-2), \
                f"{label} start {k}: final {val[k]} vs oracle {ref['obj'][o]} (|g| {gmax:.1e})"
    print(f"{label}: iterations {its.tolist()} oracle {ref['iters'].tolist()} "
          f"status {status.tolist()} best {val.max():.6f} oracle {ref['obj'].max():.6f}")


@pytest.mark.parametrize("name,n,S0,K", [("C1", None, 64, 4), ("C2", None, 64, 4),
                                         ("C3", None, 48, 4), ("C4", None, 64, 3)])
def test_hyperfit_parity(name, n, S0, K):
    gp = _gp()
    w, space, X, y, feas, (Xd, yd, fd) = _inputs(name, n)
    d = len(w.space)
    theta0 = hyper_starts(d, S0, 61)
    out = gp.hyperfit(space, Xd, yd, fd, _dev(theta0), K, PRIOR, FLOOR, max_iter=100)
    ref = gh.hyperfit(w.space, X, y, feas, theta0, K, PRIOR, FLOOR, max_iter=100)
    T, yf = gh.hyper_data(w.space, X, y, feas)
    _check_fit(w, X, y, feas, out, ref, T, yf, name)


def test_hyperfit_edges():
    gp = _gp()
    w, space, X, y, feas, (Xd, yd, fd) = _inputs("C2", 60)
    d = len(w.space)
    theta0 = hyper_starts(d, 6, 71)
    theta0[0, 0] = -800.0                  # not a kernel: ranked last
    # no iterations: the kept samples come back unchanged
    out = gp.hyperfit(space, Xd, yd, fd, _dev(theta0), 6, PRIOR, FLOOR, max_iter=0)
    keep = out["keep"].cpu().numpy()
    assert keep[-1] == 0 and sorted(keep.tolist()) == list(range(6))
    np.testing.assert_array_equal(out["theta"].cpu().numpy(), theta0[keep])
    v0 = out["value0"].cpu().numpy()
    np.testing.assert_array_equal(out["value"].cpu().numpy(), v0[keep])
    assert out["status"].cpu().numpy()[-1] == 5
    # a single sample, a single start
    out1 = gp.hyperfit(space, Xd, yd, fd, _dev(theta0[1:2]), 1, PRIOR, FLOOR, max_iter=50)
    ref1 = gh.hyperfit(w.space, X, y, feas, theta0[1:2], 1, PRIOR, FLOOR, max_iter=50)
    T, yf = gh.hyper_data(w.space, X, y, feas)
    _check_fit(w, X, y, feas, out1, ref1, T, yf, "single")
    # rejected arguments
    for K in (0, 7, 65):
        with pytest.raises(gp.GPError):
            gp.hyperfit(space, Xd, yd, fd, _dev(theta0), K, PRIOR, FLOOR)
    with pytest.raises(gp.GPError):
        gp.hyperfit(space, Xd, yd, fd, _dev(theta0), 2, (0.0, 1.0), FLOOR)


def test_hyper_rejects_invalid_observation():
    gp = _gp()
    w, space, X, y, feas, _ = _inputs("C1", 20)
    X = [c.copy() for c in X]
    X[2][3] = 99                            # an int out of its declared range
    Xd = gp.to_device_columns(space, X)
    theta = _dev(hyper_starts(len(w.space), 2, 5))
    with pytest.raises(gp.GPError, match="observation 3"):
        gp.log_posterior(space, Xd, _dev(y), _dev(feas), theta, PRIOR, FLOOR)
