"""Pins of the hyperparameter-fit oracle (Sec. 3.2, GP hyperparameter optimisation)
against facts fixed outside it: scikit-learn's GP marginal likelihood and gradient on
an explicit Euclidean embedding of every parameter type, central differences, scipy's
gamma density, closed-form optima, scipy's L-BFGS-B, recovery of the lengthscales a
sample was drawn with, and a brute-force ranking of the kept fraction.
"""
import math

import numpy as np
import pytest
from scipy import optimize, stats

from oracle import gp_hyper as gh
from oracle import gp_oracle as go
from test_oracle_pins import embed
from workloads import Param, hyper_starts, make_workload

PRIOR = (1.5, 1.0)


def _subset(name, n):
    w = make_workload(name, 256)
    X = [c[:n] for c in w.X]
    return w, X, w.y[:n], w.feasible[:n]


def _coords(p):
    """Embedding coordinates of one parameter (see embed)."""
    if p.kind in go.NUMERIC:
        return 1
    if p.kind == "cat":
        return p.levels
    return {"kendall": p.m * (p.m - 1) // 2, "spearman": p.m, "hamming": p.m * p.m}[p.dist]


@pytest.mark.parametrize("name,n", [("C1", 32), ("C2", 60), ("C5", 50)])
def test_log_posterior_matches_sklearn_on_embedding(name, n):
    """Without prior and floor, the objective is scikit-learn's log marginal likelihood
    of ConstantKernel(s) * Matern(l, 5/2) + WhiteKernel(noise) on the embedding (every
    coordinate of parameter p carries l_p), and its gradient is the sum of
    scikit-learn's log-lengthscale gradients over those coordinates."""
    from sklearn.gaussian_process import GaussianProcessRegressor
    from sklearn.gaussian_process.kernels import ConstantKernel, Matern, WhiteKernel
    w, X, y, feas = _subset(name, n)
    T, yf = gh.hyper_data(w.space, X, y, feas)
    fidx = np.nonzero(feas)[0]
    enc = [e[fidx] for e in go.encode(w.space, X)]
    E = embed(w.space, enc, np.ones(len(w.space)))
    d = len(w.space)
    rng = np.random.default_rng(3)
    for _ in range(3):
        theta = np.concatenate([rng.uniform(-1.0, 1.5, d), rng.uniform(-0.5, 0.5, 1),
                                rng.uniform(-9.0, -3.0, 1)])
        v, g = gh.log_posterior(T, yf, theta)
        counts = [_coords(p) for p in w.space]
        ls = np.repeat(np.exp(theta[:d]), counts)
        k = ConstantKernel(math.exp(theta[d])) * Matern(length_scale=ls, nu=2.5) \
            + WhiteKernel(math.exp(theta[d + 1]))
        gpr = GaussianProcessRegressor(kernel=k, alpha=0.0, optimizer=None, normalize_y=False)
        gpr.fit(E, yf)
        vs, gs = gpr.log_marginal_likelihood(gpr.kernel_.theta, eval_gradient=True)
        assert abs(v - vs) <= 1e-9 * max(abs(vs), 1.0)
        starts = np.concatenate([[0], np.cumsum(counts)])
        g_sk = np.array([gs[1 + starts[p]:1 + starts[p + 1]].sum() for p in range(d)]
                        + [gs[0], gs[-1]])
        np.testing.assert_allclose(g, g_sk, rtol=1e-7, atol=1e-8 * np.abs(g_sk).max())


@pytest.mark.parametrize("name,n", [("C2", 50), ("C3", 60), ("C5", 40)])
def test_gradient_central_differences(name, n):
    """With the gamma prior and the noise floor, the gradient matches central
    differences of the value in every coordinate."""
    w, X, y, feas = _subset(name, n)
    T, yf = gh.hyper_data(w.space, X, y, feas)
    d = len(w.space)
    theta = hyper_starts(d, 1, 11)[0]
    theta[d + 1] = -4.0
    v, g = gh.log_posterior(T, yf, theta, PRIOR, 1e-6)
    h = 1e-5
    for q in range(d + 2):
        e = np.zeros(d + 2)
        e[q] = h
        vp = gh.log_posterior(T, yf, theta + e, PRIOR, 1e-6, want_grad=False)[0]
        vm = gh.log_posterior(T, yf, theta - e, PRIOR, 1e-6, want_grad=False)[0]
        fd = (vp - vm) / (2 * h)
        assert abs(fd - g[q]) <= 1e-6 * max(abs(g[q]), 1.0), (q, fd, g[q])


def test_gamma_prior_matches_scipy():
    l = np.array([0.01, 0.3, 1.0, 2.5, 40.0])
    for shape, rate in [(1.5, 1.0), (2.0, 0.5), (0.8, 3.0)]:
        np.testing.assert_allclose(gh.gamma_logpdf(l, shape, rate),
                                   stats.gamma.logpdf(l, shape, scale=1.0 / rate), rtol=1e-12)


def test_pair_terms_sum_to_sqdist():
    """sum_p T[p] / l_p^2 is the kernel's squared distance for any lengthscales."""
    w, X, y, feas = _subset("C5", 40)
    enc = go.encode(w.space, X)
    T = gh.pair_terms(w.space, enc)
    ls = np.exp(np.random.default_rng(5).uniform(-1, 1, len(w.space)))
    r2 = sum(T[p] / ls[p] ** 2 for p in range(len(w.space)))
    np.testing.assert_allclose(r2, go.sqdist(w.space, enc, enc, ls), rtol=1e-13, atol=1e-15)
    assert np.all(np.diagonal(T, axis1=1, axis2=2) == 0.0) and T.min() >= 0.0 and T.max() <= 1.0


def test_lbfgs_quadratic_optimum():
    rng = np.random.default_rng(0)
    Q = np.linalg.qr(rng.normal(size=(8, 8)))[0]
    A = Q @ np.diag(np.geomspace(1.0, 100.0, 8)) @ Q.T
    c = rng.normal(size=8)
    fun = lambda x: (-0.5 * (x - c) @ A @ (x - c), -A @ (x - c))
    x, v, it, _ = gh.lbfgs_maximize(fun, np.zeros(8), max_iter=500, gtol=1e-10, ftol=0.0)
    np.testing.assert_allclose(x, c, atol=1e-9)
    assert it < 100


def test_lbfgs_rosenbrock():
    fun = lambda x: (-optimize.rosen(x), -optimize.rosen_der(x))
    x, v, it, _ = gh.lbfgs_maximize(fun, np.array([-1.2, 1.0]), max_iter=1000, gtol=1e-9,
                                    ftol=0.0)
    np.testing.assert_allclose(x, [1.0, 1.0], atol=1e-6)


def test_lbfgs_matches_scipy_on_objective():
    """From the same start, the oracle's L-BFGS and scipy's L-BFGS-B reach the same
    maximum of the objective (C1, 32 observations)."""
    w = make_workload("C1", 256)
    T, yf = gh.hyper_data(w.space, w.X, w.y, w.feasible)
    d = len(w.space)
    fun = lambda t: gh.log_posterior(T, yf, t, PRIOR, 1e-6)
    for seed in (1, 2):
        t0 = hyper_starts(d, 1, seed)[0]
        x, v, it, _ = gh.lbfgs_maximize(fun, t0, max_iter=500, gtol=1e-7, ftol=0.0)

        def neg(t):
            val, g = fun(t)
            return (1e300, np.zeros_like(t)) if g is None else (-val, -g)

        res = optimize.minimize(neg, t0, jac=True, method="L-BFGS-B",
                                options={"maxiter": 2000, "gtol": 1e-9, "ftol": 1e-15})
        assert abs(v - (-res.fun)) <= 1e-7 * max(abs(v), 1.0), (v, -res.fun)
        np.testing.assert_allclose(x[:d + 1], res.x[:d + 1], atol=1e-3)
        # the noise coordinate is flat where the floor dominates: compare the variance
        nv = lambda t: 1e-6 + math.exp(t)
        assert abs(nv(x[d + 1]) - nv(res.x[d + 1])) <= 1e-3 * nv(res.x[d + 1])


def test_recovers_generating_lengthscales():
    """Data drawn from the GP itself (two numeric inputs, l = 0.15 and 0.6): the fitted
    lengthscales land near the generating ones, in the right order."""
    rng = np.random.default_rng(21)
    space = [Param("a", "real", lo=0.0, hi=1.0), Param("b", "real", lo=0.0, hi=1.0)]
    n = 250
    X = [rng.random(n), rng.random(n)]
    T = gh.pair_terms(space, go.encode(space, X))
    l_true, s_true, nv = np.array([0.15, 0.6]), 1.0, 1e-4
    K = go.matern52(T[0] / l_true[0] ** 2 + T[1] / l_true[1] ** 2, s_true) + nv * np.eye(n)
    y = np.linalg.cholesky(K) @ rng.normal(size=n)
    th0 = hyper_starts(2, 16, 4)
    r = gh.hyperfit(space, X, y, np.ones(n, np.uint8), th0, 4, None, 1e-6, max_iter=200)
    l_fit = np.exp(r["theta"][r["best"]][:2])
    assert np.all(np.abs(np.log(l_fit / l_true)) < math.log(1.5)), l_fit
    assert l_fit[0] < l_fit[1]


def test_hyperfit_keeps_the_best_fraction():
    w = make_workload("C2", 256)
    d = len(w.space)
    th0 = hyper_starts(d, 24, 9)
    th0[5, 0] = 800.0                                 # overflowing setting: -inf
    r = gh.hyperfit(w.space, [c[:60] for c in w.X], w.y[:60], w.feasible[:60], th0, 5, PRIOR,
                    max_iter=30)
    assert r["obj0"][5] == -math.inf
    brute = sorted(range(len(th0)), key=lambda i: (-r["obj0"][i], i))[:5]
    assert list(r["keep"]) == brute
    assert np.all(r["obj"] >= r["obj0"][r["keep"]])
    assert r["best"] == int(np.argmax(r["obj"]))
