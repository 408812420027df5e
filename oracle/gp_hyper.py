"""CPU oracle of the GP hyperparameter fit (Sec. 3.2, GP hyperparameter optimisation).

TEST INFRASTRUCTURE ONLY: imported by tests/, the smoke check and the CPU baseline of
bench.py, never by the library or its binding. Plain float64 numpy/scipy.

What the paper fixes: the hyperparameters are the lengthscales l_i, the output scale
s and the noise variance of the kernel; they are fitted by a multistart scheme that
samples settings uniformly, keeps the fraction of highest likelihood and optimises
each kept setting with L-BFGS; gamma priors sit on the lengthscales (inputs are
normalised, so one prior serves every parameter).

READINGS (the paper gives no further detail):
  * parameters theta = (log l_1 .. log l_d, log s, t): l_i = e^theta_i, s = e^theta_d
    and noise variance = floor + e^t (floor an input, 1e-6 by default: without it the
    maximum drifts to interpolating, numerically singular kernels on nearly
    noise-free data); positivity without bounds; the uniform samples are drawn in this
    space by the caller;
  * objective: log p(y_f | theta) (the GP marginal likelihood of the feasible
    observations, zero prior mean) plus sum_i log Gamma(l_i; shape, rate), the gamma
    density in l itself (a MAP estimate of l; the log reparametrisation adds no
    Jacobian); samples are ranked by this same objective;
  * L-BFGS (Liu and Nocedal): memory of 10 pairs, the two-loop recursion for the
    direction with H0 = (s'y / y'y) I from the newest pair, backtracking (halving)
    from step 1 until the Armijo condition with c1 = 1e-4 holds (a kernel that is not
    finite and positive definite counts as a failed trial), pairs with s'y <= 1e-10 y'y are not
    stored, the first direction is the normalised steepest ascent; stop when
    max |grad| <= gtol, when the relative change of the objective is <= ftol, after
    max_iter accepted steps, or when 30 halvings do not satisfy Armijo.

Pins: tests/test_oracle_hyper.py (scikit-learn's GP marginal likelihood and its
gradient on an explicit embedding of every parameter type, central differences,
scipy's gamma density, closed-form optima, scipy's L-BFGS-B, recovery of generating
lengthscales, brute-force selection of the kept fraction).
"""
from __future__ import annotations

import math

import numpy as np
from scipy import linalg as sla
from scipy import special

from .gp_oracle import NUMERIC, PERM_DIST, SQRT5, encode, matern52, perm_dmax

LBFGS_MEMORY = 10
ARMIJO_C1 = 1e-4
MAX_HALVINGS = 30
CURVATURE_EPS = 1e-10


# ======================================================================== objective
def pair_terms(space, enc) -> np.ndarray:
    """T[p, i, j]: the squared per-parameter distance of Sec. 4.1 between configurations
    i and j, normalised to [0, 1] so that r^2 = sum_p T[p] / l_p^2 (Sec. 3.2):
    numeric (u_i - u_j)^2 of the float32 codes in float64, categorical [level differs],
    permutation semimetric / its maximum."""
    out = []
    for p, a in zip(space, enc):
        if p.kind in NUMERIC:
            d = a.astype(np.float64)[:, None] - a.astype(np.float64)[None, :]
            out.append(d * d)
        elif p.kind == "cat":
            out.append((a[:, None] != a[None, :]).astype(np.float64))
        else:
            out.append(PERM_DIST[p.dist](a, a).astype(np.float64) / perm_dmax(p))
    return np.stack(out)


def hyper_data(space, X, y, feasible):
    """(T, y_f): pair terms and targets of the feasible observations (the value model
    of Sec. 4.2 sees feasible observations only)."""
    fidx = np.nonzero(np.asarray(feasible).astype(bool))[0]
    enc = encode(space, X)
    return pair_terms(space, [e[fidx] for e in enc]), np.asarray(y, np.float64)[fidx]


def gamma_logpdf(l, shape, rate):
    """log of the gamma density rate^shape l^(shape-1) exp(-rate l) / Gamma(shape)."""
    l = np.asarray(l, np.float64)
    return shape * math.log(rate) - special.gammaln(shape) + (shape - 1.0) * np.log(l) - rate * l


def matern52_dr2(r2, s):
    """Derivative of the Matern-5/2 kernel with respect to r^2:
    d/dr [s (1 + sqrt5 r + 5 r^2/3) e^(-sqrt5 r)] / (2 r) = -(5/6) s (1 + sqrt5 r) e^(-sqrt5 r)."""
    r = np.sqrt(r2)
    return -(5.0 / 6.0) * s * (1.0 + SQRT5 * r) * np.exp(-SQRT5 * r)


def log_posterior(T, y, theta, prior=None, noise_floor=0.0, want_grad=True):
    """(value, gradient w.r.t. theta) of the objective; (-inf, None) when the kernel
    matrix is not finite or not positive definite, or the value or gradient overflows.

    value = -1/2 y' K^-1 y - 1/2 log det K - n/2 log 2 pi + sum_p log Gamma(l_p)
    d/d theta_q = 1/2 tr((alpha alpha' - K^-1) dK/d theta_q) + d prior / d theta_q
    (the textbook GP marginal likelihood and its gradient), with
      dK/d log l_p   = dk/dr^2 * (-2 T[p] / l_p^2),
      dK/d log s     = K - noise I,
      dK/d t         = e^t I   (noise = floor + e^t)."""
    theta = np.asarray(theta, np.float64)
    d, n = T.shape[0], len(y)
    if not np.all(np.isfinite(theta)):
        return -math.inf, None
    with np.errstate(over="ignore", invalid="ignore", divide="ignore"):
        l = np.exp(theta[:d])
        s = math.exp(min(theta[d], 709.0))
        en = math.exp(min(theta[d + 1], 709.0))
        noise = noise_floor + en
        r2 = np.zeros((n, n))
        for p in range(d):
            r2 += T[p] / (l[p] * l[p])
        Kf = matern52(r2, s)
        K = Kf + noise * np.eye(n)
    if not np.all(np.isfinite(K)):          # an overflowing setting is not a kernel
        return -math.inf, None
    try:
        with np.errstate(over="ignore", invalid="ignore"):
            L = np.linalg.cholesky(K)
    except np.linalg.LinAlgError:
        return -math.inf, None
    if not np.all(np.isfinite(L)):          # the factorisation overflowed
        return -math.inf, None
    alpha = sla.cho_solve((L, True), y)
    value = -0.5 * float(y @ alpha) - float(np.sum(np.log(np.diag(L)))) - 0.5 * n * math.log(2 * math.pi)
    if prior is not None:
        with np.errstate(over="ignore", invalid="ignore", divide="ignore"):
            value += float(np.sum(gamma_logpdf(l, *prior)))
    if not math.isfinite(value):
        return -math.inf, None
    if not want_grad:
        return value, None
    Kinv = sla.cho_solve((L, True), np.eye(n))
    G = np.outer(alpha, alpha) - Kinv
    dk = matern52_dr2(r2, s)
    grad = np.empty(d + 2)
    with np.errstate(over="ignore", invalid="ignore"):
        for p in range(d):
            grad[p] = 0.5 * float(np.sum(G * dk * (-2.0 * T[p] / (l[p] * l[p]))))
            if prior is not None:
                grad[p] += (prior[0] - 1.0) - prior[1] * l[p]
    grad[d] = 0.5 * float(np.sum(G * Kf))
    grad[d + 1] = 0.5 * en * float(np.trace(G))
    if not np.all(np.isfinite(grad)):
        return -math.inf, None
    return value, grad


# ========================================================================== L-BFGS
def lbfgs_maximize(fun, x0, max_iter=100, gtol=1e-5, ftol=1e-10):
    """Maximise fun (returning (value, gradient), value -inf where undefined) from x0
    with limited-memory BFGS (Liu and Nocedal) on F = -fun; see the readings in the
    module header. Returns (x, value, accepted steps, evaluations)."""
    x = np.asarray(x0, np.float64).copy()
    v, gv = fun(x)
    evals = 1
    if not np.isfinite(v):
        return x, v, 0, evals
    F, g = -v, -np.asarray(gv)
    S, Y = [], []                                   # stored pairs, oldest first
    it = 0
    while it < max_iter and np.max(np.abs(g)) > gtol:
        # direction: two-loop recursion over the stored pairs (steepest descent if none)
        if S:
            q = g.copy()
            a = [0.0] * len(S)
            for i in range(len(S) - 1, -1, -1):
                a[i] = float(S[i] @ q) / float(Y[i] @ S[i])
                q = q - a[i] * Y[i]
            r = (float(S[-1] @ Y[-1]) / float(Y[-1] @ Y[-1])) * q
            for i in range(len(S)):
                b = float(Y[i] @ r) / float(Y[i] @ S[i])
                r = r + (a[i] - b) * S[i]
            p = -r
        else:
            p = -g / math.sqrt(float(g @ g))
        slope = float(g @ p)
        if not slope < 0.0:                         # not a descent direction: restart
            S, Y = [], []
            p = -g / math.sqrt(float(g @ g))
            slope = float(g @ p)
        # backtracking line search (Armijo)
        t, accepted = 1.0, False
        for _ in range(MAX_HALVINGS + 1):
            xt = x + t * p
            vt, gvt = fun(xt)
            evals += 1
            if np.isfinite(vt) and -vt <= F + ARMIJO_C1 * t * slope:
                accepted = True
                break
            t *= 0.5
        if not accepted:
            break
        Ft, gt = -vt, -np.asarray(gvt)
        s_k, y_k = xt - x, gt - g
        if float(s_k @ y_k) > CURVATURE_EPS * float(y_k @ y_k):
            S.append(s_k)
            Y.append(y_k)
            if len(S) > LBFGS_MEMORY:
                S.pop(0)
                Y.pop(0)
        F_old = F
        x, F, g = xt, Ft, gt
        it += 1
        if abs(F_old - F) <= ftol * max(abs(F_old), abs(F), 1.0):
            break
    return x, -F, it, evals


# ======================================================================= multistart
def hyperfit(space, X, y, feasible, theta0, n_keep, prior=None, noise_floor=1e-6,
             max_iter=100, gtol=1e-5, ftol=1e-10) -> dict:
    """Multistart fit (Sec. 3.2): evaluate the objective at every sampled theta0 row,
    keep the n_keep best (lower index first on ties; -inf never ranks above a finite
    value) and run L-BFGS from each. Returns the sample objectives, the kept indices,
    the optimised thetas, their objectives and accepted steps, and the best of them."""
    T, yf = hyper_data(space, X, y, feasible)
    theta0 = np.asarray(theta0, np.float64)
    obj0 = np.array([log_posterior(T, yf, t, prior, noise_floor, want_grad=False)[0]
                     for t in theta0])
    order = np.lexsort((np.arange(len(obj0)), -obj0))
    keep = order[:min(n_keep, len(obj0))]
    fun = lambda t: log_posterior(T, yf, t, prior, noise_floor)
    out_theta, out_obj, out_it = [], [], []
    for k in keep:
        xk, vk, ik, _ = lbfgs_maximize(fun, theta0[k], max_iter, gtol, ftol)
        out_theta.append(xk)
        out_obj.append(vk)
        out_it.append(ik)
    out_obj = np.array(out_obj)
    best = int(np.lexsort((np.arange(len(out_obj)), -out_obj))[0])
    return {"obj0": obj0, "keep": keep, "theta": np.array(out_theta), "obj": out_obj,
            "iters": np.array(out_it), "best": best}
