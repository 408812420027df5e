"""CPU fp64 oracle for BaCO's GP + EI candidate scoring (Hellsten et al., arXiv 2212.11142).

TEST INFRASTRUCTURE ONLY. Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this module. The HIP library never calls
it and shares no code with it; the two meet only in the seeded raw inputs drawn by
``workloads``.

Everything here is the plain, slow definition in float64 (numpy/scipy), with library
primitives (Cholesky, triangular solves, erfc) used as single steps. Readings of the
paper where it is silent or garbled are marked READING and listed in the design notes.

Pinning status (see tests/test_oracle_pins.py): encoding, per-parameter distances,
the Matern-5/2 kernel, the GP posterior, EI, the Laplace probit classifier and the
local-search acquisition optimiser are each pinned against closed forms, brute force,
independent library routines or the paper's worked examples. Nothing in this module is
"parity unpinned".
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import List, Optional

import numpy as np
from scipy import linalg as sla
from scipy import special

NUMERIC = ("real", "int", "ord")
SQRT5 = math.sqrt(5.0)


# =============================================================================== encoding
def transformed_range(p):
    """Transformed (lo, hi) of a numeric parameter: identity or log2 (Sec. 4.1, numeric
    parameters; Sec. 4.2 on exponential parameters)."""
    t = np.log2 if p.log2 else (lambda v: v)
    if p.kind == "ord":
        vals = np.asarray(p.values, dtype=np.float64)
        return float(t(vals[0])), float(t(vals[-1]))
    return float(t(np.float64(p.lo))), float(t(np.float64(p.hi)))


def encode_numeric(p, col) -> np.ndarray:
    """Normalised code u = fl32((t(v) - t_lo) / (t_hi - t_lo)) (Sec. 3.2, input
    normalisation; Sec. 4.1/4.2, log transform of exponential parameters).

    READING: normalisation is min-max over the declared range after the optional log2;
    each operation is one IEEE float64 operation and the quotient is rounded once to
    float32 (the float32 code is what both the model and the scorer consume)."""
    col = np.asarray(col)
    if p.kind == "ord":
        v = np.asarray(p.values, dtype=np.float64)[col.astype(np.int64)]
    else:
        v = col.astype(np.float64)
    t = np.log2(v) if p.log2 else v
    t_lo, t_hi = transformed_range(p)
    den = t_hi - t_lo
    if den == 0.0:
        return np.zeros(v.shape, dtype=np.float32)
    return ((t - t_lo) / den).astype(np.float32)


def encode(space, cols) -> list:
    """Per parameter: float32 codes (numeric), int64 levels (categorical), int64
    position vectors [count, m] (permutations, pi[i] = position of item i)."""
    out = []
    for p, c in zip(space, cols):
        if p.kind in NUMERIC:
            out.append(encode_numeric(p, c))
        elif p.kind == "cat":
            out.append(np.asarray(c).astype(np.int64))
        elif p.kind == "perm":
            out.append(np.asarray(c).astype(np.int64).reshape(-1, p.m))
        else:
            raise ValueError(p.kind)
    return out


# =============================================================================== distances
def kendall(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    """Kendall distance: number of item pairs whose relative order differs between the
    two permutations (Sec. 4.1 and the Fig. 3 caption). a: [Na, m], b: [Nb, m] position
    vectors -> [Na, Nb].

    READING: the double sum printed in Sec. 4.1 is garbled (it does not count discordant
    pairs); the text and figure define the count used here."""
    m = a.shape[1]
    out = np.zeros((a.shape[0], b.shape[0]), dtype=np.int64)
    for i in range(m):
        for j in range(i + 1, m):
            oa = (a[:, i] > a[:, j])[:, None]
            ob = (b[:, i] > b[:, j])[None, :]
            out += (oa != ob)
    return out


def spearman(a, b):
    """Spearman distance: sum over items of the squared change of position (Sec. 4.1)."""
    diff = a[:, None, :] - b[None, :, :]
    return (diff * diff).sum(-1)


def perm_hamming(a, b):
    """Permutation Hamming distance: number of items whose position changed (Sec. 4.1)."""
    return (a[:, None, :] != b[None, :, :]).sum(-1)


def perm_naive(a, b):
    """Permutation treated as one categorical value: 0 if identical else 1 (Sec. 4.1,
    the naive alternative; Sec. 5.3 ablation)."""
    return (a[:, None, :] != b[None, :, :]).any(-1).astype(np.int64)


PERM_DIST = {"kendall": kendall, "spearman": spearman, "hamming": perm_hamming,
             "naive": perm_naive}


def perm_dmax(p) -> float:
    """Largest value of the permutation semimetric over m items (range normalisation).
    Kendall: m(m-1)/2 (full reversal); Spearman: (m^3 - m)/3 (reversal); Hamming: m;
    naive: 1.

    READING: permutation semimetrics are divided by their maximum so that, like the
    normalised numeric codes, they lie in [0, 1] before the lengthscale weighting."""
    m = p.m
    if p.dist == "kendall":
        return m * (m - 1) / 2.0
    if p.dist == "spearman":
        return (m ** 3 - m) / 3.0
    if p.dist == "hamming":
        return float(m)
    if p.dist == "naive":
        return 1.0
    raise ValueError(p.dist)


def param_term(p, a, b) -> np.ndarray:
    """Per-parameter distance term between code arrays a [Na] and b [Nb] (Sec. 4.1):
    numeric -> the float32 difference fl32(u_a - u_b) (its square enters the distance);
    categorical -> 1[a != b]; permutation -> the integer semimetric value."""
    if p.kind in NUMERIC:
        return (a.astype(np.float64)[:, None] - b.astype(np.float64)[None, :]).astype(np.float32)
    if p.kind == "cat":
        return (a[:, None] != b[None, :]).astype(np.int64)
    return PERM_DIST[p.dist](a, b)


def sqdist(space, ea, eb, lengthscale) -> np.ndarray:
    """Weighted squared distance r^2 = sum_i d_i^2 / l_i^2 (Sec. 3.2, second kernel
    equation) with d_i the per-parameter distance of Sec. 4.1.

    Numeric parameters use d_i = |u - u'| on the normalised codes; categorical d_i is the
    0/1 Hamming indicator (its square is itself).

    READING: each permutation semimetric is already a squared Euclidean distance of an
    embedding of the permutation (pair indicators for Kendall, positions for Spearman,
    one-hot positions for Hamming), so it enters r^2 as is, divided by its maximum;
    squaring it again would not give a positive semidefinite kernel."""
    r2 = np.zeros((ea[0].shape[0], eb[0].shape[0]), dtype=np.float64)
    for p, a, b, l in zip(space, ea, eb, lengthscale):
        l2 = float(l) * float(l)
        if p.kind in NUMERIC:
            diff = a.astype(np.float64)[:, None] - b.astype(np.float64)[None, :]
            r2 += diff * diff / l2
        elif p.kind == "cat":
            r2 += (a[:, None] != b[None, :]).astype(np.float64) / l2
        else:
            r2 += PERM_DIST[p.dist](a, b).astype(np.float64) / (perm_dmax(p) * l2)
    return r2


def matern52(r2, signal_var: float) -> np.ndarray:
    """Matern-5/2 kernel of the distance r = sqrt(r2) (Sec. 3.2, first kernel equation):
    k = s (1 + sqrt5 r + 5 r^2 / 3) exp(-sqrt5 r).

    READING: the printed quadratic coefficient lacks the 1/3 of the textbook Matern-5/2
    kernel the paper cites; without it the function is not positive definite, so the
    textbook form is used. s is the output scale, a variance multiplier."""
    r = np.sqrt(r2)
    return signal_var * (1.0 + SQRT5 * r + (5.0 / 3.0) * r2) * np.exp(-SQRT5 * r)


def kernel(space, ea, eb, lengthscale, signal_var) -> np.ndarray:
    return matern52(sqdist(space, ea, eb, lengthscale), signal_var)


# =============================================================================== normal
def norm_cdf(z):
    return 0.5 * special.erfc(-np.asarray(z, dtype=np.float64) / math.sqrt(2.0))


def norm_pdf(z):
    z = np.asarray(z, dtype=np.float64)
    return np.exp(-0.5 * z * z) / math.sqrt(2.0 * math.pi)


# =============================================================================== EI
def expected_improvement(mu, sigma, fstar):
    """Expected improvement for minimisation (Sec. 3.3): E[max(f* - f, 0)] with
    f ~ N(mu, sigma^2), i.e. (f* - mu) Phi(z) + sigma phi(z), z = (f* - mu) / sigma;
    for sigma = 0 it is max(f* - mu, 0).

    READING: 'noise free' EI uses the latent variance (no observation noise added) and
    f* = the best (lowest) observed feasible value; no exploration margin."""
    mu = np.asarray(mu, dtype=np.float64)
    sigma = np.asarray(sigma, dtype=np.float64)
    imp = fstar - mu
    out = np.maximum(imp, 0.0)
    pos = sigma > 0
    z = np.where(pos, imp / np.where(pos, sigma, 1.0), 0.0)
    ei = imp * norm_cdf(z) + sigma * norm_pdf(z)
    return np.where(pos, ei, out)


# =============================================================================== classifier
def _probit_grad_w(f, t):
    """d/df log Phi(t f) and W = -d^2/df^2 log Phi(t f) for the probit likelihood."""
    logphi = -0.5 * f * f - 0.5 * math.log(2.0 * math.pi)
    r = np.exp(logphi - special.log_ndtr(t * f))          # phi(f) / Phi(t f)
    grad = t * r
    W = r * r + t * f * r
    return grad, W


def laplace_probit_fit(K, t, tol=1e-10, max_iter=100):
    """Mode of the Laplace approximation for GP binary classification with a probit
    likelihood, by Newton's method in the numerically stable B = I + W^1/2 K W^1/2 form
    (Rasmussen & Williams 2006, Sec. 3.4; the textbook the paper cites for its GP).
    Returns (f_hat, grad at f_hat, sqrt(W) at f_hat, chol(B) at f_hat, iterations).

    READING: the paper's feasibility model is a random forest (Sec. 4.2, hidden
    constraints); this GP classifier stands in for it and shares the regression
    lengthscales, with its own output scale and no noise term."""
    n = K.shape[0]
    f = np.zeros(n)
    it = 0
    for it in range(1, max_iter + 1):
        grad, W = _probit_grad_w(f, t)
        sw = np.sqrt(W)
        B = np.eye(n) + sw[:, None] * K * sw[None, :]
        L = np.linalg.cholesky(B)
        b = W * f + grad
        c = sw * (K @ b)
        z = sla.solve_triangular(L, c, lower=True)
        z = sla.solve_triangular(L.T, z, lower=False)
        a = b - sw * z
        f_new = K @ a
        delta = np.max(np.abs(f_new - f))
        f = f_new
        if delta < tol:
            break
    grad, W = _probit_grad_w(f, t)
    sw = np.sqrt(W)
    B = np.eye(n) + sw[:, None] * K * sw[None, :]
    L = np.linalg.cholesky(B)
    return f, grad, sw, L, it


# =============================================================================== model
@dataclass
class OracleModel:
    space: list
    enc_f: list               # encoded feasible observations
    enc_all: list             # encoded observations (all)
    lengthscale: np.ndarray
    signal_var: float
    noise_var: float
    K: np.ndarray             # Gram of the feasible observations incl. noise
    L: np.ndarray             # its Cholesky factor
    alpha: np.ndarray
    fstar: float
    feas_idx: np.ndarray
    cls_signal_var: Optional[float] = None
    cls_f: Optional[np.ndarray] = None
    cls_grad: Optional[np.ndarray] = None
    cls_sw: Optional[np.ndarray] = None
    cls_L: Optional[np.ndarray] = None
    cls_iters: int = 0


def fit(space, X, y, feasible, lengthscale, signal_var, noise_var,
        cls_signal_var=None) -> OracleModel:
    """GP fit (Sec. 3.2): K = k(X_f, X_f) + noise_var I over the feasible observations
    (known-infeasible points never enter the value model, Sec. 4.2), L = chol(K),
    alpha = K^-1 y_f, f* = min y_f. With cls_signal_var, also the feasibility
    classifier on all observations, label +1 feasible / -1 infeasible."""
    feasible = np.asarray(feasible).astype(bool)
    enc = encode(space, X)
    fidx = np.nonzero(feasible)[0]
    enc_f = [e[fidx] for e in enc]
    yf = np.asarray(y, dtype=np.float64)[fidx]
    K = kernel(space, enc_f, enc_f, lengthscale, signal_var) + noise_var * np.eye(len(fidx))
    L = np.linalg.cholesky(K)
    alpha = sla.cho_solve((L, True), yf)
    model = OracleModel(space, enc_f, enc, np.asarray(lengthscale, np.float64), signal_var,
                        noise_var, K, L, alpha, float(yf.min()), fidx)
    if cls_signal_var is not None:
        t = np.where(feasible, 1.0, -1.0)
        Kc = kernel(space, enc, enc, lengthscale, cls_signal_var)
        f, grad, sw, Lb, it = laplace_probit_fit(Kc, t)
        model.cls_signal_var = cls_signal_var
        model.cls_f, model.cls_grad, model.cls_sw, model.cls_L = f, grad, sw, Lb
        model.cls_iters = it
    return model


def score(model: OracleModel, C, mask=None, eps_f=0.0, chunk=8192) -> dict:
    """Posterior mean/variance of the latent objective, EI, probability of
    feasibility and the acquisition value for candidate columns C.

    mu = k*^T K^-1 y_f, sigma^2 = s - k*^T K^-1 k* (textbook GP regression; the paper
    gives the model but not these formulas). p = Phi(fbar / sqrt(1 + V)) with
    fbar = k_c*^T grad, V = s_c - |L_B^-1 W^1/2 k_c*|^2 (Laplace probit predictive).
    acq = EI * p where p > eps_f (only configurations whose probability of feasibility
    exceeds the minimum feasible limit are considered) and the candidate is allowed,
    else 0 (Sec. 4.2)."""
    encC = encode(model.space, C)
    M = encC[0].shape[0]
    out = {k: np.empty(M) for k in ("mu", "sigma", "ei", "p_feas", "acq")}
    for lo in range(0, M, chunk):
        hi = min(M, lo + chunk)
        ec = [e[lo:hi] for e in encC]
        ks = kernel(model.space, ec, model.enc_f, model.lengthscale, model.signal_var)
        mu = ks @ model.alpha
        q = np.einsum("ij,ji->i", ks, sla.cho_solve((model.L, True), ks.T))
        var = np.maximum(model.signal_var - q, 0.0)
        sig = np.sqrt(var)
        ei = expected_improvement(mu, sig, model.fstar)
        if model.cls_signal_var is not None:
            kc = kernel(model.space, ec, model.enc_all, model.lengthscale, model.cls_signal_var)
            fbar = kc @ model.cls_grad
            v = sla.solve_triangular(model.cls_L, (model.cls_sw[:, None] * kc.T), lower=True)
            V = np.maximum(model.cls_signal_var - (v * v).sum(0), 0.0)
            p = norm_cdf(fbar / np.sqrt(1.0 + V))
        else:
            p = np.ones(hi - lo)
        allowed = np.ones(hi - lo, dtype=bool) if mask is None else np.asarray(mask[lo:hi]).astype(bool)
        acq = np.where(allowed & (p > eps_f), ei * p, 0.0)
        out["mu"][lo:hi] = mu
        out["sigma"][lo:hi] = sig
        out["ei"][lo:hi] = ei
        out["p_feas"][lo:hi] = p
        out["acq"][lo:hi] = acq
    return out


def terms(space, encC, encX) -> np.ndarray:
    """All per-parameter terms [Nc, Nx, d] as float64 (numeric entries are the float32
    differences, exactly representable)."""
    ts = [param_term(p, a, b).astype(np.float64) for p, a, b in zip(space, encC, encX)]
    return np.stack(ts, axis=-1)


# ===================================================================== local search
# Acquisition optimiser of Sec. 3.3: uniformly sampled candidates are scored, the best
# become starting points, and each start climbs through one-parameter neighbours.
# READING (the paper gives no more detail): the neighbours of a configuration, in this
# order, parameter by parameter in space order --
#   real      the transformed value (log2 if flagged) minus, then plus, 1/16 of its
#             transformed range; a step leaving the range is not a neighbour;
#   int       value - 1, value + 1 (within lo..hi);
#   ord       index - 1, index + 1 (within the values);
#   cat       every other level, ascending;
#   perm      every exchange of the positions of two items i < j, (i, j) ascending.
# A climb moves to its best neighbour (largest acquisition value, first in this order
# on ties) while that is strictly larger than the current value, for at most
# `max_steps` moves. Known-constraint masks apply to the sampled candidates only (the
# generated neighbours are checked against the declared ranges alone).
REAL_STEP_DIV = 16.0


def neighbour_moves(space) -> list:
    """(parameter index, move) of every one-parameter neighbour, in order."""
    moves = []
    for i, p in enumerate(space):
        if p.kind in NUMERIC:
            moves += [(i, -1), (i, +1)]
        elif p.kind == "cat":
            moves += [(i, j) for j in range(p.levels - 1)]
        elif p.kind == "perm":
            moves += [(i, (a, b)) for a in range(p.m) for b in range(a + 1, p.m)]
        else:
            raise ValueError(p.kind)
    return moves


def apply_move(space, row, move):
    """Neighbour of configuration `row` (one value per parameter: float real, int
    int/ord/cat, tuple perm) under `move`; None if the move leaves the declared range."""
    i, mv = move
    p = space[i]
    out = list(row)
    if p.kind == "real":
        t_lo, t_hi = transformed_range(p)
        t = math.log2(row[i]) if p.log2 else float(row[i])
        t2 = t + mv * (t_hi - t_lo) / REAL_STEP_DIV
        if not (t_lo <= t2 <= t_hi):
            return None
        out[i] = 2.0 ** t2 if p.log2 else t2
    elif p.kind == "int":
        v = int(row[i]) + mv
        if v < p.lo or v > p.hi:
            return None
        out[i] = v
    elif p.kind == "ord":
        v = int(row[i]) + mv
        if v < 0 or v >= len(p.values):
            return None
        out[i] = v
    elif p.kind == "cat":
        out[i] = mv if mv < int(row[i]) else mv + 1
    else:
        a, b = mv
        pi = list(row[i])
        pi[a], pi[b] = pi[b], pi[a]
        out[i] = tuple(pi)
    return out


def rows_of(space, cols, idx) -> list:
    """Configurations idx of raw columns as rows."""
    rows = []
    for j in idx:
        row = []
        for p, c in zip(space, cols):
            if p.kind == "real":
                row.append(float(np.asarray(c)[j]))
            elif p.kind == "perm":
                row.append(tuple(int(v) for v in np.asarray(c).reshape(-1, p.m)[j]))
            else:
                row.append(int(np.asarray(c)[j]))
        rows.append(row)
    return rows


def cols_of(space, rows) -> list:
    """Raw columns of a list of configuration rows (the formats of `workloads`)."""
    cols = []
    for i, p in enumerate(space):
        if p.kind == "real":
            cols.append(np.array([r[i] for r in rows], dtype=np.float64))
        elif p.kind == "perm":
            cols.append(np.array([r[i] for r in rows], dtype=np.int32).reshape(-1, p.m))
        else:
            cols.append(np.array([r[i] for r in rows], dtype=np.int32))
    return cols


def local_search(model: OracleModel, C, mask=None, eps_f=0.0, n_starts=8, max_steps=32) -> dict:
    """Multi-start local search (Sec. 3.3): score the candidates C, take the n_starts of
    largest acquisition value (lowest index first on ties) and climb from each.
    Returns start indices, final rows, final acquisition values and moves per start, and
    per start the margin of its decisions: the smallest gap, over the steps taken and the
    final stop, between the best neighbour value and the runner-up or the current value
    (a path whose margin exceeds the rounding of the scores is the same in any precision)."""
    space = model.space
    acq0 = score(model, C, mask, eps_f)["acq"]
    M = len(acq0)
    order = np.lexsort((np.arange(M), -acq0))
    starts = order[:min(n_starts, M)]
    moves = neighbour_moves(space)
    out_rows, out_acq, out_steps, out_margin = [], [], [], []
    for row, a in zip(rows_of(space, C, starts), acq0[starts]):
        steps, margin = 0, math.inf
        while steps < max_steps:
            nbs = [apply_move(space, row, mv) for mv in moves]
            ok = np.array([nb is not None for nb in nbs], dtype=np.uint8)
            nb_rows = [nb if nb is not None else row for nb in nbs]
            acq = score(model, cols_of(space, nb_rows), ok, eps_f)["acq"]
            j = int(np.argmax(acq))
            margin = min(margin, abs(float(acq[j]) - a))
            if not acq[j] > a:
                break
            if len(acq) > 1:
                margin = min(margin, float(acq[j] - np.max(np.delete(acq, j))))
            row, a, steps = nb_rows[j], float(acq[j]), steps + 1
        out_rows.append(row)
        out_acq.append(float(a))
        out_steps.append(steps)
        out_margin.append(margin)
    return {"start_index": starts, "rows": out_rows, "acq": np.array(out_acq),
            "steps": np.array(out_steps), "margin": np.array(out_margin)}
