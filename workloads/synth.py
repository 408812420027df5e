"""Seeded generators for the five synthetic workloads (C1..C5) and the Chain-of-Trees
example space.

Raw column formats (one numpy array per parameter, identical for the HIP library and
the oracle):

* ``real``: float64 ``[count]``, the parameter value.
* ``int``:  int32 ``[count]``, the integer value (``lo..hi`` inclusive).
* ``ord``:  int32 ``[count]``, the index of the value in ``Param.values`` (ascending).
* ``cat``:  int32 ``[count]``, the level ``0..levels-1``.
* ``perm``: int32 ``[count, m]``, row ``c`` holds ``pi`` with ``pi[i]`` = the 0-based
  position that item ``i`` takes in the new order (Sec. 4.1, permutation parameters).

Every random draw comes from a ``numpy.random.Generator`` seeded from the workload
number; candidates are drawn in independent chunks of ``CHUNK`` configurations so that
any prefix of whole chunks is the same at every requested ``M``.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Callable, List, Optional

import numpy as np

CHUNK = 4096


@dataclasses.dataclass(frozen=True)
class Param:
    name: str
    kind: str                      # 'real' | 'int' | 'ord' | 'cat' | 'perm'
    log2: bool = False             # distance on log2(value) (real/int/ord)
    lo: float = 0.0                # real/int lower bound (inclusive)
    hi: float = 1.0                # real/int upper bound (inclusive)
    values: tuple = ()             # ord: ascending values
    levels: int = 0                # cat: number of levels
    m: int = 0                     # perm: number of items
    dist: str = "spearman"         # perm: 'spearman' | 'kendall' | 'hamming' | 'naive'


@dataclasses.dataclass
class Workload:
    name: str
    space: List[Param]
    X: list                        # raw observation columns
    y: np.ndarray                  # float64 [n]; NaN where infeasible
    feasible: np.ndarray           # uint8 [n]
    C: list                        # raw candidate columns
    mask: Optional[np.ndarray]     # uint8 [M] known-constraint mask, None = all allowed
    lengthscale: np.ndarray        # float64 [d]
    signal_var: float
    noise_var: float
    cls_signal_var: Optional[float]  # None: no feasibility model (p_feas = 1)
    eps_f: float = 0.0
    description: str = ""

    @property
    def n(self) -> int:
        return int(self.y.shape[0])

    @property
    def M(self) -> int:
        return int(_count(self.C[0]))

    @property
    def d(self) -> int:
        return len(self.space)

    def candidate_slice(self, lo: int, hi: int) -> list:
        return [c[lo:hi] for c in self.C]


def _count(col: np.ndarray) -> int:
    return col.shape[0]


# --------------------------------------------------------------------------- sampling
def uniform_columns(space: List[Param], count: int, rng: np.random.Generator) -> list:
    """Draw ``count`` configurations uniformly at random from the (unconstrained) space."""
    cols = []
    for p in space:
        if p.kind == "real":
            cols.append(rng.uniform(p.lo, p.hi, size=count).astype(np.float64))
        elif p.kind == "int":
            cols.append(rng.integers(int(p.lo), int(p.hi) + 1, size=count).astype(np.int32))
        elif p.kind == "ord":
            cols.append(rng.integers(0, len(p.values), size=count).astype(np.int32))
        elif p.kind == "cat":
            cols.append(rng.integers(0, p.levels, size=count).astype(np.int32))
        elif p.kind == "perm":
            keys = rng.random((count, p.m))
            cols.append(np.argsort(keys, axis=1).astype(np.int32))
        else:
            raise ValueError(p.kind)
    return cols


def _chunked_candidates(space, M, seed, draw_chunk: Callable):
    """Concatenate independently seeded chunks of CHUNK candidates (prefix-stable in M)."""
    parts = []
    nchunks = (M + CHUNK - 1) // CHUNK
    for c in range(nchunks):
        rng = np.random.default_rng([seed, 7, c])
        parts.append(draw_chunk(rng, CHUNK))
    cols = [np.concatenate([p[i] for p in parts], axis=0)[:M] for i in range(len(space))]
    return cols


def _standardise_feasible(logrt: np.ndarray, feasible: np.ndarray) -> np.ndarray:
    f = feasible.astype(bool)
    mu = logrt[f].mean()
    sd = logrt[f].std()
    y = (logrt - mu) / sd
    y = y.astype(np.float64)
    y[~f] = np.nan
    return y


def _inversions(perm_rows: np.ndarray, ref: np.ndarray) -> np.ndarray:
    """Synthetic-objective feature: number of item pairs ordered differently from ``ref``."""
    m = perm_rows.shape[1]
    out = np.zeros(perm_rows.shape[0], dtype=np.int64)
    for i in range(m):
        for j in range(i + 1, m):
            out += ((perm_rows[:, i] < perm_rows[:, j]) != (ref[i] < ref[j]))
    return out


# --------------------------------------------------------------------------- C1
def _c1(M: int, n: int = 32) -> Workload:
    seed = 1001
    space = [
        Param("x0", "real", lo=0.0, hi=1.0),
        Param("x1", "real", lo=0.0, hi=1.0),
        Param("i0", "int", lo=1, hi=64),
        Param("o0", "ord", log2=True, values=(1, 2, 4, 8, 16)),
        Param("c0", "cat", levels=3),
    ]
    rng = np.random.default_rng(seed)
    X = uniform_columns(space, n, rng)
    a = rng.uniform(0.5, 1.0, size=4)
    om = rng.normal(size=(4, 5))
    ph = rng.uniform(0.0, 2 * math.pi, size=4)
    noise = rng.normal(size=n)

    def feat(cols):
        return np.stack([cols[0], cols[1], (cols[2] - 1) / 63.0, cols[3] / 4.0, cols[4] / 2.0], 1)

    z = feat(X)
    y = (a[None, :] * np.sin(2 * math.pi * z @ om.T + ph[None, :])).sum(1) + 0.01 * noise
    C = _chunked_candidates(space, M, seed, lambda r, k: uniform_columns(space, k, r))
    return Workload("C1", space, X, y.astype(np.float64), np.ones(n, np.uint8), C, None,
                    np.full(5, 0.5), 1.0, 1e-4, None, 0.0,
                    f"tiny mixed space d=5, n={n}")


# --------------------------------------------------------------------------- C2
def _c2(M: int) -> Workload:
    seed = 1002
    space = [
        Param("chunk", "ord", log2=True, values=tuple(2 ** k for k in range(9))),
        Param("unroll", "ord", log2=True, values=(1, 2, 4, 8)),
        Param("sched", "cat", levels=3),
        Param("threads", "int", lo=1, hi=64),
        Param("split", "int", lo=1, hi=32),
        Param("order", "perm", m=5, dist="kendall"),
    ]
    n = 128
    rng = np.random.default_rng(seed)
    X = uniform_columns(space, n, rng)
    G = rng.normal(size=(4, 4))
    A = G.T @ G / 4.0
    b = rng.normal(size=4)
    c = rng.normal(0.0, 0.5, size=3)
    pi0 = rng.permutation(5)
    eta = rng.normal(size=n)
    z = np.stack([X[0] / 8.0, X[1] / 3.0, (X[3] - 1) / 63.0, (X[4] - 1) / 31.0], 1)
    logrt = (np.einsum("ni,ij,nj->n", z, A, z) + z @ b + c[X[2]]
             + 0.3 * _inversions(X[5], pi0) / 10.0 + 0.05 * eta)
    feas = np.ones(n, np.uint8)
    y = _standardise_feasible(logrt, feas)
    C = _chunked_candidates(space, M, seed, lambda r, k: uniform_columns(space, k, r))
    d = len(space)
    return Workload("C2", space, X, y, feas, C, None, np.full(d, math.sqrt(d) / 2), 1.0, 1e-4,
                    None, 0.0, "sparse-tensor-schedule space d=6 (perm m=5, Kendall), n=128")


# --------------------------------------------------------------------------- C3
def _c3_space():
    vals = tuple(2 ** k for k in range(11))
    names = ["G0", "G1", "G2", "L0", "L1", "L2", "T0", "T1", "T2", "V"]
    return [Param(nm, "ord", log2=True, values=vals) for nm in names]


def c3_known_feasible(cols) -> np.ndarray:
    """Known constraints of the GPU-tile space, on level indices (= log2 of the value):
    T_k | L_k | G_k for k = 0..2, V | T_0, L_0 * L_1 * L_2 <= 1024."""
    e = [np.asarray(c) for c in cols]
    G, L, T, V = e[0:3], e[3:6], e[6:9], e[9]
    ok = np.ones(e[0].shape[0], dtype=bool)
    for k in range(3):
        ok &= (T[k] <= L[k]) & (L[k] <= G[k])
    ok &= V <= T[0]
    ok &= (L[0] + L[1] + L[2]) <= 10
    return ok


def _expand(prefix: np.ndarray, lo: np.ndarray, hi: np.ndarray) -> np.ndarray:
    """Children of every prefix row: values lo..hi (inclusive, none if hi < lo) appended,
    each prefix's children consecutive and ascending (lexicographic order is kept)."""
    cnt = np.maximum(hi - lo + 1, 0)
    rows = np.repeat(np.arange(len(prefix)), cnt)
    start = np.repeat(np.cumsum(cnt) - cnt, cnt)
    val = np.repeat(lo, cnt) + (np.arange(cnt.sum()) - start)
    return np.concatenate([prefix[rows], val[:, None].astype(prefix.dtype)], axis=1)


def c3_chain_leaves() -> np.ndarray:
    """Every known-feasible configuration of the GPU-tile space as level indices, one
    row each, in lexicographic order of the parameters G0 G1 G2 L0 L1 L2 T0 T1 T2 V (the
    leaves of its single tree: all ten parameters are linked by the constraints)."""
    P = np.zeros((1, 0), np.int8)
    for _ in range(3):                                    # G_k: any level
        P = _expand(P, np.zeros(len(P), np.int64), np.full(len(P), 10))
    for k in range(3):                                    # L_k <= G_k, sum L <= 10
        used = P[:, 3:3 + k].astype(np.int64).sum(axis=1)
        P = _expand(P, np.zeros(len(P), np.int64),
                    np.minimum(P[:, k].astype(np.int64), 10 - used))
    for k in range(3):                                    # T_k <= L_k
        P = _expand(P, np.zeros(len(P), np.int64), P[:, 3 + k].astype(np.int64))
    return _expand(P, np.zeros(len(P), np.int64), P[:, 6].astype(np.int64))  # V <= T_0


def _c3_feasible_uniform(space, count, rng):
    """Uniform draw from the known-feasible set, by exact counting: the three local
    sizes (exponents L_k, sum <= 10) are drawn with probability proportional to the
    number of feasible completions, then the rest of each chain given them (T_0 with
    weight T_0 + 1 for the V <= T_0 choices)."""
    trip, wts = [], []
    for a in range(11):
        for b in range(11 - a):
            for c in range(11 - a - b):
                w = (a + 1) * (a + 2) // 2 * (11 - a)
                w *= (b + 1) * (11 - b) * (c + 1) * (11 - c)
                trip.append((a, b, c))
                wts.append(w)
    trip = np.array(trip)
    p = np.array(wts, dtype=np.float64)
    p /= p.sum()
    L = trip[rng.choice(len(trip), size=count, p=p)]
    u = rng.random((count, 8))
    # T0 in 0..L0 with weight T0+1: inverse CDF of (t+1)(t+2)/2 / ((L0+1)(L0+2)/2)
    tot = (L[:, 0] + 1) * (L[:, 0] + 2) / 2.0
    T0 = np.floor((np.sqrt(1.0 + 8.0 * u[:, 0] * tot) - 1.0) / 2.0).astype(np.int64)
    T0 = np.minimum(T0, L[:, 0])
    V = np.floor(u[:, 1] * (T0 + 1)).astype(np.int64)
    T1 = np.floor(u[:, 2] * (L[:, 1] + 1)).astype(np.int64)
    T2 = np.floor(u[:, 3] * (L[:, 2] + 1)).astype(np.int64)
    G = [L[:, k] + np.floor(u[:, 4 + k] * (11 - L[:, k])).astype(np.int64) for k in range(3)]
    cols = [G[0], G[1], G[2], L[:, 0], L[:, 1], L[:, 2], T0, T1, T2, V]
    return [c.astype(np.int32) for c in cols]


def _c3(M: int) -> Workload:
    seed = 1003
    space = _c3_space()
    n = 256
    rng = np.random.default_rng(seed)
    X = _c3_feasible_uniform(space, n, rng)
    e = np.stack(X, 1).astype(np.float64)
    w = rng.normal(size=10)
    h = e @ w + 0.1 * rng.normal(size=n)
    n_inf = int(math.floor(0.3 * n))
    feas = np.ones(n, np.uint8)
    feas[np.argsort(-h, kind="stable")[:n_inf]] = 0
    G = rng.normal(size=(10, 10))
    A = G.T @ G / 10.0
    b = rng.normal(size=10)
    z = e / 10.0
    logrt = np.einsum("ni,ij,nj->n", z, A, z) + z @ b + 0.1 * rng.normal(size=n)
    y = _standardise_feasible(logrt, feas)

    def chunk(r, k):
        half = k // 2
        base = _c3_feasible_uniform(space, half, r)
        nb = [c.copy() for c in base]
        which = r.integers(0, len(space), size=half)
        shift = r.integers(1, 11, size=half)          # a different level of that param
        for i in range(len(space)):
            sel = which == i
            nb[i][sel] = (nb[i][sel] + shift[sel]) % 11
        return [np.concatenate([base[i], nb[i]]).astype(np.int32) for i in range(len(space))]

    C = _chunked_candidates(space, M, seed, chunk)
    mask = c3_known_feasible(C).astype(np.uint8)
    d = len(space)
    return Workload("C3", space, X, y, feas, C, mask, np.full(d, math.sqrt(d) / 2), 1.0, 1e-4,
                    1.0, 0.0, "GPU-tile space d=10 ordinals, known constraints masked, "
                    "hidden constraints (30% infeasible), n=256")


# --------------------------------------------------------------------------- C4
def _c4(M: int) -> Workload:
    seed = 1004
    space = ([Param(f"b{k}", "cat", levels=2) for k in range(12)]
             + [Param(f"u{k}", "ord", log2=True, values=(1, 2, 4, 8, 16, 32)) for k in range(6)]
             + [Param(f"p{k}", "int", lo=1, hi=128) for k in range(2)])
    n = 512
    rng = np.random.default_rng(seed)
    X = uniform_columns(space, n, rng)

    def feat(cols):
        return np.stack([c.astype(np.float64) for c in cols[:12]]
                        + [cols[12 + k] / 5.0 for k in range(6)]
                        + [(cols[18 + k] - 1) / 127.0 for k in range(2)], 1)

    z = feat(X)
    w = rng.normal(size=20)
    s = z @ w + 0.1 * rng.normal(size=n)
    n_inf = int(math.floor(0.3 * n))
    feas = np.ones(n, np.uint8)
    feas[np.argsort(-s, kind="stable")[:n_inf]] = 0
    main = rng.choice(20, size=8, replace=False)
    beta = rng.normal(size=8)
    pairs = np.stack([rng.choice(20, size=2, replace=False) for _ in range(10)])
    gam = rng.normal(size=10)
    logrt = (z[:, main] @ beta + (z[:, pairs[:, 0]] * z[:, pairs[:, 1]]) @ gam
             + 0.1 * rng.normal(size=n))
    y = _standardise_feasible(logrt, feas)
    C = _chunked_candidates(space, M, seed, lambda r, k: uniform_columns(space, k, r))
    d = len(space)
    return Workload("C4", space, X, y, feas, C, None, np.full(d, math.sqrt(d) / 2), 1.0, 1e-4,
                    1.0, 0.0, "FPGA-pragma space d=20 (12 binary cat, 6 ord, 2 int), n=512, "
                    "30% infeasible")


# --------------------------------------------------------------------------- C5
def _c5(M: int) -> Workload:
    seed = 1005
    space = ([Param(f"o{k}", "ord", log2=True, values=tuple(2 ** j for j in range(7)))
              for k in range(6)]
             + [Param(f"r{k}", "real", lo=0.0, hi=1.0) for k in range(2)]
             + [Param(f"c{k}", "cat", levels=8) for k in range(2)]
             + [Param("pa", "perm", m=7, dist="spearman"), Param("pb", "perm", m=7, dist="hamming")])
    n = 2048
    rng = np.random.default_rng(seed)
    X = uniform_columns(space, n, rng)
    z = np.stack([X[k] / 6.0 for k in range(6)] + [X[6], X[7]], 1)
    G = rng.normal(size=(8, 8))
    A = G.T @ G / 8.0
    b = rng.normal(size=8)
    cc = rng.normal(0.0, 0.5, size=(2, 8))
    ref_a = rng.permutation(7)
    ref_b = rng.permutation(7)
    disp = ((X[10] - ref_a[None, :]) ** 2).sum(1)          # squared displacement of items
    moved = (X[11] != ref_b[None, :]).sum(1)                # items not at their ref position
    logrt = (np.einsum("ni,ij,nj->n", z, A, z) + z @ b + cc[0, X[8]] + cc[1, X[9]]
             + 0.5 * disp / 112.0 + 0.5 * moved / 7.0 + 0.1 * rng.normal(size=n))
    feas = np.ones(n, np.uint8)
    y = _standardise_feasible(logrt, feas)
    ls = np.exp(rng.uniform(math.log(0.1), math.log(10.0), size=len(space)))
    C = _chunked_candidates(space, M, seed, lambda r, k: uniform_columns(space, k, r))
    return Workload("C5", space, X, y, feas, C, None, ls, 1.0, 1e-4, None, 0.0,
                    "stress d=12 (2 perms m=7 Spearman/Hamming), n=2048, "
                    "lengthscales log-uniform [0.1, 10]")


WORKLOADS = {
    "C1": (_c1, 4096),
    "C2": (_c2, 65536),
    "C3": (_c3, 262144),
    "C4": (_c4, 1048576),
    "C5": (_c5, 1048576),
}


def make_workload(name: str, M: Optional[int] = None, n: Optional[int] = None) -> Workload:
    """Build workload ``name`` with its full candidate count, or the first ``M``. ``n``
    overrides the observation count of C1 (same draws for the default n = 32), which
    gives large-n cases of the same space."""
    fn, full = WORKLOADS[name]
    M = full if M is None else int(M)
    if n is None:
        return fn(M)
    if name != "C1":
        raise ValueError("only C1 takes an observation count")
    return fn(M, int(n))


# --------------------------------------------------------------------------- CoT example
def cot_example_space():
    """The five-parameter example space of the Chain-of-Trees passage (Sec. 4.2)."""
    return [
        Param("p1", "ord", values=(2, 4)),
        Param("p2", "ord", values=(2, 4)),
        Param("p3", "ord", values=(1, 4)),
        Param("p4", "ord", values=(1, 2, 4)),
        Param("p5", "ord", values=(2, 4, 8)),
    ]


def cot_example_constraints(vals) -> np.ndarray:
    """Its three known constraints on parameter values: p1>=p2, p4>=p3, p5>=2*p4."""
    p1, p2, p3, p4, p5 = [np.asarray(v) for v in vals]
    return (p1 >= p2) & (p4 >= p3) & (p5 >= 2 * p4)


# --------------------------------------------------------------------- hyper starts
# Log-uniform box of the sampled hyperparameter settings (the caller's random draws for
# the multistart fit): lengthscales and output scale in [0.1, 10], noise variance in
# [1e-6, 1]. Inputs are normalised to [0, 1] and y is standardised, so one box serves
# every workload.
HYPER_BOX_LOG_L = (math.log(0.1), math.log(10.0))
HYPER_BOX_LOG_S = (math.log(0.1), math.log(10.0))
HYPER_BOX_LOG_NOISE = (math.log(1e-6), math.log(1.0))


def hyper_starts(d: int, count: int, seed: int) -> np.ndarray:
    """count x (d + 2) settings (log l_1..log l_d, log s, log noise) drawn uniformly in
    the box above from numpy's generator seeded with `seed`."""
    rng = np.random.default_rng(seed)
    lo = np.array([HYPER_BOX_LOG_L[0]] * d + [HYPER_BOX_LOG_S[0], HYPER_BOX_LOG_NOISE[0]])
    hi = np.array([HYPER_BOX_LOG_L[1]] * d + [HYPER_BOX_LOG_S[1], HYPER_BOX_LOG_NOISE[1]])
    return lo + (hi - lo) * rng.random((count, d + 2))
