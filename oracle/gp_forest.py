"""CPU oracle of the random-forest feasibility model (Sec. 4.2, hidden constraints).

TEST INFRASTRUCTURE ONLY: imported by tests/, the smoke check and the CPU baseline of
bench.py, never by the library or its binding. Plain Python integers, fractions and
numpy.

What the paper fixes: a random forest is fitted to the feasible / infeasible labels of
the observations and predicts a probability of feasibility for every configuration,
which multiplies the expected improvement.

READINGS (the paper gives no further detail; classification forests as usually
defined: CART trees on bootstrap samples with a random feature subset per node):
  * features, one per parameter in space order: REAL and INT values, ORD index, CAT
    level (an ordered code), PERM one feature per item (its position);
  * tree t draws its bootstrap sample of n observation indices with replacement, index
    i from word i of the stream (t, 0); node k (breadth-first numbering, root 0,
    children numbered in order when their parent splits, left first) considers
    mtry = max(1, floor(sqrt(F))) features: a partial Fisher-Yates shuffle of 0..F-1
    with word q of the stream (t, k + 1) choosing position q + floor(u (F - q) / 2^64);
    streams are Philox4x64-10 with key (seed, 0) and counter (t, s, b, 3) for block b of
    stream s; words are used in order, four per block;
  * a split of a node on feature f at threshold v sends x_f <= v left; candidate
    thresholds are the node's distinct values of f except the largest; the quality of
    a split is the Gini impurity of the children weighted by their sizes, equivalently
    Q = pos_L neg_L / c_L + pos_R neg_R / c_R (pos/neg: feasible/infeasible counts,
    bootstrap duplicates counted); the best split has the smallest Q, then the
    smallest feature index, then the smallest threshold, compared exactly (rational
    arithmetic);
  * a node becomes a leaf when it is pure, has fewer than min_split samples, is at
    max_depth, has no candidate threshold, or its best split does not lower Q below
    the node's own pos neg / c; a leaf predicts pos / c;
  * the forest predicts the mean of its trees' leaf values, summed in tree order.

Pins: tests/test_oracle_forest.py (scikit-learn's decision tree on data without ties,
brute-force best split with rationals, numpy's Philox stream, a threshold rule
recovered from noisy labels, invariants of the fitted trees).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from fractions import Fraction
from typing import List

import numpy as np

from .gp_cot import philox4x64, uniform_index


def features(space, cols) -> np.ndarray:
    """[N, F] float64 feature matrix of raw columns (see the readings)."""
    out = []
    for p, c in zip(space, cols):
        c = np.asarray(c)
        if p.kind == "perm":
            out += [c.reshape(-1, p.m)[:, i].astype(np.float64) for i in range(p.m)]
        else:
            out.append(c.astype(np.float64))
    return np.stack(out, axis=1)


def stream_words(seed: int, t: int, s: int, count: int) -> List[int]:
    out, b = [], 0
    while len(out) < count:
        out += philox4x64((t, s, b, 3), (seed, 0))
        b += 1
    return out[:count]


@dataclass
class Tree:
    feature: List[int] = field(default_factory=list)     # -1 for a leaf
    threshold: List[float] = field(default_factory=list)
    left: List[int] = field(default_factory=list)        # right child = left + 1
    value: List[float] = field(default_factory=list)     # leaf: pos / c
    depth: List[int] = field(default_factory=list)


def best_split(x: np.ndarray, lab: np.ndarray):
    """(Q, threshold) of the best split of one feature over the node's samples (x with
    duplicates, lab in {0, 1}), or None without a candidate threshold."""
    order = np.argsort(x, kind="stable")
    xs, ls = x[order], lab[order]
    c = len(xs)
    pos = int(ls.sum())
    best = None
    pl = 0
    for i in range(c - 1):
        pl += int(ls[i])
        if xs[i] == xs[i + 1]:
            continue
        cl, cr = i + 1, c - i - 1
        pr = pos - pl
        q = Fraction(pl * (cl - pl), cl) + Fraction(pr * (cr - pr), cr)
        if best is None or q < best[0]:
            best = (q, float(xs[i]))
    return best


def fit_tree(X: np.ndarray, y: np.ndarray, t: int, seed: int, max_depth: int, min_split: int,
             bootstrap: bool = True, mtry: int = None) -> Tree:
    n, F = X.shape
    mtry = max(1, int(math.isqrt(F))) if mtry is None else mtry
    if bootstrap:
        idx = np.array([uniform_index(u, n) for u in stream_words(seed, t, 0, n)], dtype=np.int64)
    else:
        idx = np.arange(n)
    tree = Tree()
    samples = [idx]
    tree.feature.append(-1); tree.threshold.append(0.0); tree.left.append(-1)
    tree.value.append(0.0); tree.depth.append(0)
    k = 0
    while k < len(tree.feature):                                   # breadth first
        s = samples[k]
        lab = y[s].astype(np.int64)
        c, pos = len(s), int(lab.sum())
        tree.value[k] = pos / c
        if pos == 0 or pos == c or c < min_split or tree.depth[k] >= max_depth:
            k += 1
            continue
        perm = list(range(F))
        for q, u in enumerate(stream_words(seed, t, k + 1, mtry)):
            r = q + uniform_index(u, F - q)
            perm[q], perm[r] = perm[r], perm[q]
        best = None                                                 # (Q, feature, thr)
        for f in sorted(perm[:mtry]):
            b = best_split(X[s, f], lab)
            if b is not None and (best is None or b[0] < best[0]):
                best = (b[0], f, b[1])
        if best is None or not best[0] < Fraction(pos * (c - pos), c):
            k += 1
            continue
        _, f, thr = best
        go_left = X[s, f] <= thr
        tree.feature[k], tree.threshold[k], tree.left[k] = f, thr, len(tree.feature)
        for part in (s[go_left], s[~go_left]):
            samples.append(part)
            tree.feature.append(-1); tree.threshold.append(0.0); tree.left.append(-1)
            tree.value.append(0.0); tree.depth.append(tree.depth[k] + 1)
        k += 1
    return tree


def fit_forest(space, X_cols, feasible, n_trees: int, seed: int, max_depth: int = 16,
               min_split: int = 2) -> List[Tree]:
    X = features(space, X_cols)
    y = np.asarray(feasible).astype(np.int64)
    return [fit_tree(X, y, t, seed, max_depth, min_split) for t in range(n_trees)]


def tree_predict(tree: Tree, X: np.ndarray) -> np.ndarray:
    out = np.empty(len(X))
    for j, x in enumerate(X):
        k = 0
        while tree.feature[k] >= 0:
            k = tree.left[k] + (0 if x[tree.feature[k]] <= tree.threshold[k] else 1)
        out[j] = tree.value[k]
    return out


def predict(space, forest: List[Tree], C_cols) -> np.ndarray:
    """Probability of feasibility: the mean of the trees' leaf values (float64)."""
    X = features(space, C_cols)
    acc = np.zeros(len(X))
    for tree in forest:
        acc = acc + tree_predict(tree, X)
    return acc / len(forest)
