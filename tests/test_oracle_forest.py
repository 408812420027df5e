"""Pins of the random-forest oracle (Sec. 4.2, hidden constraints) against facts fixed
outside it: numpy's Philox bit generator for its random streams, a brute-force best
split from the definition of the Gini impurity with exact rationals, scikit-learn's
decision tree on data without ties, a feasibility rule recovered from noisy labels, and
invariants of the fitted trees.
"""
import math
from fractions import Fraction

import numpy as np
import pytest

from oracle import gp_forest as gf
from workloads import Param, make_workload

M64 = (1 << 64) - 1


def _numpy_block(ctr, key):
    c = list(ctr)
    for q in range(4):
        if c[q] > 0:
            c[q] -= 1
            break
        c[q] = M64
    bg = np.random.Philox(key=np.array(key, dtype=np.uint64), counter=np.array(c, dtype=np.uint64))
    return [int(v) for v in bg.random_raw(4)]


def test_streams_are_philox():
    w = gf.stream_words(77, 5, 9, 6)
    assert w[:4] == _numpy_block((5, 9, 0, 3), (77, 0))
    assert w[4:] == _numpy_block((5, 9, 1, 3), (77, 0))[:2]


def _gini_weighted(labels_left, labels_right):
    """sum over children of |child| * (1 - sum_k p_k^2), exact."""
    tot = Fraction(0)
    for part in (labels_left, labels_right):
        c = len(part)
        if c == 0:
            continue
        pk = [Fraction(sum(1 for v in part if v == k), c) for k in (0, 1)]
        tot += c * (1 - sum(p * p for p in pk))
    return tot


@pytest.mark.parametrize("seed", range(6))
def test_best_split_is_the_gini_minimum(seed):
    rng = np.random.default_rng(seed)
    n = 14
    x = rng.integers(0, 5, n).astype(np.float64)          # ties included
    lab = rng.integers(0, 2, n)
    got = gf.best_split(x, lab)
    cands = []
    for v in sorted(set(x.tolist()))[:-1]:
        g = _gini_weighted(lab[x <= v].tolist(), lab[x > v].tolist())
        cands.append((g, v))
    if not cands:
        assert got is None
        return
    g, v = min(cands)
    assert got[1] == v and 2 * got[0] == g


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_tree_matches_sklearn(seed):
    """No bootstrap, every feature at every node: the CART tree of scikit-learn (Gini,
    best splitter); continuous features, so split qualities do not tie."""
    from sklearn.tree import DecisionTreeClassifier
    rng = np.random.default_rng(seed)
    n, F = 300, 5
    X = rng.random((n, F))
    y = ((X[:, 0] + 0.5 * X[:, 1] ** 2 - 0.3 * X[:, 2] > 0.6) ^ (rng.random(n) < 0.1)).astype(np.int64)
    for depth in (3, 6, 50):
        t = gf.fit_tree(X, y, 0, 0, max_depth=depth, min_split=2, bootstrap=False, mtry=F)
        sk = DecisionTreeClassifier(criterion="gini", max_depth=depth, random_state=0).fit(X, y)
        np.testing.assert_allclose(gf.tree_predict(t, X), sk.predict_proba(X)[:, 1], rtol=0, atol=0)
        assert sum(1 for f in t.feature if f < 0) == sk.get_n_leaves()


def test_tree_invariants():
    w = make_workload("C3", 256)
    X = gf.features(w.space, w.X)
    y = np.asarray(w.feasible).astype(np.int64)
    t = gf.fit_tree(X, y, 3, 11, max_depth=8, min_split=2)
    n_nodes = len(t.feature)
    for k in range(n_nodes):
        if t.feature[k] >= 0:
            l = t.left[k]
            assert l > k and t.depth[l] == t.depth[l + 1] == t.depth[k] + 1
        assert 0.0 <= t.value[k] <= 1.0 and t.depth[k] <= 8
    kids = sorted(t.left[k] + d for k in range(n_nodes) if t.feature[k] >= 0 for d in (0, 1))
    assert kids == list(range(1, n_nodes))                # breadth-first, each node once
    # every feature at every node, no depth limit, no bootstrap: leaves are pure
    # (distinct inputs)
    t2 = gf.fit_tree(X, y, 0, 0, max_depth=10 ** 6, min_split=2, bootstrap=False,
                     mtry=X.shape[1])
    p = gf.tree_predict(t2, X)
    assert np.all((p == 0) | (p == 1)) and np.array_equal(p, y)


def test_forest_recovers_a_rule():
    """Feasible iff x0 + x1 < 1 (two reals, an unused int), 5% label noise: held-out
    accuracy of the forest's 1/2 cut well above the noise floor's complement."""
    space = [Param("a", "real", lo=0.0, hi=1.0), Param("b", "real", lo=0.0, hi=1.0),
             Param("c", "int", lo=1, hi=20)]
    rng = np.random.default_rng(4)
    def draw(n):
        cols = [rng.random(n), rng.random(n), rng.integers(1, 21, n).astype(np.int32)]
        return cols, (cols[0] + cols[1] < 1.0)
    Xc, truth = draw(600)
    feas = (truth ^ (rng.random(600) < 0.05)).astype(np.uint8)
    forest = gf.fit_forest(space, Xc, feas, n_trees=32, seed=3, max_depth=12)
    Tc, ttruth = draw(2000)
    p = gf.predict(space, forest, Tc)
    assert np.all((p >= 0) & (p <= 1))
    assert np.mean((p >= 0.5) == ttruth) > 0.93


def test_features_layout():
    space = [Param("r", "real", lo=0, hi=1), Param("p", "perm", m=3), Param("c", "cat", levels=4)]
    cols = [np.array([0.25, 0.5]), np.array([[2, 0, 1], [0, 1, 2]], np.int32), np.array([3, 1], np.int32)]
    np.testing.assert_array_equal(gf.features(space, cols),
                                  [[0.25, 2, 0, 1, 3], [0.5, 0, 1, 2, 1]])
