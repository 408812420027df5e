"""GPU parity of the random-forest feasibility model (Sec. 4.2, hidden constraints)
against the oracle. Both sides take every random choice from the same counter-based
streams and compare split qualities exactly, so the trees must be identical node for
node (features, children, thresholds and leaf values bit for bit) and the predicted
probabilities identical after the fp32 rounding of the fp64 mean.
"""
import numpy as np
import pytest

from oracle import gp_forest as gf
from workloads import Param, make_workload

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _announce(request):
    print(f"\n[gpu] {request.node.nodeid}", flush=True)
    yield


def _gp():
    from paper_2212_11142_amd import gp
    return gp


def _dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _oracle_arrays(tree):
    feat = np.array(tree.feature, np.int32)
    left = np.array(tree.left, np.int32)
    val = np.array([th if f >= 0 else v for f, th, v in zip(tree.feature, tree.threshold, tree.value)])
    return feat, left, val


def _fit_both(name, n=None, T=8, depth=12, seed=5, feasible=None):
    gp = _gp()
    w = make_workload(name, 4096)
    X = [c[:n] for c in w.X] if n else w.X
    feas = (w.feasible[:n] if n else w.feasible) if feasible is None else feasible
    space = gp.Space(w.space)
    f = gp.Forest(space, gp.to_device_columns(space, X), _dev(np.asarray(feas, np.uint8)), T,
                  depth, 2, seed)
    ref = gf.fit_forest(w.space, X, feas, T, seed, depth, 2)
    return w, space, f, ref


@pytest.mark.parametrize("name,n,T", [("C1", None, 8), ("C2", None, 8), ("C3", None, 16),
                                      ("C4", None, 8), ("C5", 700, 4)])
def test_trees_identical(name, n, T):
    w, space, f, ref = _fit_both(name, n, T)
    nodes = 0
    for t in range(T):
        feat, left, val = f.tree(t)
        rf, rl, rv = _oracle_arrays(ref[t])
        assert np.array_equal(feat, rf), f"{name} tree {t}: features"
        assert np.array_equal(left, rl), f"{name} tree {t}: children"
        assert np.array_equal(val, rv), f"{name} tree {t}: values {np.nonzero(val != rv)[0][:5]}"
        nodes += len(feat)
    print(f"{name}: {T} trees, {nodes} nodes identical")


@pytest.mark.parametrize("name,n", [("C2", None), ("C5", 600)])
def test_trees_identical_permutation_and_real_features(name, n):
    """C2 and C5 are all feasible: labels from a rule on a permutation position, an
    ordinal and (C5) a real, with noise, so that their features get split on."""
    gp = _gp()
    w = make_workload(name, 4096)
    X = [c[:n] for c in w.X] if n else w.X
    Xf = gf.features(w.space, X)
    rng = np.random.default_rng(8)
    score = Xf[:, -1] + 0.5 * Xf[:, 0] + (Xf[:, 7] * 3 if name == "C5" else 0)
    feas = ((score > np.median(score)) ^ (rng.random(len(score)) < 0.1)).astype(np.uint8)
    space = gp.Space(w.space)
    f = gp.Forest(space, gp.to_device_columns(space, X), _dev(feas), 8, 12, 2, 3)
    ref = gf.fit_forest(w.space, X, feas, 8, 3, 12, 2)
    used = set()
    for t in range(8):
        feat, left, val = f.tree(t)
        rf, rl, rv = _oracle_arrays(ref[t])
        assert np.array_equal(feat, rf) and np.array_equal(left, rl) and np.array_equal(val, rv)
        used |= set(feat[feat >= 0].tolist())
    kinds = [p.kind for p in w.space for _ in range(p.m if p.kind == "perm" else 1)]
    assert any(kinds[f] == "perm" for f in used), used
    assert name != "C5" or any(kinds[f] == "real" for f in used), used


@pytest.mark.parametrize("name", ["C3", "C4"])
def test_predict_identical(name):
    gp = _gp()
    w, space, f, ref = _fit_both(name, None, 16)
    C = [c[:4096] for c in w.C]
    rng = np.random.default_rng(1)
    ei = rng.random(4096).astype(np.float32)
    mask = (rng.random(4096) < 0.8).astype(np.uint8)
    p, acq = f.predict(gp.to_device_columns(space, C), _dev(ei), _dev(mask), 0.3)
    pr = gf.predict(w.space, ref, C).astype(np.float32)
    p = p.cpu().numpy()
    assert np.array_equal(p, pr), f"{name}: {np.nonzero(p != pr)[0][:5]}"
    want = np.where((mask != 0) & (pr >= np.float32(0.3)), ei * pr, np.float32(0.0))
    assert np.array_equal(acq.cpu().numpy(), want)
    assert 0.0 < pr.mean() < 1.0


def test_predict_full_size_sampled():
    """A million candidates of C4: rows checked one by one against the oracle."""
    gp = _gp()
    w = make_workload("C4")
    space = gp.Space(w.space)
    f = gp.Forest(space, gp.to_device_columns(space, w.X), _dev(w.feasible), 32, 16, 2, 9)
    ref = gf.fit_forest(w.space, w.X, w.feasible, 32, 9, 16, 2)
    p, _ = f.predict(gp.to_device_columns(space, w.C))
    p = p.cpu().numpy()
    rows = np.array([0, 1, 777, 65536, 500001, len(p) - 1])
    pr = gf.predict(w.space, ref, [c[rows] for c in w.C]).astype(np.float32)
    assert np.array_equal(p[rows], pr)
    assert np.all((p >= 0) & (p <= 1))


def test_forest_edges():
    gp = _gp()
    w = make_workload("C2", 256)
    space = gp.Space(w.space)
    X = gp.to_device_columns(space, w.X)
    # depth 0: each tree is its bootstrap sample's feasible fraction
    f0 = gp.Forest(space, X, _dev(w.feasible), 4, 0, 2, 1)
    r0 = gf.fit_forest(w.space, w.X, w.feasible, 4, 1, 0, 2)
    for t in range(4):
        feat, left, val = f0.tree(t)
        assert len(feat) == 1 and feat[0] == -1 and val[0] == r0[t].value[0]
    # all feasible: probability 1 everywhere
    ones = np.ones(len(w.feasible), np.uint8)
    f1 = gp.Forest(space, X, _dev(ones), 4, 8, 2, 1)
    p, _ = f1.predict(gp.to_device_columns(space, [c[:100] for c in w.C]))
    assert np.all(p.cpu().numpy() == 1.0)
    # a single observation
    X1 = gp.to_device_columns(space, [c[:1] for c in w.X])
    fs = gp.Forest(space, X1, _dev(w.feasible[:1]), 2, 8, 2, 1)
    assert fs.tree(0)[0].tolist() == [-1]
    # rejected: too many features, an invalid observation
    big = gp.Space([Param(f"p{k}", "perm", m=8) for k in range(16)])
    with pytest.raises(gp.GPError):
        gp.Forest(big, [_dev(np.zeros((4, 8), np.int32))] * 16, _dev(np.ones(4, np.uint8)), 2)
    bad = [c.copy() for c in w.X]
    bad[3][5] = 1000                                  # an int beyond its declared range
    with pytest.raises(gp.GPError, match="observation 5"):
        gp.Forest(space, gp.to_device_columns(space, bad), _dev(w.feasible), 2)
