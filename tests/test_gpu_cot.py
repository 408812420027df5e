"""GPU parity of the Chain-of-Trees sampler and membership test (Sec. 4.2, known
constraints) against the oracle: both draw from the same counter-based generator, so
sampled configurations must be identical bit for bit (REAL values included), and
membership masks identical.
"""
import numpy as np
import pytest

from oracle import gp_cot as gc
from workloads import (Param, c3_chain_leaves, cot_example_constraints, cot_example_space,
                       make_workload)

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


def _same_cols(got, ref, label):
    for p, (g, r) in enumerate(zip(got, ref)):
        g = g.cpu().numpy()
        assert g.dtype == r.dtype and g.shape == r.shape, (label, p, g.dtype, r.dtype)
        assert np.array_equal(g, r), f"{label}: column {p} differs at {np.nonzero(g != r)[0][:5]}"


def _example():
    space = cot_example_space()
    ch = gc.chain_from_predicates(space, [[0, 1], [2, 3, 4]],
                                  [lambda v: v[0] >= v[1],
                                   lambda v: v[1] >= v[0] and v[2] >= 2 * v[1]])
    return space, ch


def test_example_sample_and_member():
    gp = _gp()
    space, ch = _example()
    dc = gp.Chain(gp.Space(space), ch.trees, ch.leaves)
    cols = dc.sample(5000, seed=5)
    _same_cols(cols, gc.sample(ch, 5000, seed=5), "example sample")
    assert dc.member(cols).cpu().numpy().all()
    # every point of the dense grid: membership equals the constraints
    import itertools
    grid = list(itertools.product(*[range(len(p.values)) for p in space]))
    gcols = [np.array([g[p] for g in grid], np.int32) for p in range(5)]
    vals = [np.array([space[p].values[g[p]] for g in grid]) for p in range(5)]
    got = dc.member([_dev(c) for c in gcols]).cpu().numpy()
    np.testing.assert_array_equal(got, cot_example_constraints(vals).astype(np.uint8))
    np.testing.assert_array_equal(got, gc.member(ch, gcols))


def test_free_parameters_bit_exact():
    gp = _gp()
    space = [Param("a", "int", lo=-3, hi=9), Param("r", "real", lo=-2.5, hi=5.0),
             Param("p", "perm", m=7), Param("o", "ord", values=(1, 2, 4)),
             Param("c", "cat", levels=3), Param("q", "perm", m=2),
             Param("s", "real", lo=1e-3, hi=1e3), Param("i", "int", lo=1, hi=64)]
    ch = gc.chain_from_predicates(space, [[3, 4], [7]],
                                  [lambda v: v[0] != 4 or v[1] != 0, lambda v: v[0] % 3 != 0])
    dc = gp.Chain(gp.Space(space), ch.trees, ch.leaves)
    for seed, off, M in [(11, 0, 3000), (2 ** 63 + 5, 123456789, 777)]:
        cols = dc.sample(M, seed=seed, offset=off)
        _same_cols(cols, gc.sample(ch, M, seed=seed, offset=off), f"free seed={seed}")
        assert dc.member(cols).cpu().numpy().all()
    # consecutive offsets concatenate
    a = dc.sample(500, seed=9, offset=0)
    b = dc.sample(700, seed=9, offset=500)
    c = dc.sample(1200, seed=9, offset=0)
    for x, y, z in zip(a, b, c):
        assert np.array_equal(np.concatenate([x.cpu().numpy(), y.cpu().numpy()]), z.cpu().numpy())


def _c3_chain(gp):
    w = make_workload("C3", 65536)
    Lv = c3_chain_leaves()
    ch = gc.Chain(w.space, [list(range(10))], [Lv.astype(np.int64)])
    return w, ch, gp.Chain(gp.Space(w.space), ch.trees, [Lv.astype(np.int32)])


def test_c3_sample_and_member():
    """The GPU-tile space (one tree of ten parameters, 9,339,902 leaves)."""
    gp = _gp()
    w, ch, dc = _c3_chain(gp)
    cols = dc.sample(4096, seed=3, offset=1000)
    _same_cols(cols, gc.sample(ch, 4096, seed=3, offset=1000), "C3 sample")
    got = dc.member([_dev(c) for c in w.C]).cpu().numpy()
    np.testing.assert_array_equal(got, w.mask)
    np.testing.assert_array_equal(got, gc.member(ch, w.C))
    # full size: a million draws, all feasible; rows checked one by one
    M = 1 << 20
    big = dc.sample(M, seed=77)
    assert dc.member(big).cpu().numpy().all()
    host = [c.cpu().numpy() for c in big]
    for j in (0, 1, 4095, 65537, 500000, M - 1):
        one = gc.sample(ch, 1, seed=77, offset=j)
        assert all(h[j] == o[0] for h, o in zip(host, one)), j
    # leaf frequencies: each leaf has probability 1/9339902; the counts of the first
    # tree level (G0 = level g) must follow the number of leaves under it
    Lv = ch.leaves[0]
    expect = np.bincount(Lv[:, 0], minlength=11) / len(Lv)
    seen = np.bincount(host[0], minlength=11) / M
    assert np.abs(seen - expect).max() < 5e-3


def test_member_out_of_range_and_edges():
    gp = _gp()
    space, ch = _example()
    dc = gp.Chain(gp.Space(space), ch.trees, ch.leaves)
    cols = [np.array([0, 1, 2, -1], np.int32), np.zeros(4, np.int32), np.zeros(4, np.int32),
            np.array([2, 2, 2, 2], np.int32), np.array([2, 2, 2, 2], np.int32)]
    got = dc.member([_dev(c) for c in cols]).cpu().numpy()
    np.testing.assert_array_equal(got, gc.member(ch, cols))
    assert got[2] == 0 and got[3] == 0
    assert dc.sample(0, seed=1)[0].shape[0] == 0


def test_chain_rejected():
    gp = _gp()
    space, ch = _example()
    sp = gp.Space(space)
    bad = ch.leaves[1].copy()
    bad[[2, 3]] = bad[[3, 2]]                          # out of lexicographic order
    with pytest.raises(gp.GPError, match="tree 1, leaf 3"):
        gp.Chain(sp, ch.trees, [ch.leaves[0], bad])
    oor = ch.leaves[0].copy()
    oor[1, 1] = 2                                      # value index out of range
    with pytest.raises(gp.GPError, match="tree 0, leaf 1"):
        gp.Chain(sp, ch.trees, [oor, ch.leaves[1]])
    with pytest.raises(gp.GPError):
        gp.Chain(sp, [[0, 1], [1, 2]], ch.leaves)      # a parameter in two trees
    rs = gp.Space([Param("r", "real", lo=0.0, hi=1.0)])
    with pytest.raises(gp.GPError):
        gp.Chain(rs, [[0]], [np.zeros((1, 1), np.int32)])
