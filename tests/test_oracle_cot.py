"""Pins of the Chain-of-Trees oracle (Sec. 4.2, known constraints) against facts fixed
outside it: numpy's Philox4x64-10 bit generator, the leaves drawn in the paper's figure
and the configuration its text names, brute-force evaluation of the constraints, the
closed-form size of the GPU-tile space's feasible set, and the uniformity of the leaf
draw (against the biased child-by-child draw the paper rejects).
"""
import itertools
import json
import math
import os

import numpy as np
import pytest
from scipy import stats

from oracle import gp_cot as gc
from workloads import (Param, c3_chain_leaves, c3_known_feasible, cot_example_constraints,
                       cot_example_space, make_workload)

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
M64 = (1 << 64) - 1


def _numpy_block(ctr, key):
    """numpy's Philox increments its 256-bit counter before each block: start one below."""
    c = list(ctr)
    for q in range(4):          # subtract 1 with borrow
        if c[q] > 0:
            c[q] -= 1
            break
        c[q] = M64
    bg = np.random.Philox(key=np.array(key, dtype=np.uint64), counter=np.array(c, dtype=np.uint64))
    return [int(v) for v in bg.random_raw(4)]


@pytest.mark.parametrize("ctr,key", [((0, 0, 0, 0), (0, 0)), ((1, 0, 0, 0), (7, 0)),
                                     ((12345, 3, 0, 0), (2024, 0)),
                                     ((M64, M64, 5, 9), (M64, M64)),
                                     ((0, 0, 0, 1), (0xDEADBEEF, 0x12345678))])
def test_philox_matches_numpy(ctr, key):
    assert gc.philox4x64(ctr, key) == _numpy_block(ctr, key)


def test_word_layout():
    w = gc.words(99, 17, 6)
    assert w[:4] == gc.philox4x64((17, 0, 0, 0), (99, 0))
    assert w[4:] == gc.philox4x64((17, 1, 0, 0), (99, 0))[:2]


def test_uniform_index_and_unit_double():
    for k in range(1, 10):
        c = 1 << k
        for u in (0, 1, 12345678901234567, M64):
            assert gc.uniform_index(u, c) == u >> (64 - k)
    assert gc.uniform_index(M64, 7) == 6 and gc.uniform_index(0, 7) == 0
    assert gc.unit_double(0) == 0.0 and gc.unit_double(M64) == 1.0 - 2.0 ** -53


def _example_chain():
    space = cot_example_space()
    trees = [[0, 1], [2, 3, 4]]
    preds = [lambda v: v[0] >= v[1], lambda v: v[1] >= v[0] and v[2] >= 2 * v[1]]
    return space, gc.chain_from_predicates(space, trees, preds)


def test_example_chain_is_the_figure():
    space, ch = _example_chain()
    g = json.load(open(os.path.join(GOLDEN, "cot_example_leaves.json")))
    for t, key in enumerate(("tree1", "tree2")):
        vals = [[space[p].values[i] for p, i in zip(ch.trees[t], row)] for row in ch.leaves[t]]
        assert vals == g[key]
    # the configuration the text names is in the chain; so is every product of leaves
    named = json.load(open(os.path.join(GOLDEN, "cot_example.json")))["feasible_example"]
    cols = [np.array([space[p].values.index(v)]) for p, v in enumerate(named)]
    assert gc.member(ch, cols)[0] == 1


def test_membership_equals_the_constraints():
    """Every point of the dense grid: member of the chain iff the constraints hold."""
    space, ch = _example_chain()
    grid = list(itertools.product(*[range(len(p.values)) for p in space]))
    cols = [np.array([g[p] for g in grid]) for p in range(5)]
    vals = [np.array([space[p].values[g[p]] for g in grid]) for p in range(5)]
    np.testing.assert_array_equal(gc.member(ch, cols), cot_example_constraints(vals))
    bad = [c.copy() for c in cols]
    bad[4][0] = 3                                       # out of range: not a member
    assert gc.member(ch, bad)[0] == 0


def _chi2_p(counts):
    return stats.chisquare(counts).pvalue


def test_leaf_draw_is_uniform_and_child_draw_is_not():
    """Uniform over the 21 feasible configurations; the child-by-child draw (uniform
    child at each level) gives the right tree's lone p3 = 4 path half of the mass."""
    space, ch = _example_chain()
    N = 21000
    cols = gc.sample(ch, N, seed=5)
    assert gc.member(ch, cols).all()
    keys = list(zip(*[c.tolist() for c in cols]))
    feasible = [g for g in itertools.product(*[range(len(p.values)) for p in space])
                if gc.member(ch, [np.array([v]) for v in g])[0]]
    counts = np.array([keys.count(g) for g in feasible])
    assert len(feasible) == 21 and counts.sum() == N
    assert _chi2_p(counts) > 1e-4
    # child-by-child draw on the right tree, with the same random words
    rng = np.random.default_rng(0)
    right = ch.leaves[1]
    picks = []
    for _ in range(7000):
        rows = right
        for lvl in range(3):
            kids = sorted(set(rows[:, lvl].tolist()))
            v = kids[rng.integers(len(kids))]
            rows = rows[rows[:, lvl] == v]
        picks.append(tuple(rows[0].tolist()))
    cnt = np.array([picks.count(tuple(r)) for r in right.tolist()])
    assert _chi2_p(cnt) < 1e-10
    assert abs(cnt[-1] / 7000 - 0.5) < 0.03               # (4, 4, 8) alone under p3 = 4


def test_free_parameters():
    """Parameters outside every tree: INT/ORD/CAT uniform, REAL in its range, PERM a
    uniform permutation."""
    space = [Param("a", "int", lo=3, hi=9), Param("r", "real", lo=-2.0, hi=5.0),
             Param("p", "perm", m=3), Param("o", "ord", values=(1, 2, 4)),
             Param("c", "cat", levels=3)]
    ch = gc.chain_from_predicates(space, [[3, 4]], [lambda v: v[0] != 4 or v[1] != 0])
    N = 6000
    cols = gc.sample(ch, N, seed=11)
    assert cols[0].min() == 3 and cols[0].max() == 9
    assert cols[1].min() >= -2.0 and cols[1].max() < 5.0
    perms = [tuple(r) for r in cols[2].tolist()]
    assert all(sorted(p) == [0, 1, 2] for p in perms)
    pc = np.array([perms.count(p) for p in itertools.permutations(range(3))])
    assert _chi2_p(pc) > 1e-4
    assert _chi2_p(np.bincount(cols[0] - 3, minlength=7)) > 1e-4
    assert gc.member(ch, cols).all()
    assert not np.any((cols[3] == 2) & (cols[4] == 0))


def test_c3_chain():
    """The GPU-tile space: its leaf count equals the closed-form count of the
    constraints, every leaf is feasible, the leaves are strictly lexicographic, and chain
    membership of the workload's candidates equals the constraint mask."""
    Lv = c3_chain_leaves()
    f = lambda l: (l + 1) * (11 - l)
    f0 = lambda l: (l + 1) * (l + 2) // 2 * (11 - l)
    closed = sum(f0(a) * f(b) * f(c) for a in range(11) for b in range(11) for c in range(11)
                 if a + b + c <= 10)
    assert len(Lv) == closed == 9339902
    assert c3_known_feasible([Lv[:, q] for q in range(10)]).all()
    flat = np.ravel_multi_index([Lv[:, q].astype(np.int64) for q in range(10)], [11] * 10)
    assert np.all(np.diff(flat) > 0)
    w = make_workload("C3", 20000)
    ch = gc.Chain(w.space, [list(range(10))], [Lv.astype(np.int64)])
    np.testing.assert_array_equal(gc.member(ch, w.C), w.mask)
    assert 0 < w.mask.sum() < len(w.mask)
