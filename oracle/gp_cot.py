"""CPU oracle of the Chain-of-Trees sampler and membership test (Sec. 4.2, known
constraints).

TEST INFRASTRUCTURE ONLY: imported by tests/, the smoke check and the CPU baseline of
bench.py, never by the library or its binding. Plain Python integers and numpy.

What the paper fixes: the feasible configurations of every group of co-dependent
parameters are computed beforehand and kept as a tree (one level per parameter, one
node per value, a root-to-leaf path per feasible partial configuration); parameters of
different trees are independent, so any combination of leaves is feasible; random
configurations are drawn uniformly over the leaves of each tree (not by choosing a
child uniformly at each level, which is biased); membership in the chain replaces the
evaluation of the constraints.

READINGS (the paper gives no further detail):
  * a tree is given by its parameters (its levels, in order) and its leaves, each a
    tuple of value indices (INT: value - lo, ORD: index, CAT: level); REAL and PERM
    parameters are not in trees;
  * parameters outside every tree are drawn uniformly: INT/ORD/CAT index uniform,
    REAL uniform in its declared range, PERM a uniform permutation (Fisher-Yates);
  * random words: Philox4x64-10 (Salmon, Moraes, Dror, Shaw: "Parallel random numbers:
    as easy as 1, 2, 3", SC 2011) with key (seed, 0); configuration j uses the blocks
    of counter (offset + j, b, 0, 0), b = 0, 1, ..., four words per block, in order:
    one word per tree (tree order), then per free parameter in space order one word
    (REAL, INT, ORD, CAT) or m - 1 words (PERM, used for i = m-1 .. 1);
  * an index uniform in [0, c) from a 64-bit word u is floor(u c / 2^64); a REAL is
    lo + (hi - lo) x with x = floor(u / 2^11) 2^-53 (each operation rounded once);
  * Fisher-Yates on the identity position vector: for i = m-1 .. 1, swap entries i and
    floor(u c / 2^64) with c = i + 1.

Pins: tests/test_oracle_cot.py (numpy's Philox bit generator, the paper's example
chain and configuration, brute-force membership against the constraints, closed-form
leaf count of the GPU-tile space, uniformity against the biased child-by-child draw).
"""
from __future__ import annotations

import itertools
from dataclasses import dataclass
from typing import List, Sequence

import numpy as np

M64 = (1 << 64) - 1
PHILOX_M = (0xD2E7470EE14C6C93, 0xCA5A826395121157)
PHILOX_W = (0x9E3779B97F4A7C15, 0xBB67AE8584CAA73B)


def philox4x64(ctr: Sequence[int], key: Sequence[int], rounds: int = 10) -> List[int]:
    """Philox4x64 block: each round multiplies words 0 and 2 by the two constants, and
    mixes the high halves with words 1 and 3 and the round key; the key is bumped by
    the two Weyl constants between rounds."""
    x = [int(v) & M64 for v in ctr]
    k0, k1 = int(key[0]) & M64, int(key[1]) & M64
    for r in range(rounds):
        if r:
            k0 = (k0 + PHILOX_W[0]) & M64
            k1 = (k1 + PHILOX_W[1]) & M64
        p0, p1 = PHILOX_M[0] * x[0], PHILOX_M[1] * x[2]
        x = [(p1 >> 64) ^ x[1] ^ k0, p1 & M64, (p0 >> 64) ^ x[3] ^ k1, p0 & M64]
    return x


def words(seed: int, j: int, count: int) -> List[int]:
    """The first `count` random words of configuration j (counter (j, b, 0, 0))."""
    out = []
    b = 0
    while len(out) < count:
        out += philox4x64((j, b, 0, 0), (seed, 0))
        b += 1
    return out[:count]


def uniform_index(u: int, c: int) -> int:
    return (u * c) >> 64


def unit_double(u: int) -> float:
    return float(u >> 11) * 2.0 ** -53


# ===================================================================== the chain
def value_count(p) -> int:
    if p.kind == "int":
        return int(p.hi) - int(p.lo) + 1
    if p.kind == "ord":
        return len(p.values)
    if p.kind == "cat":
        return p.levels
    raise ValueError(f"{p.kind} parameters are not in trees")


def raw_value(p, idx: int) -> int:
    """Raw column entry of value index idx (INT: the value, ORD/CAT: the index)."""
    return int(p.lo) + idx if p.kind == "int" else idx


def value_index(p, raw: int) -> int:
    return raw - int(p.lo) if p.kind == "int" else raw


@dataclass
class Chain:
    space: list
    trees: List[List[int]]          # parameter indices per tree, level order
    leaves: List[np.ndarray]        # per tree: [n_leaves, k] value indices, lexicographic


def chain_from_predicates(space, trees, predicates) -> Chain:
    """Leaves of each tree by brute force over the product of its parameters' values:
    predicates[t] takes the tuple of *raw* values (INT value, ORD value, CAT level) of
    tree t's parameters and says whether the partial configuration is feasible."""
    leaves = []
    for tree, pred in zip(trees, predicates):
        ranges = [range(value_count(space[p])) for p in tree]
        lv = []
        for idx in itertools.product(*ranges):           # lexicographic
            vals = tuple(space[p].values[i] if space[p].kind == "ord" else raw_value(space[p], i)
                         for p, i in zip(tree, idx))
            if pred(vals):
                lv.append(tuple(idx))
        leaves.append(np.array(lv, dtype=np.int64).reshape(-1, len(tree)))
    return Chain(space, [list(t) for t in trees], leaves)


def words_per_config(chain: Chain) -> int:
    in_tree = {p for t in chain.trees for p in t}
    w = len(chain.trees)
    for i, p in enumerate(chain.space):
        if i in in_tree:
            continue
        w += p.m - 1 if p.kind == "perm" else 1
    return w


def sample(chain: Chain, M: int, seed: int, offset: int = 0) -> list:
    """M configurations as raw columns (the formats of `workloads`)."""
    space = chain.space
    in_tree = {p for t in chain.trees for p in t}
    cols = []
    for p in space:
        if p.kind == "real":
            cols.append(np.zeros(M, np.float64))
        elif p.kind == "perm":
            cols.append(np.zeros((M, p.m), np.int32))
        else:
            cols.append(np.zeros(M, np.int32))
    W = words_per_config(chain)
    for j in range(M):
        u = words(seed, offset + j, W)
        q = 0
        for tree, lv in zip(chain.trees, chain.leaves):
            leaf = lv[uniform_index(u[q], len(lv))]
            q += 1
            for p, idx in zip(tree, leaf):
                cols[p][j] = raw_value(space[p], idx)
        for i, p in enumerate(space):
            if i in in_tree:
                continue
            if p.kind == "real":
                x = unit_double(u[q])
                cols[i][j] = float(p.lo) + (float(p.hi) - float(p.lo)) * x
                q += 1
            elif p.kind == "perm":
                pi = list(range(p.m))
                for k in range(p.m - 1, 0, -1):
                    r = uniform_index(u[q], k + 1)
                    q += 1
                    pi[k], pi[r] = pi[r], pi[k]
                cols[i][j] = pi
            else:
                cols[i][j] = raw_value(p, uniform_index(u[q], value_count(p)))
                q += 1
    return cols


def member(chain: Chain, cols) -> np.ndarray:
    """1 where every tree's partial configuration of the row is one of its leaves (row
    membership through numpy's flat index of the value-index tuple and isin; a value
    outside its parameter's range is not a member)."""
    space = chain.space
    M = len(np.asarray(cols[0]))
    ok = np.ones(M, bool)
    for tree, lv in zip(chain.trees, chain.leaves):
        dims = [value_count(space[p]) for p in tree]
        idx = [np.asarray(value_index(space[p], np.asarray(cols[p]).astype(np.int64)))
               for p in tree]
        inr = np.ones(M, bool)
        for a, c in zip(idx, dims):
            inr &= (a >= 0) & (a < c)
        flat = np.ravel_multi_index([np.where(inr, a, 0) for a in idx], dims)
        leaf_flat = np.ravel_multi_index([lv[:, q] for q in range(len(tree))], dims)
        ok &= inr & np.isin(flat, leaf_flat)
    return ok.astype(np.uint8)
