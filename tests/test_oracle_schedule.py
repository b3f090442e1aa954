"""Pins of the oracle's schedule and validator (CPU only).

The oracle's level assignment is computed two independent ways -- the
recursive height and peeling ready vertices off the graph (the activation
rule of Section 3.2, Algorithm 1) -- and both are checked against closed forms for the shapes of Section 5 (complete
binary trees with 256 leaves have 511 vertices; chains; left-branching trees).
"""
import json
import os

import numpy as np
import pytest

import oracle
from paper_1712_04048_amd import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _forest(seed, N=2, shuffle=False):
    rng = np.random.Generator(np.random.PCG64(seed))
    trees = []
    for _ in range(int(rng.integers(1, 7))):
        kind = int(rng.integers(0, 4))
        L = int(rng.integers(1, 12))
        if N == 1:
            trees.append(W.chain(L))
        elif kind == 0:
            trees.append(W.random_split_tree(L, rng))
        elif kind == 1:
            trees.append(W.left_branching_tree(L))
        elif kind == 2:
            trees.append(W.right_branching_tree(L))
        else:
            trees.append(W.complete_tree(1 << int(rng.integers(0, 4))))
    child, parent, _, _ = W.assemble(trees, N, rng, shuffle_ids=shuffle)
    return child, parent


@pytest.mark.parametrize("seed", range(40))
def test_recursive_levels_equal_algorithm1(seed):
    N = 1 if seed % 5 == 0 else 2
    child, parent = _forest(seed, N=N, shuffle=seed % 2 == 1)
    assert oracle.validate(child, parent) == oracle.OK
    T1, l1 = oracle.levels(child, "recursive")
    T2, l2 = oracle.levels(child, "frontier")
    assert T1 == T2
    assert np.array_equal(l1, l2)


def test_brute_force_levels_tiny():
    """Every forest on up to 5 vertices with 1..2 child slots: the level is the
    longest downward path, found here by enumerating paths."""
    rng = np.random.Generator(np.random.PCG64(7))
    for _ in range(300):
        V = int(rng.integers(1, 6))
        # random parent function that is a forest: parent id > child id
        parent = np.full(V, -1, dtype=np.int32)
        slots = {}
        for v in range(V - 1):
            if rng.random() < 0.8:
                p = int(rng.integers(v + 1, V))
                if slots.get(p, 0) < 2:
                    slots[p] = slots.get(p, 0) + 1
                    parent[v] = p
        child = np.full((V, 2), -1, dtype=np.int32)
        fill = {}
        for v in range(V):
            if parent[v] >= 0:
                p = parent[v]
                child[p, fill.get(p, 0)] = v
                fill[p] = fill.get(p, 0) + 1
        # brute force: longest path down, by enumerating all descending walks
        def longest(v):
            best = 0
            stack = [(v, 0)]
            while stack:
                u, d = stack.pop()
                best = max(best, d)
                for c in child[u]:
                    if c >= 0:
                        stack.append((c, d + 1))
            return best
        want = np.array([longest(v) for v in range(V)], dtype=np.int32)
        T, lev = oracle.levels(child, "frontier")
        assert np.array_equal(lev, want)
        assert T == want.max() + 1


def test_complete_tree_closed_form():
    with open(os.path.join(GOLDEN, "complete_tree_256.json")) as f:
        g = json.load(f)
    K = 3
    trees = [W.complete_tree(g["leaves"]) for _ in range(K)]
    rng = np.random.Generator(np.random.PCG64(0))
    child, parent, _, _ = W.assemble(trees, 2, rng)
    assert child.shape[0] == K * g["vertices_per_tree"]
    s = oracle.schedule(child, parent)
    assert s["T"] == g["levels"]
    sizes = np.diff(s["level_offsets"])
    assert list(sizes) == [K * g["leaves"] >> t for t in range(g["levels"])]


def test_chain_and_left_branching_closed_forms():
    rng = np.random.Generator(np.random.PCG64(0))
    lengths = [3, 7, 1, 5]
    child, parent, _, _ = W.assemble([W.chain(n) for n in lengths], 1, rng)
    s = oracle.schedule(child, parent)
    assert s["T"] == max(lengths)
    assert list(np.diff(s["level_offsets"])) == [sum(n > t for n in lengths) for t in range(max(lengths))]
    leaves = [2, 6, 4]
    child, parent, _, _ = W.assemble([W.left_branching_tree(L) for L in leaves], 2, rng)
    s = oracle.schedule(child, parent)
    assert s["T"] == max(leaves)
    want = [sum(leaves)] + [sum(L > t for L in leaves) for t in range(1, max(leaves))]
    assert list(np.diff(s["level_offsets"])) == want


@pytest.mark.parametrize("seed", range(10))
def test_layout_invariants(seed):
    child, parent = _forest(100 + seed, shuffle=True)
    V = parent.shape[0]
    pull = np.where(np.all(child < 0, axis=1), 0, -1).astype(np.int32)
    pull[pull >= 0] = np.arange((pull >= 0).sum())
    s = oracle.schedule(child, parent, pull_idx=pull, push_idx=None)
    order, pos, lev = s["order"], s["pos"], s["level"]
    assert sorted(order) == list(range(V))
    assert np.array_equal(pos[order], np.arange(V))
    keys = [(lev[v], v) for v in order]
    assert keys == sorted(keys)
    for p in range(V):
        v = order[p]
        for k in range(child.shape[1]):
            c = child[v, k]
            assert s["child_pos"][p, k] == (pos[c] if c >= 0 else -1)
            if c >= 0:
                assert s["child_pos"][p, k] < s["level_offsets"][lev[v]]
        assert s["parent_pos"][p] == (pos[parent[v]] if parent[v] >= 0 else -1)
        assert s["pull_pos"][p] == pull[v]
    assert list(s["pull_list"]) == [p for p in range(V) if s["pull_pos"][p] >= 0]


def _tree3():
    # 0, 1 leaves; 2 = (0, 1) root
    child = np.array([[-1, -1], [-1, -1], [0, 1]], dtype=np.int32)
    parent = np.array([2, 2, -1], dtype=np.int32)
    return child, parent


def test_validate_negative_cases():
    child, parent = _tree3()
    assert oracle.validate(child, parent) == oracle.OK
    c = child.copy(); c[2, 1] = 3
    assert oracle.validate(c, parent) == oracle.ERR_RANGE
    p = parent.copy(); p[0] = -2
    assert oracle.validate(child, p) == oracle.ERR_RANGE
    c = child.copy(); c[2, 1] = 0                       # duplicate child
    assert oracle.validate(c, parent) == oracle.ERR_MULTIPARENT
    c = np.array([[-1, -1], [0, -1], [0, 1]], dtype=np.int32)   # 0 has two parents
    assert oracle.validate(c, np.array([1, 2, -1], dtype=np.int32)) == oracle.ERR_MULTIPARENT
    p = parent.copy(); p[1] = -1                        # parent array disagrees
    assert oracle.validate(child, p) == oracle.ERR_MISMATCH
    p = parent.copy(); p[2] = 0                         # extra parent pointer
    assert oracle.validate(child, p) == oracle.ERR_MISMATCH
    # 2-cycle: 3 <-> 4 plus the valid tree
    c = np.array([[-1, -1], [-1, -1], [0, 1], [4, -1], [3, -1]], dtype=np.int32)
    p = np.array([2, 2, -1, 4, 3], dtype=np.int32)
    assert oracle.validate(c, p) == oracle.ERR_CYCLE
    c = np.array([[0, -1]], dtype=np.int32)             # self loop
    assert oracle.validate(c, np.array([0], dtype=np.int32)) == oracle.ERR_CYCLE
    pull = np.array([0, 0, -1], dtype=np.int32)
    assert oracle.validate(child, parent, pull, 2) == oracle.ERR_DUP_PULL
    assert oracle.validate(child, parent, np.array([0, 2, -1], np.int32), 2) == oracle.ERR_RANGE
    assert oracle.validate(child, parent, None, 0, np.array([0, 5, -1], np.int32), 5) == oracle.ERR_RANGE
    # priority: range beats everything else
    c = np.array([[-1, -1], [0, 7], [0, 1]], dtype=np.int32)
    assert oracle.validate(c, parent) == oracle.ERR_RANGE
