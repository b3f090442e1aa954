"""Pins of the oracle on graph inputs and wider child-sum vertices (CPU).

Graph-structured cells (Section 2, panel (d) of the recurrent-structures
figure) let a vertex's state be read by several vertices.  Reverse-mode
differentiation then sums what each reader sends back, which is exactly what
the tree obtained by copying every shared vertex once per reader computes,
with tied copies: its states equal the graph's bit for bit, its parameter
gradients equal the graph's up to summation order, and the gradient of a
shared input row is the sum over the copies' rows.  That unfolding is built
here from the graph alone and run through the oracle's tree path.  The
child-sum cell of Section 3.1 is written for any number of child slots N;
N = 3 and 4 and the graph inputs are also checked against central finite
differences over every parameter and input element.
"""
import itertools

import numpy as np
import pytest

import oracle
from paper_1712_04048_amd import workloads as W
from test_oracle_numerics import _fd_check


def _dag_workload(seed, N=2, n=12, cell=W.CELL_TREE_LSTM, inputs="all", labels="root",
                  H=5, D=4):
    rng = np.random.Generator(np.random.PCG64(seed))
    graphs = [W.random_dag(int(rng.integers(3, n)), N, rng) for _ in range(3)]
    kw = dict(cell=cell, N=N, H=H, C=3, sigma=0.5, rng=rng, labels=labels, dag=True)
    if cell == W.CELL_TREE_LSTM:
        kw.update(D=D, inputs=inputs)
    else:
        kw.update(loss=W.LOSS_L2)
    wl = W.make_workload("dag%d" % seed, graphs, **kw)
    wl.b[:] = (0.3 * rng.standard_normal(wl.b.shape)).astype(np.float32)
    return wl


def _unfold(wl):
    """Tree unfolding of a graph workload: every vertex copied once per path
    from a root; copies pull their own X row holding the original's values;
    only roots are labelled."""
    V, N = wl.V, wl.N
    read = W.read_by_someone(wl.child)
    child, orig = [], []

    def emit(v):
        kids = [emit(int(c)) if c >= 0 else -1 for c in wl.child[v]]
        child.append(kids)
        orig.append(v)
        return len(child) - 1

    roots = [v for v in range(V) if not read[v]]
    for r in roots:
        emit(r)
    child = np.array(child, dtype=np.int32).reshape(-1, N)
    orig = np.array(orig)
    parent = np.full(len(orig), -1, dtype=np.int32)
    for v, ks in enumerate(child):
        for c in ks:
            if c >= 0:
                parent[c] = v
    pulls = wl.pull_idx[orig]
    pull_idx = np.full(len(orig), -1, dtype=np.int32)
    has = np.nonzero(pulls >= 0)[0]
    pull_idx[has] = np.arange(has.size)
    X = wl.X[pulls[has]]
    push_idx = np.full(len(orig), -1, dtype=np.int32)
    is_root = parent < 0
    push_idx[is_root] = wl.push_idx[orig[is_root]]
    Y = wl.Y
    tw = W.Workload(name="unfolded", cell=wl.cell, prec=wl.prec, loss=wl.loss, N=N, D=wl.D,
                    H=wl.H, C=wl.C, child=child, parent=parent, pull_idx=pull_idx,
                    push_idx=push_idx, X=X, Y=Y, Wx=wl.Wx, U=wl.U, b=wl.b, Ws=wl.Ws, bs=wl.bs,
                    tree_offsets=np.array([0, len(orig)]))
    return tw, orig, pulls


@pytest.mark.parametrize("seed,N,cell", [(0, 2, 0), (1, 2, 0), (2, 3, 0), (3, 1, 0),
                                         (4, 2, 1), (5, 4, 0)])
def test_dag_equals_tree_unfolding(seed, N, cell):
    wl = _dag_workload(seed, N=N, cell=cell, n=10)
    read_count = np.bincount(wl.child[wl.child >= 0], minlength=wl.V)
    assert read_count.max() >= 2, "the generator must share some vertex"
    tw, orig, pulls = _unfold(wl)
    assert oracle.validate(tw.child, tw.parent) == oracle.OK
    g = oracle.run(wl)
    t = oracle.run(tw)
    assert np.array_equal(t["h"], g["h"][orig])
    if "c" in g:
        assert np.array_equal(t["c"], g["c"][orig])
    assert abs(t["loss"] - g["loss"]) <= 1e-14 * abs(g["loss"])
    for k in ("dWx", "dU", "db", "dWs", "dbs"):
        if k in g:
            scale = max(np.abs(g[k]).max(), 1e-30)
            assert np.abs(t[k] - g[k]).max() <= 1e-12 * scale, k
    # a shared input row: the sum over its copies
    dX = np.zeros_like(g["dX"])
    np.add.at(dX, pulls[pulls >= 0], t["dX"])
    assert np.abs(dX - g["dX"]).max() <= 1e-12 * max(np.abs(g["dX"]).max(), 1e-30)
    # per-vertex totals: dL/dh of a graph vertex is the sum over its copies
    dh = np.zeros_like(g["dh"])
    np.add.at(dh, orig, t["dh"])
    assert np.abs(dh - g["dh"]).max() <= 1e-12 * max(np.abs(g["dh"]).max(), 1e-30)


@pytest.mark.parametrize("seed,N", [(10, 2), (11, 3)])
def test_finite_differences_dag(seed, N):
    wl = _dag_workload(seed, N=N, n=7, H=3, D=2, labels="all")
    assert _fd_check(wl) > 50


def test_finite_differences_dag_same_child_twice():
    # vertex 2 reads vertex 0 in both slots; vertex 3 reads 1 and 2, vertex 4 reads 0 and 3
    graph = [[-1, -1], [-1, -1], [0, 0], [1, 2], [0, 3]]
    wl = W.make_workload("twice", [graph], N=2, D=2, H=3, C=3, sigma=0.6, seed=12,
                         inputs="all", labels="all", dag=True)
    assert _fd_check(wl) > 50


def test_finite_differences_dag_treefc():
    wl = _dag_workload(13, N=2, n=7, cell=W.CELL_TREE_FC, H=3, labels="all")
    assert _fd_check(wl) > 20


@pytest.mark.parametrize("N", [3, 4])
def test_finite_differences_nary_childsum(N):
    rng = np.random.Generator(np.random.PCG64(20 + N))
    trees = [W.nary_tree(int(L), N, rng) for L in (1, 4, 7)]
    wl = W.make_workload("n%d" % N, trees, N=N, D=2, H=3, C=3, sigma=0.6, rng=rng,
                         inputs="all", labels="all")
    wl.b[:] = (0.3 * rng.standard_normal(wl.b.shape)).astype(np.float32)
    assert (wl.child >= 0).sum(axis=1).max() >= 3
    assert _fd_check(wl) > 50


def test_nary_slot_permutation_invariance():
    """Child-sum is symmetric in the slots: moving the children to other
    slots changes nothing but the rounding of the c sum."""
    rng = np.random.Generator(np.random.PCG64(25))
    trees = [W.nary_tree(9, 4, rng) for _ in range(3)]
    wl = W.make_workload("n4", trees, N=4, D=3, H=4, C=3, sigma=0.5, rng=rng, labels="all")
    r = oracle.run(wl)
    wl2 = W.make_workload("n4", trees, N=4, D=3, H=4, C=3, sigma=0.5,
                          rng=np.random.Generator(np.random.PCG64(25)), labels="all")
    wl2.X, wl2.Wx, wl2.U, wl2.b, wl2.Ws, wl2.bs = wl.X, wl.Wx, wl.U, wl.b, wl.Ws, wl.bs
    wl2.push_idx = wl.push_idx
    wl2.child = np.ascontiguousarray(wl.child[:, ::-1])
    r2 = oracle.run(wl2)
    for k in ("h", "c", "dU", "dWx", "dX"):
        np.testing.assert_allclose(r[k], r2[k], rtol=0, atol=1e-14 * max(1, np.abs(r[k]).max()))


def test_dag_order_modes_agree():
    wl = _dag_workload(30, N=2, n=15, labels="all")
    r0 = oracle.run(wl, order_mode=0)
    r1 = oracle.run(wl, order_mode=1)
    assert np.array_equal(r0["h"], r1["h"]) and np.array_equal(r0["c"], r1["c"])
    for k in ("dh", "dc", "dU", "dWx", "db", "dX"):
        np.testing.assert_allclose(r0[k], r1[k], rtol=0, atol=1e-13 * max(1, np.abs(r0[k]).max()))


def _longest_path_levels(child):
    V, N = child.shape
    memo = {}

    def depth(v):     # longest chain of child links below v, by enumeration
        if v not in memo:
            best = 0
            for c in child[v]:
                if c >= 0:
                    best = max(best, 1 + depth(int(c)))
            memo[v] = best
        return memo[v]

    return np.array([depth(v) for v in range(V)], dtype=np.int32)


@pytest.mark.parametrize("seed", range(30))
def test_dag_levels_peel_recursive_bruteforce(seed):
    rng = np.random.Generator(np.random.PCG64(100 + seed))
    N = int(rng.integers(1, 5))
    graphs = [W.random_dag(int(rng.integers(1, 25)), N, rng, p_child=0.6, window=8)
              for _ in range(int(rng.integers(1, 5)))]
    child, _, _, _ = W.assemble(graphs, N, rng, shuffle_ids=bool(seed % 2))
    assert oracle.validate(child, None) == oracle.OK
    T1, l1 = oracle.levels(child, "recursive")
    T2, l2 = oracle.levels(child, "frontier")
    want = _longest_path_levels(child)
    assert np.array_equal(l1, want) and np.array_equal(l2, want)
    assert T1 == T2 == int(want.max()) + 1


def test_dag_validation():
    # a shared child is an error for trees, fine for graphs
    child = np.array([[-1, -1], [0, -1], [0, 1]])
    assert oracle.validate(child, np.array([1, 2, -1])) == oracle.ERR_MULTIPARENT
    assert oracle.validate(child, None) == oracle.OK
    # cycles and ranges are still caught
    assert oracle.validate(np.array([[1, -1], [2, -1], [0, -1]]), None) == oracle.ERR_CYCLE
    assert oracle.validate(np.array([[5, -1]]), None) == oracle.ERR_RANGE
    assert oracle.validate(np.array([[0, -1]]), None) == oracle.ERR_CYCLE
    assert oracle.validate(child, None, np.array([0, 0, -1]), 1) == oracle.ERR_DUP_PULL
