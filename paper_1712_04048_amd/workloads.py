"""Seeded synthetic workloads shaped like the paper's benchmarks (Section 5).

This module only *draws inputs*: graph shapes, parameters, leaf inputs,
labels and targets.  It contains none of the method's arithmetic, so both the
CPU oracle (test infrastructure) and the GPU path consume exactly the arrays it
returns.

Graph convention (Section 3.1, the four message APIs; Algorithm 1 inputs):
  * ``child``  [V, N] int32: global id of child slot k of vertex v, or -1.
  * ``parent`` [V]    int32: global id of v's parent, or -1 for a root.
  * ``pull_idx`` [V]  int32: row of ``X`` that v pulls, or -1 (no input).
  * ``push_idx`` [V]  int32: class label (cross-entropy) or row of ``Y``
    (L2) that v's pushed state is scored against, or -1 (no loss term).
Vertex ids are post-order inside each graph, graph k occupying
``[tree_offsets[k], tree_offsets[k+1])``, unless ``shuffle_ids`` relabels them.

Stand-ins: the paper trains on SST parse trees, PTB sentences and Fold's
synthetic complete trees; none of those data sets is used here.  Only their
shapes are imitated (leaf-count distributions, lengths, branching), with every
value drawn from ``numpy.random.Generator(PCG64(seed))``.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

CELL_TREE_LSTM = 0
CELL_TREE_FC = 1
PREC_FP32 = 0
PREC_BF16 = 1
LOSS_CE = 0
LOSS_L2 = 1
LOSS_NONE = 2     # no loss head: the pushed states go to an external consumer


@dataclass
class Workload:
    name: str
    cell: int
    prec: int
    loss: int
    N: int
    D: int
    H: int
    C: int
    child: np.ndarray
    parent: np.ndarray
    pull_idx: np.ndarray
    push_idx: np.ndarray
    X: np.ndarray
    Y: np.ndarray
    Wx: np.ndarray
    U: np.ndarray
    b: np.ndarray
    Ws: np.ndarray
    bs: np.ndarray
    tree_offsets: np.ndarray
    meta: dict = field(default_factory=dict)
    # graph inputs (panel (d) of the recurrent-structures figure, Section 2):
    # a vertex may be the child of several vertices; ``parent`` is then not
    # passed to the library or the oracle (it holds -1 throughout)
    dag: bool = False

    @property
    def V(self) -> int:
        return int(self.parent.shape[0])

    @property
    def n_x(self) -> int:
        return int(self.X.shape[0])

    @property
    def n_y(self) -> int:
        return int(self.Y.shape[0])

    @property
    def n_push(self) -> int:
        """Upper bound (exclusive) of valid ``push_idx`` values."""
        return self.C if self.loss == LOSS_CE else self.n_y

    @property
    def K(self) -> int:
        return int(self.tree_offsets.shape[0] - 1)


# --------------------------------------------------------------------------
# tree shapes, each returned as a local child list in post-order
# --------------------------------------------------------------------------

def random_split_tree(n_leaves: int, rng: np.random.Generator) -> List[List[int]]:
    """Full binary tree with ``n_leaves`` leaves from recursive uniform splits.

    A subtree with L = 1 is a leaf; otherwise the split s is drawn uniformly
    from {1, ..., L-1}, the left subtree gets s leaves and the right L - s.
    The split of a vertex is drawn before its subtrees are built.
    """
    out: List[List[int]] = []

    def build(L: int) -> int:
        if L == 1:
            out.append([-1, -1])
            return len(out) - 1
        s = int(rng.integers(1, L))
        left = build(s)
        right = build(L - s)
        out.append([left, right])
        return len(out) - 1

    build(int(n_leaves))
    return out


def complete_tree(n_leaves: int) -> List[List[int]]:
    """Complete binary tree (n_leaves a power of two), as in Fold's Tree-FC."""
    assert n_leaves >= 1 and (n_leaves & (n_leaves - 1)) == 0
    out: List[List[int]] = []

    def build(L: int) -> int:
        if L == 1:
            out.append([-1, -1])
            return len(out) - 1
        left = build(L // 2)
        right = build(L // 2)
        out.append([left, right])
        return len(out) - 1

    build(n_leaves)
    return out


def left_branching_tree(n_leaves: int) -> List[List[int]]:
    """I_1 = (leaf_1, leaf_2), I_j = (I_{j-1}, leaf_{j+1}); depth = n_leaves - 1."""
    out: List[List[int]] = [[-1, -1]]
    cur = 0
    for _ in range(1, n_leaves):
        out.append([-1, -1])
        leaf = len(out) - 1
        out.append([cur, leaf])
        cur = len(out) - 1
    return out


def right_branching_tree(n_leaves: int) -> List[List[int]]:
    """Mirror of ``left_branching_tree``: I_j = (leaf_j, I_{j+1})."""
    out: List[List[int]] = []

    def build(first: int) -> int:
        if first == n_leaves - 1:
            out.append([-1, -1])
            return len(out) - 1
        out.append([-1, -1])
        leaf = len(out) - 1
        rest = build(first + 1)
        out.append([leaf, rest])
        return len(out) - 1

    build(0)
    return out


def chain(length: int) -> List[List[int]]:
    """Sequence graph: vertex t has child t-1 (one child slot)."""
    return [[t - 1] for t in range(length)]


def nary_tree(n_leaves: int, N: int, rng: np.random.Generator) -> List[List[int]]:
    """Tree whose internal vertices have between 2 and N children (random
    recursive splits of the leaf range into up to N non-empty parts), with
    the filled slots placed at random among the N."""
    out: List[List[int]] = []

    def build(L: int) -> int:
        if L == 1:
            out.append([-1] * N)
            return len(out) - 1
        parts = int(rng.integers(2, min(N, L) + 1))
        cuts = np.sort(rng.choice(np.arange(1, L), size=parts - 1, replace=False))
        sizes = np.diff(np.concatenate([[0], cuts, [L]]))
        kids = [build(int(sz)) for sz in sizes]
        slots = np.sort(rng.choice(N, size=parts, replace=False))
        row = [-1] * N
        for s_, k in zip(slots, kids):
            row[int(s_)] = k
        out.append(row)
        return len(out) - 1

    build(int(n_leaves))
    return out


def random_dag(n_vertices: int, N: int, rng: np.random.Generator,
               p_child: float = 0.7, window: int = 6) -> List[List[int]]:
    """Directed acyclic graph in topological order: vertex v fills each of
    its N slots with probability p_child by a vertex drawn from the `window`
    vertices before it, so vertices are often read by several vertices
    (and occasionally twice by one).  The first vertex is always a leaf."""
    out: List[List[int]] = []
    for v in range(n_vertices):
        row = []
        for _ in range(N):
            if v > 0 and rng.random() < p_child:
                row.append(int(rng.integers(max(0, v - window), v)))
            else:
                row.append(-1)
        out.append(row)
    return out


# --------------------------------------------------------------------------
# assembling a batch
# --------------------------------------------------------------------------

def assemble(trees: List[List[List[int]]], N: int, rng: np.random.Generator,
             shuffle_ids: bool = False):
    """Concatenate local child lists into global ``child``/``parent`` arrays."""
    sizes = [len(t) for t in trees]
    offsets = np.zeros(len(trees) + 1, dtype=np.int64)
    offsets[1:] = np.cumsum(sizes)
    V = int(offsets[-1])
    child = np.full((V, N), -1, dtype=np.int64)
    for k, t in enumerate(trees):
        base = int(offsets[k])
        for i, ch in enumerate(t):
            assert len(ch) <= N
            for s, c in enumerate(ch):
                if c >= 0:
                    child[base + i, s] = base + c
    perm = None
    if shuffle_ids:
        perm = rng.permutation(V)          # old id -> new id
        newchild = np.full_like(child, -1)
        newchild[perm] = np.where(child >= 0, perm[np.maximum(child, 0)], -1)
        child = newchild
    parent = np.full(V, -1, dtype=np.int64)
    for v in range(V):
        for c in child[v]:
            if c >= 0:
                parent[c] = v
    return child.astype(np.int32), parent.astype(np.int32), offsets.astype(np.int64), perm


def read_by_someone(child: np.ndarray) -> np.ndarray:
    """Vertices that some child link points at (the others are roots)."""
    V = child.shape[0]
    read = np.zeros(V, dtype=bool)
    c = child[child >= 0]
    read[c] = True
    return read


def make_workload(name: str, trees: List[List[List[int]]], *, cell: int = CELL_TREE_LSTM,
                  prec: int = PREC_FP32, loss: int = LOSS_CE, N: int = 2, D: int = 16,
                  H: int = 16, C: int = 5, sigma: float = 0.1, seed: int = 0,
                  rng: Optional[np.random.Generator] = None,
                  inputs: str = "leaves", labels: str = "root",
                  shuffle_ids: bool = False, dag: bool = False) -> Workload:
    """Draw inputs, parameters and labels for a batch of graphs.

    ``inputs``: "leaves" (childless vertices pull an input row), "all", or
    "none".  ``labels``: "root", "all" or "none".  Draw order after the
    shapes: X, the cell parameters, the classifier, then labels or targets.
    ``dag``: the graphs may share vertices between readers (no parent array).
    """
    if rng is None:
        rng = np.random.Generator(np.random.PCG64(seed))
    child, parent, offsets, _ = assemble(trees, N, rng, shuffle_ids)
    if dag:
        parent[:] = -1
    V = parent.shape[0]
    is_leaf = np.all(child < 0, axis=1)
    if inputs == "leaves":
        has_x = is_leaf
    elif inputs == "all":
        has_x = np.ones(V, dtype=bool)
    elif inputs == "none":
        has_x = np.zeros(V, dtype=bool)
    else:
        raise ValueError(inputs)
    if cell == CELL_TREE_FC:
        D = H
        has_x = is_leaf
    pull_idx = np.full(V, -1, dtype=np.int32)
    rows = np.nonzero(has_x)[0]
    pull_idx[rows] = np.arange(rows.size, dtype=np.int32)
    X = rng.standard_normal((rows.size, D)).astype(np.float32)

    if cell == CELL_TREE_LSTM:
        Wx = (sigma * rng.standard_normal((D, 4 * H))).astype(np.float32)
        U = (sigma * rng.standard_normal((H, 4 * H))).astype(np.float32)
        b = np.zeros(4 * H, dtype=np.float32)
    else:
        Wx = np.zeros((0, 0), dtype=np.float32)
        U = (sigma * rng.standard_normal((N * H, H))).astype(np.float32)
        b = np.zeros(H, dtype=np.float32)

    is_root = ~read_by_someone(child)
    if labels == "root":
        has_lab = is_root
    elif labels == "all":
        has_lab = np.ones(V, dtype=bool)
    elif labels == "none":
        has_lab = np.zeros(V, dtype=bool)
    else:
        raise ValueError(labels)
    push_idx = np.full(V, -1, dtype=np.int32)
    if loss == LOSS_NONE:
        Ws = np.zeros((0, 0), dtype=np.float32)
        bs = np.zeros(0, dtype=np.float32)
        Y = np.zeros((0, H), dtype=np.float32)
    elif loss == LOSS_CE:
        Ws = (sigma * rng.standard_normal((H, C))).astype(np.float32)
        bs = np.zeros(C, dtype=np.float32)
        lab_rows = np.nonzero(has_lab)[0]
        push_idx[lab_rows] = rng.integers(0, C, size=lab_rows.size).astype(np.int32)
        Y = np.zeros((0, H), dtype=np.float32)
    else:
        Ws = np.zeros((0, 0), dtype=np.float32)
        bs = np.zeros(0, dtype=np.float32)
        lab_rows = np.nonzero(has_lab)[0]
        push_idx[lab_rows] = np.arange(lab_rows.size, dtype=np.int32)
        Y = rng.uniform(-1.0, 1.0, size=(lab_rows.size, H)).astype(np.float32)
    return Workload(name=name, cell=cell, prec=prec, loss=loss, N=N, D=D, H=H, C=C,
                    child=child, parent=parent, pull_idx=pull_idx, push_idx=push_idx,
                    X=X, Y=Y, Wx=Wx, U=U, b=b, Ws=Ws, bs=bs, tree_offsets=offsets, dag=dag)


# --------------------------------------------------------------------------
# the five benchmark-shaped configurations
# --------------------------------------------------------------------------

def sst_leaf_counts(K: int, rng: np.random.Generator) -> np.ndarray:
    """Parse-tree sizes: round(LogNormal(2.843, 0.450)) clipped to [2, 56].

    Mean about 19 leaves, range [2, 56], as for the sentiment-treebank trees
    of Section 5 (whose data is not used).
    """
    raw = rng.lognormal(mean=2.843, sigma=0.450, size=K)
    return np.clip(np.rint(raw), 2, 56).astype(np.int64)


def config_tiny_treelstm(seed: int = 0, shuffle_ids: bool = False) -> Workload:
    """Binary child-sum Tree-LSTM, D=H=64, 8 random-split trees with 4..16 leaves."""
    rng = np.random.Generator(np.random.PCG64(seed))
    leaves = rng.integers(4, 17, size=8)
    trees = [random_split_tree(int(L), rng) for L in leaves]
    return make_workload("treelstm_tiny_d64_h64_bs8", trees, N=2, D=64, H=64, C=5,
                         sigma=0.1, rng=rng, inputs="leaves", labels="root",
                         shuffle_ids=shuffle_ids)


def config_varlstm(seed: int = 0, K: int = 64) -> Workload:
    """Var-LSTM: 64 chains with lengths uniform in [10, 100], D=H=512."""
    rng = np.random.Generator(np.random.PCG64(seed))
    lengths = rng.integers(10, 101, size=K)
    trees = [chain(int(n)) for n in lengths]
    return make_workload("varlstm_chains_d512_h512_bs64", trees, N=1, D=512, H=512, C=5,
                         sigma=0.05, rng=rng, inputs="all", labels="root")


def config_treefc(seed: int = 0, K: int = 64, leaves: int = 256, H: int = 512) -> Workload:
    """Tree-FC over 64 complete binary trees with 256 leaves (511 vertices, 9 levels)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    trees = [complete_tree(leaves) for _ in range(K)]
    return make_workload(f"treefc_complete{leaves}_h{H}_bs{K}", trees, cell=CELL_TREE_FC,
                         loss=LOSS_L2, N=2, D=H, H=H, C=0, sigma=0.05, rng=rng,
                         inputs="leaves", labels="root")


def config_treelstm_sst(seed: int = 0, K: int = 256, D: int = 300, H: int = 512) -> Workload:
    """Tree-LSTM D=300, H=512 over 256 parse-shaped trees, CE at every vertex."""
    rng = np.random.Generator(np.random.PCG64(seed))
    leaves = sst_leaf_counts(K, rng)
    trees = [random_split_tree(int(L), rng) for L in leaves]
    return make_workload(f"treelstm_sst_d{D}_h{H}_bs{K}", trees, N=2, D=D, H=H, C=5,
                         sigma=0.05, rng=rng, inputs="leaves", labels="all")


def config_treelstm_deep_bf16(seed: int = 0, K: int = 256, D: int = 300, H: int = 1024,
                              lo: int = 32, hi: int = 128) -> Workload:
    """Tree-LSTM H=1024 in bf16 MFMA; 32..128 leaves, half the trees left-branching."""
    rng = np.random.Generator(np.random.PCG64(seed))
    leaves = rng.integers(lo, hi + 1, size=K)
    trees = []
    for k, L in enumerate(leaves):
        if k < K // 2:
            trees.append(left_branching_tree(int(L)))
        else:
            trees.append(random_split_tree(int(L), rng))
    return make_workload(f"treelstm_deep_d{D}_h{H}_bs{K}_bf16", trees, prec=PREC_BF16, N=2,
                         D=D, H=H, C=5, sigma=0.03, rng=rng, inputs="leaves", labels="all")


WORKLOADS = {
    "tiny": config_tiny_treelstm,
    "varlstm": config_varlstm,
    "treefc": config_treefc,
    "sst": config_treelstm_sst,
    "deep_bf16": config_treelstm_deep_bf16,
}
