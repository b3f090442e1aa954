"""GPU parity of the graph variants and the generic engine (through the C ABI).

Graph inputs (no parent array: a vertex may be read by several vertices,
Section 2, panel (d) of the recurrent-structures figure) and child-sum
vertices with three or four slots (the Section 3.1 figure for N > 2) run the
generic engine: per task, separate products and elementwise gate kernels,
each child link's gradient in its own row, summed per vertex in a fixed
order.  Schedules must equal the oracle's bit for bit (levels by peeling),
with the in-link lists the backward sums over; states, loss and gradients
must meet the fp32 bar of parity.check_fp32.  Also here: the generic engine
on trees (CAVS_GENERIC=1) and the forward fusion ablation
(CAVS_UNFUSED_FWD_GATES=1).
"""
import numpy as np
import pytest
import torch

import oracle
from parity import check_fp32, oracle_sharded
from paper_1712_04048_amd import binding as B
from paper_1712_04048_amd import workloads as W
from paper_1712_04048_amd.runner import Batch

pytestmark = pytest.mark.gpu

ALL_KEYS = ["h", "c", "loss", "dWx", "dU", "db", "dWs", "dbs", "dX"]


@pytest.fixture(scope="module")
def ctx():
    c = B.Context(0)
    yield c
    c.close()


def _parity(ctx, wl, label=""):
    print("parity %s V=%d N=%d H=%d dag=%s" % (label or wl.name, wl.V, wl.N, wl.H, wl.dag),
          flush=True)
    got = Batch(wl, ctx).run()
    ref64 = oracle_sharded(wl)
    ref32 = oracle_sharded(wl, precision="f32")
    return check_fp32(got, ref64, ref32, ALL_KEYS, label or wl.name)


def _dags(seed, N, n_graphs, lo, hi, D=12, H=64, inputs="all", labels="all", window=6,
          p_child=0.7, shuffle=True):
    rng = np.random.Generator(np.random.PCG64(seed))
    graphs = [W.random_dag(int(rng.integers(lo, hi)), N, rng, p_child=p_child, window=window)
              for _ in range(n_graphs)]
    wl = W.make_workload("dag_s%d_n%d" % (seed, N), graphs, N=N, D=D, H=H, C=5, sigma=0.3,
                         rng=rng, inputs=inputs, labels=labels, shuffle_ids=shuffle, dag=True)
    wl.b[:] = (0.1 * rng.standard_normal(wl.b.shape)).astype(np.float32)
    return wl


def _in_links(child_pos):
    V, N = child_pos.shape
    lists = [[] for _ in range(V)]
    for e, c in enumerate(child_pos.reshape(-1)):
        if c >= 0:
            lists[c].append(e)
    off = np.zeros(V + 1, dtype=np.int64)
    off[1:] = np.cumsum([len(x) for x in lists])
    return off, np.array([e for x in lists for e in x], dtype=np.int64)


@pytest.mark.parametrize("seed,N", [(0, 1), (1, 2), (2, 3), (3, 4), (4, 2)])
def test_dag_schedule_bit_exact(ctx, seed, N):
    wl = _dags(seed, N, 30 + 10 * seed, 2, 30)
    print("dag schedule seed=%d N=%d V=%d" % (seed, N, wl.V), flush=True)
    got = Batch(wl, ctx).schedule().host()
    want = oracle.schedule(wl.child, None, wl.pull_idx, wl.push_idx)
    assert got["T"] == want["T"]
    for k in ("level", "order", "pos", "child_pos", "parent_pos", "pull_pos", "push_pos",
              "level_offsets", "pull_list"):
        assert np.array_equal(got[k], want[k]), k
    off, edges = _in_links(want["child_pos"])
    assert np.array_equal(got["in_offsets"], off)
    assert np.array_equal(got["in_edges"][: edges.size], edges)


@pytest.mark.parametrize("N", [3, 4])
def test_nary_tree_schedule_bit_exact(ctx, N):
    rng = np.random.Generator(np.random.PCG64(50 + N))
    trees = [W.nary_tree(int(L), N, rng) for L in rng.integers(1, 40, size=60)]
    wl = W.make_workload("n%d" % N, trees, N=N, D=8, H=64, C=5, rng=rng, shuffle_ids=True)
    got = Batch(wl, ctx).schedule().host()
    want = oracle.schedule(wl.child, wl.parent, wl.pull_idx, wl.push_idx)
    assert got["T"] == want["T"]
    for k in ("level", "order", "pos", "child_pos", "parent_pos", "pull_pos", "push_pos",
              "level_offsets", "pull_list"):
        assert np.array_equal(got[k], want[k]), k


def _status(ctx, child, parent, pull=None, n_x=0):
    dev = ctx.torch_device
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(dev)
    child = np.asarray(child)
    try:
        B.schedule(ctx, t(child), None if parent is None else t(parent),
                   None if pull is None else t(pull), None, n_x=n_x, n_push=0)
        return B.OK
    except B.CavsError as e:
        return e.status


def test_dag_schedule_validation(ctx):
    cases = [
        (np.array([[-1, -1], [0, -1], [0, 1]]), None, None, 0),          # shared child: fine
        (np.array([[1, -1], [2, -1], [0, -1]]), None, None, 0),          # cycle
        (np.array([[0, -1]]), None, None, 0),                             # self loop
        (np.array([[5, -1], [-1, -1]]), None, None, 0),                   # range
        (np.array([[-1, -1], [0, 0]]), None, np.array([0, 0]), 1),        # duplicate pull
        (np.array([[-1, -1, -1], [0, -1, -1], [0, 1, -1]]),               # N = 3 tree with
         np.array([1, 2, -1]), None, 0),                                  # a shared child
        (np.array([[-1, -1, -1], [0, -1, -1], [1, -1, -1]]),
         np.array([2, 2, -1]), None, 0),                                  # N = 3 mismatch
    ]
    for i, (c, p, pl, nx) in enumerate(cases):
        want = oracle.validate(c, p, pl, nx)
        got = _status(ctx, c, p, pl, nx)
        assert got == want, (i, got, want)
    assert _status(ctx, np.array([[-1, -1], [0, -1], [0, 1]]), None) == B.OK


@pytest.mark.parametrize("seed,N", [(10, 1), (11, 2), (12, 3), (13, 4)])
def test_dag_parity(ctx, seed, N):
    _parity(ctx, _dags(seed, N, 20, 3, 30), label="dag_n%d" % N)


def test_dag_parity_same_child_twice_and_leaf_inputs(ctx):
    graphs = [[[-1, -1], [-1, -1], [0, 0], [1, 2], [0, 3]]] * 7
    rng = np.random.Generator(np.random.PCG64(14))
    graphs += [W.random_dag(int(n), 2, rng) for n in rng.integers(2, 25, size=10)]
    wl = W.make_workload("twice", graphs, N=2, D=8, H=64, C=5, sigma=0.3, rng=rng,
                         inputs="leaves", labels="root", dag=True)
    _parity(ctx, wl)


def test_dag_parity_wide_levels(ctx):
    """Levels of several hundred positions at H = 512 (several product
    tiles per level, long lazy products), four slots."""
    wl = _dags(15, 4, 160, 10, 40, D=300, H=512, inputs="leaves", window=10, shuffle=False)
    sizes = np.diff(oracle.schedule(wl.child, None)["level_offsets"])
    assert sizes.max() >= 300
    _parity(ctx, wl, label="dag_wide_n4_h512")


@pytest.mark.parametrize("N", [3, 4])
def test_nary_tree_parity(ctx, N):
    rng = np.random.Generator(np.random.PCG64(60 + N))
    trees = [W.nary_tree(int(L), N, rng) for L in rng.integers(1, 30, size=40)]
    wl = W.make_workload("nary%d" % N, trees, N=N, D=16, H=128, C=5, sigma=0.2, rng=rng,
                         inputs="all" if N == 3 else "leaves", labels="all")
    _parity(ctx, wl)


def test_dag_inference_matches_training_forward(ctx):
    wl = _dags(16, 3, 25, 3, 30)
    b = Batch(wl, ctx)
    train = b.run(backward=False)
    b.h.fill_(float("nan"))
    b.c.fill_(float("nan"))
    b.loss.fill_(float("nan"))
    got = b.run_infer()
    for k in train:
        assert np.array_equal(got[k], train[k]), k


def test_dag_unsupported_combinations(ctx):
    rng = np.random.Generator(np.random.PCG64(17))
    graphs = [W.random_dag(8, 2, rng) for _ in range(3)]
    wl = W.make_workload("fcdag", graphs, cell=W.CELL_TREE_FC, loss=W.LOSS_L2, N=2, H=64,
                         rng=rng, dag=True)
    with pytest.raises(B.CavsError) as e:
        Batch(wl, ctx).run()
    assert e.value.status == B.ERR_UNSUPPORTED
    wl = _dags(18, 2, 5, 3, 10)
    wl.prec = W.PREC_BF16
    with pytest.raises(B.CavsError) as e:
        Batch(wl, ctx).run()
    assert e.value.status == B.ERR_UNSUPPORTED


@pytest.mark.parametrize("maker", ["tiny", "sst_reduced", "varlstm_reduced"])
def test_generic_engine_on_trees(ctx, monkeypatch, maker):
    monkeypatch.setenv("CAVS_GENERIC", "1")
    wl = {"tiny": lambda: W.config_tiny_treelstm(0),
          "sst_reduced": lambda: W.config_treelstm_sst(1, K=24),
          "varlstm_reduced": lambda: W.config_varlstm(2, K=6)}[maker]()
    _parity(ctx, wl, label="generic_" + maker)


def test_generic_engine_full_size_sst(ctx, monkeypatch):
    monkeypatch.setenv("CAVS_GENERIC", "1")
    _parity(ctx, W.config_treelstm_sst(0), label="generic_full_sst")


@pytest.mark.parametrize("case", ["sst_reduced", "varlstm_reduced", "tile_forest", "tiny"])
def test_unfused_forward_gates_ablation(ctx, monkeypatch, case):
    """The forward fusion ablation: the same level product kernels store the
    pre-activations, an elementwise kernel applies the gates."""
    monkeypatch.setenv("CAVS_UNFUSED_FWD_GATES", "1")
    if case == "tile_forest":
        rng = np.random.Generator(np.random.PCG64(35))
        trees = [W.random_split_tree(int(L), rng) for L in rng.integers(2, 14, size=420)]
        wl = W.make_workload(case, trees, N=2, D=32, H=256, C=5, rng=rng, labels="all")
    else:
        wl = {"sst_reduced": lambda: W.config_treelstm_sst(2, K=16),
              "varlstm_reduced": lambda: W.config_varlstm(0, K=6),
              "tiny": lambda: W.config_tiny_treelstm(2)}[case]()
    _parity(ctx, wl, label="unfused_fwd_" + case)


def test_unfused_forward_gates_ablation_bf16(ctx, monkeypatch):
    monkeypatch.setenv("CAVS_UNFUSED_FWD_GATES", "1")
    wl = W.config_treelstm_deep_bf16(1, K=8, D=300, H=1024, lo=8, hi=40)
    sub_rand = list(range(wl.K // 2, wl.K))
    from parity import subset, check
    sub = subset(wl, sub_rand)
    got = Batch(sub, ctx).run()
    want = oracle_sharded(sub, bf16=True)
    check(got, want, ALL_KEYS, 2e-2, "unfused_fwd_bf16", floor=0.1)
