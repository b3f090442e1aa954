"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Schedules must match bit for bit.  fp32 states, loss and gradients must
match the fp64 oracle under the floored relative error of parity.rel_err (1%
floor) to max(1e-4, 2 x the error of the oracle's own fp32 build), element by
element (parity.check_fp32).  bf16 runs are compared with the bf16-emulating
oracle: element-wise (10% floor) to 2e-2 where the graphs are shallow,
normwise to 2e-2 through deep chains (see _parity_bf16).
"""
import numpy as np
import pytest
import torch

import oracle
from parity import check, check_fp32, oracle_sharded, subset
from paper_1712_04048_amd import binding as B
from paper_1712_04048_amd import workloads as W
from paper_1712_04048_amd.runner import Batch

pytestmark = pytest.mark.gpu

TOL_FP32 = 1e-4
ALL_KEYS = ["h", "c", "loss", "dWx", "dU", "db", "dWs", "dbs", "dX"]


@pytest.fixture(scope="module")
def ctx():
    c = B.Context(0)
    yield c
    c.close()


def _forest(seed, N=2, shuffle=False, max_trees=40, max_leaves=40):
    rng = np.random.Generator(np.random.PCG64(seed))
    trees = []
    for _ in range(int(rng.integers(1, max_trees))):
        L = int(rng.integers(1, max_leaves))
        kind = int(rng.integers(0, 4))
        if N == 1:
            trees.append(W.chain(L))
        elif kind == 0:
            trees.append(W.random_split_tree(L, rng))
        elif kind == 1:
            trees.append(W.left_branching_tree(L))
        elif kind == 2:
            trees.append(W.right_branching_tree(L))
        else:
            trees.append(W.complete_tree(1 << int(rng.integers(0, 6))))
    return W.make_workload("forest", trees, N=N, D=4, H=64, C=5, rng=rng,
                           inputs="leaves" if seed % 3 else "all",
                           labels="all" if seed % 2 else "root", shuffle_ids=shuffle)


def _gpu_schedule(ctx, wl):
    b = Batch(wl, ctx)
    s = b.schedule()
    return s.host()


def _compare_schedule(got, want):
    assert got["T"] == want["T"]
    for k in ("level", "order", "pos", "child_pos", "parent_pos", "pull_pos", "push_pos",
              "level_offsets", "pull_list"):
        assert np.array_equal(got[k], want[k]), k
    assert got["n_pull"] == want["n_pull"]


@pytest.mark.parametrize("seed", range(12))
def test_schedule_bit_exact(ctx, seed):
    N = 1 if seed % 4 == 0 else 2
    wl = _forest(seed, N=N, shuffle=seed % 2 == 1)
    print("schedule case seed=%d V=%d N=%d" % (seed, wl.V, N), flush=True)
    got = _gpu_schedule(ctx, wl)
    want = oracle.schedule(wl.child, wl.parent, wl.pull_idx, wl.push_idx)
    _compare_schedule(got, want)
    assert got["n_labelled"] == int((wl.push_idx >= 0).sum())


@pytest.mark.parametrize("maker", ["sst", "varlstm", "treefc", "deep_bf16", "big",
                                   "deep_chains_leaf_inputs", "deep_chains_all_inputs"])
def test_schedule_bit_exact_benchmark_shapes(ctx, maker):
    if maker == "big":   # > 65536 vertices, more than 64 radix tiles
        rng = np.random.Generator(np.random.PCG64(5))
        trees = [W.random_split_tree(int(L), rng) for L in rng.integers(2, 300, size=500)]
        wl = W.make_workload("big", trees, N=2, D=4, H=64, C=5, rng=rng, shuffle_ids=True)
        assert wl.V > 65536
    elif maker.startswith("deep_chains"):
        # T > 256: the level sort takes two 8-bit passes, and its last pass
        # also lists the pulling positions
        rng = np.random.Generator(np.random.PCG64(6))
        trees = [W.chain(600), W.chain(257), W.chain(1)]
        trees += [W.random_split_tree(int(L), rng) for L in rng.integers(2, 60, size=80)]
        inputs = "all" if maker.endswith("all_inputs") else "leaves"
        wl = W.make_workload(maker, trees, N=2, D=4, H=64, C=5, rng=rng, inputs=inputs,
                             shuffle_ids=True)
    else:
        wl = W.WORKLOADS[maker](0)
    print("schedule shape %s V=%d" % (maker, wl.V), flush=True)
    got = _gpu_schedule(ctx, wl)
    want = oracle.schedule(wl.child, wl.parent, wl.pull_idx, wl.push_idx)
    _compare_schedule(got, want)


def _forest_of_size(V, seed):
    """Random binary trees topped up with single-vertex trees to exactly V vertices."""
    rng = np.random.Generator(np.random.PCG64(seed))
    trees, n = [], 0
    while True:
        t = W.random_split_tree(int(rng.integers(2, 80)), rng)
        if n + len(t) > V:
            break
        trees.append(t)
        n += len(t)
    trees += [W.chain(1)] * (V - n)
    wl = W.make_workload("forest%d" % V, trees, N=2, D=4, H=64, C=5, rng=rng, shuffle_ids=True)
    assert wl.V == V
    return wl


# 16384 vertices is the most the one-workgroup scheduler takes; one more goes
# through the multi-launch path
@pytest.mark.parametrize("V", [16384, 16385])
def test_schedule_bit_exact_at_one_workgroup_limit(ctx, V):
    wl = _forest_of_size(V, V)
    print("schedule V=%d" % V, flush=True)
    _compare_schedule(_gpu_schedule(ctx, wl), oracle.schedule(wl.child, wl.parent, wl.pull_idx,
                                                              wl.push_idx))


def test_schedule_bit_exact_many_input_rows(ctx):
    # input row ids spread over 300000 rows (more than the one-workgroup
    # scheduler tracks), so a small batch also takes the multi-launch path
    wl = _forest(3)
    pull = np.where(wl.pull_idx >= 0, wl.pull_idx * 250 + 11, -1).astype(np.int32)
    n_x = 300000
    assert pull.max() < n_x
    dev = ctx.torch_device
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(dev)
    got = B.schedule(ctx, t(wl.child), t(wl.parent), t(pull), t(wl.push_idx), n_x=n_x,
                     n_push=wl.n_push).host()
    _compare_schedule(got, oracle.schedule(wl.child, wl.parent, pull, wl.push_idx))


def _raw_schedule_status(ctx, child, parent, pull=None, push=None, n_x=0, n_push=0):
    dev = ctx.torch_device
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(dev)
    try:
        B.schedule(ctx, t(child), t(parent), None if pull is None else t(pull),
                   None if push is None else t(push), n_x=n_x, n_push=n_push)
        return B.OK
    except B.CavsError as e:
        return e.status


# pad > 0 appends isolated vertices, past the one-workgroup scheduler's limit
@pytest.mark.parametrize("pad", [0, 16400])
def test_schedule_rejects_invalid_graphs(ctx, pad):
    child = np.array([[-1, -1], [-1, -1], [0, 1]])
    parent = np.array([2, 2, -1])
    cases = []
    c = child.copy(); c[2, 1] = 3; cases.append((c, parent, None, None, 0, 0))
    p = parent.copy(); p[0] = -2; cases.append((child, p, None, None, 0, 0))
    c = child.copy(); c[2, 1] = 0; cases.append((c, parent, None, None, 0, 0))
    cases.append((np.array([[-1, -1], [0, -1], [0, 1]]), np.array([1, 2, -1]), None, None, 0, 0))
    p = parent.copy(); p[1] = -1; cases.append((child, p, None, None, 0, 0))
    p = parent.copy(); p[2] = 0; cases.append((child, p, None, None, 0, 0))
    cases.append((np.array([[-1, -1], [-1, -1], [0, 1], [4, -1], [3, -1]]),
                  np.array([2, 2, -1, 4, 3]), None, None, 0, 0))
    cases.append((np.array([[0, -1]]), np.array([0]), None, None, 0, 0))
    cases.append((child, parent, np.array([0, 0, -1]), None, 2, 0))
    cases.append((child, parent, np.array([0, 2, -1]), None, 2, 0))
    cases.append((child, parent, None, np.array([0, 5, -1]), 0, 5))
    cases.append((np.array([[-1, -1], [0, 7], [0, 1]]), parent, None, None, 0, 0))
    for i, (c, p, pl, ps, nx, npush) in enumerate(cases):
        if pad:
            c = np.vstack([c, -np.ones((pad, c.shape[1]), np.int64)])
            p = np.concatenate([p, -np.ones(pad, np.int64)])
            pl = None if pl is None else np.concatenate([pl, -np.ones(pad, np.int64)])
            ps = None if ps is None else np.concatenate([ps, -np.ones(pad, np.int64)])
        want = oracle.validate(c, p, pl, nx, ps, npush)
        got = _raw_schedule_status(ctx, c, p, pl, ps, nx, npush)
        assert want != oracle.OK
        assert got == want, (i, got, want)
    # a valid graph still schedules after the failures
    assert _raw_schedule_status(ctx, child, parent) == B.OK


def _parity(ctx, wl, keys=ALL_KEYS, label=""):
    print("parity %s V=%d H=%d" % (label or wl.name, wl.V, wl.H), flush=True)
    got = Batch(wl, ctx).run()
    ref64 = oracle_sharded(wl)
    ref32 = oracle_sharded(wl, precision="f32")
    return check_fp32(got, ref64, ref32, keys, label or wl.name)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_parity_tiny_treelstm(ctx, seed):
    _parity(ctx, W.config_tiny_treelstm(seed))


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_parity_tiny_treelstm_shuffled_ids(ctx, seed):
    _parity(ctx, W.config_tiny_treelstm(seed, shuffle_ids=True))


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_parity_sst_shaped_reduced(ctx, seed):
    _parity(ctx, W.config_treelstm_sst(seed, K=12))


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_parity_varlstm_reduced(ctx, seed):
    _parity(ctx, W.config_varlstm(seed, K=6))


@pytest.mark.parametrize("H,N", [(256, 2), (256, 1), (768, 2)])
def test_parity_hidden_widths(ctx, H, N):
    """Widths that are not multiples of 512 split the small-level products
    over four wavefronts instead of eight; the forests have levels on both
    sides of the tile threshold and every vertex labelled."""
    rng = np.random.default_rng(7 * H + N)
    if N == 2:
        trees = [W.random_split_tree(int(L), rng) for L in rng.integers(2, 40, size=40 if H < 768 else 24)]
    else:
        trees = [W.chain(int(L)) for L in rng.integers(5, 60, size=24)]
    wl = W.make_workload("widths_h%d_n%d" % (H, N), trees, N=N, D=32, H=H, C=5, rng=rng,
                         labels="all")
    _parity(ctx, wl)


@pytest.mark.parametrize("case", ["trees_fp32", "chains_fp32", "trees_bf16"])
def test_parity_tile_levels(ctx, case):
    """Forests whose internal levels reach the LDS-tiled products (levels of
    300 positions or more; 64-position forward tiles from 1024): every
    state, the loss and every gradient against the oracle, so the tiled
    forward and backward products are checked element by element, not only
    through properties at full size."""
    rng = np.random.Generator(np.random.PCG64({"trees_fp32": 31, "chains_fp32": 32,
                                               "trees_bf16": 33}[case]))
    if case == "chains_fp32":
        trees = [W.chain(int(L)) for L in rng.integers(3, 9, size=330)]
        wl = W.make_workload(case, trees, N=1, D=32, H=256, C=5, rng=rng, inputs="all",
                             labels="all")
    elif case == "trees_fp32":
        trees = [W.random_split_tree(int(L), rng) for L in rng.integers(2, 14, size=420)]
        wl = W.make_workload(case, trees, N=2, D=32, H=256, C=5, rng=rng, labels="all")
    else:
        # the bf16-emulating oracle rounds every product operand: 300 cherries
        # keep it to about half a minute and still give one 300-position level
        wl = W.make_workload(case, [W.complete_tree(2)] * 300, prec=W.PREC_BF16, N=2, D=32,
                             H=256, C=5, rng=rng, labels="all")
    sizes = np.diff(oracle.schedule(wl.child, wl.parent, wl.pull_idx, wl.push_idx)["level_offsets"])
    assert sizes[1] >= 300
    if case != "trees_bf16":
        assert sizes[2] >= 300
    if case == "trees_fp32":
        assert sizes[1] >= 1024
    if case == "trees_bf16":
        _parity_bf16(ctx, wl, case, elementwise=True)
    else:
        _parity(ctx, wl, label=case)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_parity_treefc_reduced(ctx, seed):
    _parity(ctx, W.config_treefc(seed, K=2, leaves=64))


def test_parity_treefc_cross_entropy(ctx):
    rng = np.random.Generator(np.random.PCG64(3))
    trees = [W.random_split_tree(int(L), rng) for L in rng.integers(1, 30, size=7)]
    wl = W.make_workload("fc_ce", trees, cell=W.CELL_TREE_FC, loss=W.LOSS_CE, N=2, H=64, C=5,
                         sigma=0.2, rng=rng, labels="all")
    _parity(ctx, wl)


@pytest.mark.parametrize("case", ["forest_n2_h128", "chains_n1_h192", "unary_slots_h64"])
def test_parity_treefc_tiles(ctx, case):
    """Tree-FC levels of >= 300 positions (the LDS-ring tiles) with a ragged
    last row tile: binary forests, one-slot chains at H = 192 (three unit
    tiles), and vertices with only slot 0 or only slot 1 filled."""
    rng = np.random.Generator(np.random.PCG64(21))
    if case == "forest_n2_h128":
        trees = [W.random_split_tree(int(L), rng) for L in rng.integers(2, 13, size=450)]
        kw = dict(N=2, H=128)
    elif case == "chains_n1_h192":
        trees = [W.chain(int(n)) for n in rng.integers(2, 11, size=400)]
        kw = dict(N=1, H=192)
    else:
        trees = [[[-1, -1], [0, -1], [-1, -1], [1, 2]]] * 331 + [[[-1, -1], [-1, 0]]] * 70
        kw = dict(N=2, H=64)
    wl = W.make_workload("fc_" + case, trees, cell=W.CELL_TREE_FC, loss=W.LOSS_L2, D=kw["H"],
                         C=0, sigma=0.1, rng=rng, inputs="leaves", labels="all", **kw)
    wl.b[:] = (0.1 * rng.standard_normal(wl.b.shape)).astype(np.float32)
    sizes = np.diff(oracle.schedule(wl.child, wl.parent)["level_offsets"])
    assert sizes[1] >= 300 and sizes[1] % 64 != 0
    _parity(ctx, wl, label=case)


EDGE = {
    "single_vertex_trees": lambda rng: ([[[-1, -1]]] * 37, dict()),
    "chain_len1_and_mixed": lambda rng: ([W.chain(1), W.chain(3), W.chain(1), W.chain(70)],
                                         dict(N=1, inputs="all", labels="all")),
    "left_branching": lambda rng: ([W.left_branching_tree(L) for L in (2, 9, 33)],
                                   dict(labels="all")),
    "right_branching": lambda rng: ([W.right_branching_tree(L) for L in (2, 9, 33)],
                                    dict(labels="all")),
    "unary_vertices": lambda rng: ([[[-1, -1], [0, -1], [-1, -1], [1, 2], [-1, 3]]] * 5,
                                   dict(labels="all")),
    "inputs_everywhere": lambda rng: ([W.random_split_tree(int(L), rng) for L in (5, 17, 3, 40)],
                                      dict(inputs="all", labels="all")),
    "leaves_without_input": lambda rng: ([W.random_split_tree(int(L), rng) for L in (5, 17, 3)],
                                         dict(inputs="none", labels="all")),
    "no_labels": lambda rng: ([W.random_split_tree(int(L), rng) for L in (5, 6)],
                              dict(labels="none")),
    "wide_ragged_level": lambda rng: ([W.random_split_tree(int(L), rng)
                                       for L in rng.integers(1, 9, size=150)],
                                      dict(labels="all")),
}


@pytest.mark.parametrize("case", sorted(EDGE))
def test_parity_edge_cases(ctx, case):
    rng = np.random.Generator(np.random.PCG64(11))
    trees, kw = EDGE[case](rng)
    args = dict(N=2, D=12, H=64, C=5, sigma=0.3, rng=rng)
    args.update(kw)
    wl = W.make_workload(case, trees, **args)
    wl.b[:] = (0.1 * rng.standard_normal(wl.b.shape)).astype(np.float32)
    _parity(ctx, wl, label=case)


@pytest.mark.parametrize("cell", [W.CELL_TREE_LSTM, W.CELL_TREE_FC])
def test_empty_batch(ctx, cell):
    """No graphs at all: zero levels, loss 0, every gradient overwritten with
    zeros (the outputs are poisoned first), as the oracle gives."""
    rng = np.random.Generator(np.random.PCG64(4))
    kw = dict(N=2, D=12, H=64, C=5) if cell == W.CELL_TREE_LSTM else \
        dict(cell=cell, loss=W.LOSS_L2, N=2, H=64)
    wl = W.make_workload("empty", [], rng=rng, **kw)
    assert wl.V == 0
    b = Batch(wl, ctx)
    b.schedule()
    assert b.sched.T == 0
    b.alloc()
    for g in b.grads.values():
        g.fill_(float("nan"))
    b.loss.fill_(float("nan"))
    got = b.run()
    want = oracle.run(wl)
    assert got["loss"] == want["loss"] == 0.0
    for k, v in b.grads.items():
        assert np.array_equal(got[k], want[k]), k
    b.loss.fill_(float("nan"))
    assert b.run_infer()["loss"] == 0.0


@pytest.mark.parametrize("maker", ["sst", "varlstm", "treefc"])
def test_full_size_parity(ctx, maker):
    """The benchmark-size batches in the benchmark's launch configuration
    (the SST-shaped Tree-LSTM at H = 512 reaches the 32x32 / 64x32 level
    tiles with the XCD map, the four-wavefront backward split-K and the
    full-length lazy products): every state, the loss and every gradient
    against the fp64 oracle, element by element."""
    wl = W.WORKLOADS[maker](0)
    sizes = np.diff(oracle.schedule(wl.child, wl.parent)["level_offsets"])
    print("full-size %s V=%d levels=%s" % (maker, wl.V, sizes.tolist()), flush=True)
    if maker == "sst":
        assert sizes[1] >= 1024 and (sizes[1:] >= 300).sum() >= 4
        assert ((sizes > 128) & (sizes < 300)).any()
    _parity(ctx, wl, label="full_" + maker)


# ---------------------------------------------------------------------------
# Inference (cavs_infer): the forward without anything kept for a backward.
# Same kernels, so h, c and the loss must equal cavs_forward's bit for bit;
# against the oracle, the forward's tolerance.
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("maker", ["tiny", "sst", "varlstm", "treefc", "deep_bf16"])
def test_infer_bit_identical_to_forward_full_size(ctx, maker):
    wl = W.WORKLOADS[maker](0)
    print("infer vs forward %s V=%d" % (maker, wl.V), flush=True)
    b = Batch(wl, ctx)
    train = b.run(backward=False)
    b.h.fill_(float("nan"))
    if b.c is not None:
        b.c.fill_(float("nan"))
    b.loss.fill_(float("nan"))
    got = b.run_infer()
    assert b.ws_infer.numel() < b.ws.numel()
    for k in train:
        assert np.array_equal(got[k], train[k]), k


def _infer_parity(ctx, wl, bf16=False):
    print("infer parity %s V=%d H=%d" % (wl.name, wl.V, wl.H), flush=True)
    got = Batch(wl, ctx).run_infer()
    want = oracle.run(wl, backward=False, bf16=bf16)
    keys = [k for k in ("h", "c", "loss") if k in want]
    if bf16:
        return check(got, want, keys, TOL_BF16, "infer_" + wl.name, floor=1.0)
    want32 = oracle.run(wl, backward=False, precision="f32")
    return check_fp32(got, want, want32, keys, "infer_" + wl.name)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_infer_parity_reduced(ctx, seed):
    _infer_parity(ctx, W.config_treelstm_sst(seed, K=12))
    _infer_parity(ctx, W.config_varlstm(seed, K=6))
    _infer_parity(ctx, W.config_treefc(seed, K=2, leaves=64))
    _infer_parity(ctx, W.config_tiny_treelstm(seed, shuffle_ids=seed == 1))


@pytest.mark.parametrize("case", ["single_vertex_trees", "no_labels", "leaves_without_input",
                                  "inputs_everywhere"])
def test_infer_parity_edge_cases(ctx, case):
    rng = np.random.Generator(np.random.PCG64(12))
    trees, kw = EDGE[case](rng)
    args = dict(N=2, D=12, H=64, C=5, sigma=0.3, rng=rng)
    args.update(kw)
    wl = W.make_workload(case, trees, **args)
    _infer_parity(ctx, wl)


def test_infer_parity_bf16_reduced(ctx):
    wl = W.config_treelstm_deep_bf16(0, K=4, D=300, H=1024, lo=8, hi=40)
    _infer_parity(ctx, wl, bf16=True)


def test_infer_rejects_short_workspace(ctx):
    wl = W.config_tiny_treelstm(0)
    b = Batch(wl, ctx)
    b.schedule()
    b.alloc()
    need = B.infer_workspace_bytes(b.params, b.sched)
    assert 0 < need < b.ws.numel()
    with pytest.raises(B.CavsError) as e:
        B.infer(ctx, b.params, b.sched, b.X, b.Y, b.ws[:need - 1], b.h, b.c, b.loss)
    assert e.value.status == B.ERR_WORKSPACE
    B.infer(ctx, b.params, b.sched, b.X, b.Y, b.ws[:need], b.h, b.c, b.loss)
    torch.cuda.synchronize()
    assert np.isfinite(b.loss.item())


def test_runs_on_the_callers_stream():
    """A context bound to a non-default stream (default priority) enqueues
    everything there, and set_stream moves it: the outputs equal those of a
    run on the default stream bit for bit."""
    wl = W.config_treelstm_sst(1, K=24)
    c1 = B.Context(0)
    side = torch.cuda.Stream()
    c2 = B.Context(0, stream=side)
    try:
        ref = Batch(wl, c1).run()
        b = Batch(wl, c2)
        torch.cuda.synchronize()
        with torch.cuda.stream(side):
            got = b.run()
        for k in ref:
            assert np.array_equal(np.asarray(got[k]), np.asarray(ref[k])), k
        c2.set_stream(torch.cuda.current_stream())
        got2 = b.run()
        for k in ref:
            assert np.array_equal(np.asarray(got2[k]), np.asarray(ref[k])), k
    finally:
        c2.close()
        c1.close()


def test_graph_captured_replays_match_eager():
    """forward + backward captured into a HIP graph (torch's stream capture
    of the library's launches on a side stream) and replayed three times,
    with eager runs and synchronisations in between: every replay gives the
    eager run's outputs bit for bit."""
    wl = W.config_treelstm_sst(3, K=24)
    side = torch.cuda.Stream()
    c = B.Context(0, stream=side)
    try:
        b = Batch(wl, c)
        with torch.cuda.stream(side):
            ref = b.run()
        g = torch.cuda.CUDAGraph()
        torch.cuda.synchronize()
        with torch.cuda.graph(g, stream=side):
            b.forward()
            b.backward()
        torch.cuda.synchronize()
        for rep in range(3):
            for t in b.grads.values():
                t.fill_(float("nan"))
            b.h.fill_(float("nan"))
            with torch.cuda.stream(side):
                g.replay()
            torch.cuda.synchronize()
            got = b.results()
            for k in ref:
                assert np.array_equal(np.asarray(got[k]), np.asarray(ref[k])), (rep, k)
            with torch.cuda.stream(side):
                b.forward()
                b.backward()
            c.sync()
        del g
    finally:
        c.close()


def test_determinism_bitwise(ctx):
    wl = W.config_treelstm_sst(0, K=24)
    b = Batch(wl, ctx)
    r1 = b.run()
    r2 = b.run()
    for k in r1:
        assert np.array_equal(np.asarray(r1[k]), np.asarray(r2[k])), k


@pytest.mark.parametrize("entry", ["forward", "infer"])
def test_forward_rejects_bad_arguments(ctx, entry):
    call = B.forward if entry == "forward" else B.infer
    wl = W.config_tiny_treelstm(0)
    b = Batch(wl, ctx)
    b.schedule()
    b.alloc()
    small = torch.empty(16, dtype=torch.uint8, device=ctx.torch_device)
    with pytest.raises(B.CavsError) as e:
        call(ctx, b.params, b.sched, b.X, b.Y, small, b.h, b.c, b.loss)
    assert e.value.status == B.ERR_WORKSPACE
    p = B.Params(**{**b.params.__dict__, "H": 48})
    with pytest.raises(B.CavsError) as e:
        call(ctx, p, b.sched, b.X, b.Y, b.ws, b.h, b.c, b.loss)
    assert e.value.status in (B.ERR_UNSUPPORTED, B.ERR_WORKSPACE)
    p = B.Params(**{**b.params.__dict__, "N": 1})
    with pytest.raises(B.CavsError) as e:
        call(ctx, p, b.sched, b.X, b.Y, b.ws, b.h, b.c, b.loss)
    assert e.value.status == B.ERR_ARG
    with pytest.raises(B.CavsError) as e:   # no h_out
        call(ctx, b.params, b.sched, b.X, b.Y, b.ws, None, b.c, b.loss)
    assert e.value.status == B.ERR_ARG


# ---------------------------------------------------------------------------
# bf16 matrix products (fp32 accumulation) against the oracle that rounds the
# same operands to bf16; the error against the plain fp64 oracle is reported.
#
# Shallow graphs are held element by element (10% floor) to 2e-2.  Through
# deep chains the bound is applied normwise (max|g - o| / max|o| <= 2e-2):
# the emulating oracle cannot follow the GPU bit for bit there -- an fp32-vs-
# fp64 difference of ~1e-7 occasionally falls on the other side of a bf16
# rounding point, moves that operand by half a bf16 ulp (2e-3), and the
# perturbation spreads through U at every later level; after tens of levels
# the two differ by about an ulp everywhere, and element-wise errors of
# elements near 10% of the maximum reach 1-3e-2.  The element-wise figure is
# printed alongside.  Deep cases: the reduced H = 1024 batches whose first
# half is left-branching (8-40 levels), chains of 40, and the persistent /
# ablation runs of those batches.
# ---------------------------------------------------------------------------
TOL_BF16 = 2e-2


def _parity_bf16(ctx, wl, label, elementwise=False):
    print("bf16 parity %s V=%d H=%d (%s)" % (label, wl.V, wl.H,
                                            "element-wise" if elementwise else "normwise"),
          flush=True)
    got = Batch(wl, ctx).run()
    want = oracle_sharded(wl, bf16=True)
    from parity import rel_err
    elem = {k: rel_err(got[k], want[k], 0.1) for k in ALL_KEYS if k in want and k != "loss"}
    plain = oracle_sharded(wl, bf16=False)
    vs64 = {k: rel_err(got[k], plain[k], 1.0) for k in ALL_KEYS if k in plain and k != "loss"}
    print("  element-wise (floor 0.1) vs bf16-emulating oracle:", elem)
    print("  normwise vs fp64 oracle:", vs64)
    errs = check(got, want, ALL_KEYS, TOL_BF16, label, floor=0.1 if elementwise else 1.0)
    print("  checked:", errs)
    return errs


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_parity_bf16_deep_reduced(ctx, seed):
    wl = W.config_treelstm_deep_bf16(seed, K=4, D=300, H=1024, lo=8, hi=40)
    _parity_bf16(ctx, wl, "deep_bf16_reduced_%d" % seed)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_parity_bf16_random_split_half_elementwise(ctx, seed):
    """The random-split half of the H = 1024 bf16 configuration (the
    left-branching half is the deep case), element by element."""
    wl = W.config_treelstm_deep_bf16(seed, K=8, D=300, H=1024, lo=8, hi=40)
    sub = subset(wl, list(range(wl.K // 2, wl.K)))
    _parity_bf16(ctx, sub, "deep_bf16_random_half_%d" % seed, elementwise=True)


def test_parity_bf16_small_shapes(ctx):
    rng = np.random.Generator(np.random.PCG64(21))
    trees = [W.random_split_tree(int(L), rng) for L in (1, 3, 9, 20)] + [W.left_branching_tree(12)]
    wl = W.make_workload("bf16_inputs_everywhere", trees, prec=W.PREC_BF16, N=2, D=36, H=64,
                         C=5, sigma=0.2, rng=rng, inputs="all", labels="all")
    _parity_bf16(ctx, wl, "bf16_inputs_everywhere", elementwise=True)
    wl = W.make_workload("bf16_chains", [W.chain(n) for n in (1, 7, 40)], prec=W.PREC_BF16, N=1,
                         D=64, H=128, C=5, sigma=0.1, rng=rng, inputs="all", labels="all")
    _parity_bf16(ctx, wl, "bf16_chains")


def test_parity_bf16_two_row_split_k(ctx):
    """bf16 levels of 64 positions or more below the tile threshold run the
    split-K products with two 16-position row tiles per workgroup and four
    contraction wavefronts; at H = 256 every level takes split-K (no tiles,
    no XCD loop), for one and for two child slots.  Level sizes: trees
    138 / 67 (the second row-tile pair ragged) / 2 / 2; chains 70 / 70 /
    64 / 63 / 63 (both sides of the 64-position switch)."""
    rng = np.random.Generator(np.random.PCG64(33))
    trees = [W.complete_tree(2)] * 65 + [W.left_branching_tree(4)] * 2
    wl = W.make_workload("bf16_two_rows_trees", trees, prec=W.PREC_BF16, N=2, D=32, H=256, C=5,
                         sigma=0.2, rng=rng, labels="all")
    _parity_bf16(ctx, wl, "bf16_two_rows_trees", elementwise=True)
    chains = [W.chain(2)] * 6 + [W.chain(3)] + [W.chain(5)] * 63
    wl = W.make_workload("bf16_two_rows_chains", chains, prec=W.PREC_BF16, N=1, D=32, H=256, C=5,
                         sigma=0.2, rng=rng, inputs="all", labels="all")
    _parity_bf16(ctx, wl, "bf16_two_rows_chains", elementwise=True)


def test_full_size_bf16_states_on_sampled_graphs(ctx):
    """Config of 256 trees, H=1024, half left-branching (T=128), bf16 products:
    full batch on the GPU, states of eight sampled graphs (three
    left-branching, five random-split) against the oracle run on those
    graphs alone (a graph's states depend only on itself)."""
    wl = W.config_treelstm_deep_bf16(0)
    print("full-size deep_bf16 V=%d" % wl.V, flush=True)
    got = Batch(wl, ctx).run()
    rng = np.random.Generator(np.random.PCG64(2))
    trees = sorted(rng.choice(wl.K // 2, size=3, replace=False).tolist() +
                   (wl.K // 2 + rng.choice(wl.K // 2, size=5, replace=False)).tolist())
    sub = subset(wl, trees)
    want = oracle_sharded(sub, backward=False, bf16=True)
    ids = np.concatenate([np.arange(wl.tree_offsets[k], wl.tree_offsets[k + 1]) for k in trees])
    check({k: got[k][ids] for k in ("h", "c")}, want, ["h", "c"], TOL_BF16, "deep_bf16_full",
          floor=1.0)
    assert np.isfinite(got["loss"])
    assert np.all(got["dWx"][:, wl.H:2 * wl.H] == 0.0)
    for k in ("dWx", "dU", "db", "dWs", "dbs", "dX"):
        assert np.all(np.isfinite(got[k])), k


def test_persistent_level_loop_opt_in(ctx, monkeypatch):
    """The opt-in persistent small-level loop (one cooperative launch with
    grid barriers) gives the same results as per-level launches."""
    monkeypatch.setenv("CAVS_PERSIST", "1")
    _parity(ctx, W.config_treelstm_sst(1, K=16), label="persistent_fp32")
    wl = W.config_treelstm_deep_bf16(1, K=4, D=300, H=1024, lo=8, hi=40)
    _parity_bf16(ctx, wl, "persistent_bf16")
    monkeypatch.delenv("CAVS_PERSIST")


def test_persistent_barrier_timeout_reaches_the_caller(ctx, monkeypatch):
    """The persistent loop's grid barrier is bounded.  With the failure hook
    set to give up at once, every waiting workgroup records the error and the
    kernel still runs to its end (nobody waits); cavs_sync reports it, and
    the next run without the hook is clean."""
    wl = W.config_treelstm_sst(1, K=16)
    monkeypatch.setenv("CAVS_PERSIST", "1")
    monkeypatch.setenv("CAVS_PERSIST_SPIN", "-1")
    b = Batch(wl, ctx)
    with pytest.raises(B.CavsError) as e:
        b.run()
    assert e.value.status == B.ERR_HIP
    assert "grid barrier" in str(e.value)
    monkeypatch.delenv("CAVS_PERSIST_SPIN")
    _parity(ctx, wl, label="persistent_after_timeout")
    monkeypatch.delenv("CAVS_PERSIST")


def test_eager_weight_gradients_ablation(ctx, monkeypatch):
    """The lazy-batching ablation (dU formed level by level and summed into
    the output, CAVS_EAGER_DW=1) gives the oracle's gradients too."""
    monkeypatch.setenv("CAVS_EAGER_DW", "1")
    _parity(ctx, W.config_treelstm_sst(2, K=16), label="eager_dw_fp32")
    rng = np.random.Generator(np.random.PCG64(34))
    trees = [W.random_split_tree(int(L), rng) for L in rng.integers(2, 14, size=420)]
    _parity(ctx, W.make_workload("eager_dw_tiles", trees, N=2, D=32, H=256, C=5, rng=rng,
                                 labels="all"))
    _parity(ctx, W.config_varlstm(1, K=6), label="eager_dw_chains")
    _parity(ctx, W.config_tiny_treelstm(1), label="eager_dw_tiny")
    wl = W.config_treelstm_deep_bf16(2, K=4, D=300, H=1024, lo=8, hi=40)
    _parity_bf16(ctx, wl, "eager_dw_bf16")
    monkeypatch.delenv("CAVS_EAGER_DW")


def test_two_stream_lazy_products_ablation(ctx, monkeypatch):
    """The two-stream variant (dW_x and dX on a second stream beside dU,
    CAVS_TWO_STREAM=1) gives the oracle's gradients; its states and loss are
    the single-stream ones bit for bit (only the backward's lazy phase
    changes streams)."""
    wl = W.config_treelstm_sst(3, K=16)
    base = Batch(wl, ctx).run()
    monkeypatch.setenv("CAVS_TWO_STREAM", "1")
    got = Batch(wl, ctx).run()
    for k in ("h", "c", "loss", "dX"):
        assert np.array_equal(got[k], base[k]), k
    _parity(ctx, wl, label="two_stream_sst")
    _parity(ctx, W.config_varlstm(2, K=6), label="two_stream_chains")
    rng = np.random.Generator(np.random.PCG64(36))
    trees = [W.random_split_tree(int(L), rng) for L in rng.integers(2, 14, size=420)]
    _parity(ctx, W.make_workload("two_stream_tiles", trees, N=2, D=32, H=256, C=5, rng=rng,
                                 labels="all", inputs="all"))
    monkeypatch.delenv("CAVS_TWO_STREAM")


def test_unfused_backward_gates_ablation(ctx, monkeypatch):
    """The fusion ablation (every level's dA from the elementwise kernel,
    CAVS_UNFUSED_BWD_GATES=1) gives the oracle's gradients too."""
    monkeypatch.setenv("CAVS_UNFUSED_BWD_GATES", "1")
    _parity(ctx, W.config_treelstm_sst(0, K=16), label="unfused_fp32")
    _parity(ctx, W.config_varlstm(2, K=6), label="unfused_chains")
    _parity(ctx, W.config_tiny_treelstm(2), label="unfused_tiny")
    wl = W.config_treelstm_deep_bf16(0, K=4, D=300, H=1024, lo=8, hi=40)
    _parity_bf16(ctx, wl, "unfused_bf16")
    monkeypatch.delenv("CAVS_UNFUSED_BWD_GATES")
