"""cavs_schedule_static, the entry point for callers that cannot allocate:
through the C ABI, its schedule must equal cavs_schedule's bit for bit, on
two calls in a row that share the library's static scratch -- a batch that
takes the multi-launch scheduler (more than 16384 vertices), then a smaller
one that takes the one-workgroup scheduler -- and a forward + backward on
the static schedule must equal one on the workspace schedule.  A batch too
large for the static array is refused on the host."""
import numpy as np
import pytest
import torch

from paper_1712_04048_amd import binding as B
from paper_1712_04048_amd import workloads as W
from paper_1712_04048_amd.runner import Batch

pytestmark = pytest.mark.gpu


def _forest(seed, n_trees, lo, hi):
    rng = np.random.Generator(np.random.PCG64(seed))
    trees = [W.random_split_tree(int(L), rng) for L in rng.integers(lo, hi, size=n_trees)]
    return W.make_workload("static%d" % seed, trees, N=2, D=8, H=64, C=5, rng=rng,
                           labels="all", shuffle_ids=True)


def _both(ctx, wl):
    dev = ctx.torch_device
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(dev)
    args = (t(wl.child), t(wl.parent), t(wl.pull_idx), t(wl.push_idx))
    kw = dict(n_x=wl.n_x, n_push=wl.n_push)
    ref = B.alloc_schedule(ctx, wl.V, wl.N, wl.n_x)
    B.run_schedule(ctx, ref, *args, **kw)
    got = B.alloc_schedule(ctx, wl.V, wl.N, wl.n_x)
    for v in got.tensors.values():
        v.fill_(-7)
    B.run_schedule_static(ctx, got, *args, **kw)
    a, b = ref.host(), got.host()
    assert a["T"] == b["T"]
    for k in a:
        assert np.array_equal(np.asarray(a[k]), np.asarray(b[k])), k


def test_static_schedule_equals_workspace_schedule():
    ctx = B.Context(0)
    try:
        big = _forest(1, 700, 2, 50)
        assert 16384 < big.V and B.lib().cavs_schedule_workspace_bytes(
            big.V, 2, big.n_x) <= B.SCHEDULE_STATIC_BYTES
        print("static schedule V=%d" % big.V, flush=True)
        _both(ctx, big)
        small = _forest(2, 40, 2, 30)
        print("static schedule V=%d" % small.V, flush=True)
        _both(ctx, small)
        # the static schedule drives a forward + backward like the other
        b1, b2 = Batch(small, ctx), Batch(small, ctx)
        b1.schedule()
        b2.sched = B.alloc_schedule(ctx, small.V, small.N, small.n_x)
        B.run_schedule_static(ctx, b2.sched, b2.child, b2.parent, b2.pull_idx, b2.push_idx,
                              n_x=small.n_x, n_push=small.n_push)
        r1, r2 = b1.run(), b2.run()
        for k in r1:
            assert np.array_equal(np.asarray(r1[k]), np.asarray(r2[k])), k
    finally:
        ctx.close()


def test_static_schedule_refuses_what_does_not_fit():
    ctx = B.Context(0)
    try:
        V = 200000
        assert B.lib().cavs_schedule_workspace_bytes(V, 2, V) > B.SCHEDULE_STATIC_BYTES
        dev = ctx.torch_device
        child = torch.full((V, 2), -1, dtype=torch.int32, device=dev)
        parent = torch.full((V,), -1, dtype=torch.int32, device=dev)
        pull = torch.arange(V, dtype=torch.int32, device=dev)
        s = B.alloc_schedule(ctx, V, 2, V)
        with pytest.raises(B.CavsError) as e:
            B.run_schedule_static(ctx, s, child, parent, pull, None, n_x=V, n_push=0)
        assert e.value.status == B.ERR_WORKSPACE
        assert "static" in str(e.value)
    finally:
        ctx.close()
