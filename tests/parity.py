"""Helpers shared by the GPU parity tests (no method arithmetic here)."""
import numpy as np

from paper_1712_04048_amd import workloads as W


FLOOR = 0.1


def rel_err(got, ref, floor=FLOOR):
    """Per-tensor max relative error with a floor:
    max_i |g_i - o_i| / max(|o_i|, floor * max|o|).

    Elements at or above floor * max|o| are held to a pure relative error;
    smaller ones to an absolute error of tol * floor * max|o|.  The floor is
    needed because fp32 rounding error scales with the magnitude of a whole
    dot product (about sqrt(K) * 2^-24 of its terms for length K), not with
    each output element, and compounds level by level.
    """
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    if ref.size == 0:
        return 0.0
    scale = np.abs(ref).max()
    if scale == 0.0:
        return float(np.abs(got).max())
    den = np.maximum(np.abs(ref), floor * scale)
    return float((np.abs(got - ref) / den).max())


def normwise_err(got, ref):
    """max |g - o| / max |o| (reported alongside)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    scale = np.abs(ref).max() if ref.size else 0.0
    if scale == 0.0:
        return float(np.abs(got).max()) if got.size else 0.0
    return float(np.abs(got - ref).max() / scale)


def check(gpu: dict, ref: dict, keys, tol, label="", floor=FLOOR):
    """Fails if any tensor's rel_err (with the given floor) exceeds tol.
    floor=1.0 makes the test normwise: max |g - o| / max |o|."""
    errs = {}
    for k in keys:
        if k not in ref:
            continue
        if k == "loss":
            errs[k] = abs(gpu[k] - ref[k]) / max(abs(ref[k]), 1e-30)
        else:
            errs[k] = rel_err(gpu[k], ref[k], floor)
    bad = {k: v for k, v in errs.items() if not v <= tol}
    assert not bad, "%s: errors above %g: %s (all: %s)" % (label, tol, bad, errs)
    return errs


def subset(wl: W.Workload, trees) -> W.Workload:
    """The workload restricted to the given graphs (ids renumbered in order;
    X / Y rows restricted to the rows those graphs use)."""
    keep = np.concatenate([np.arange(wl.tree_offsets[k], wl.tree_offsets[k + 1]) for k in trees])
    newid = -np.ones(wl.V, dtype=np.int64)
    newid[keep] = np.arange(keep.size)
    child = wl.child[keep]
    child = np.where(child >= 0, newid[np.maximum(child, 0)], -1).astype(np.int32)
    parent = wl.parent[keep]
    parent = np.where(parent >= 0, newid[np.maximum(parent, 0)], -1).astype(np.int32)
    pull = wl.pull_idx[keep]
    rows = pull[pull >= 0]
    newrow = -np.ones(max(wl.n_x, 1), dtype=np.int64)
    newrow[rows] = np.arange(rows.size)
    pull = np.where(pull >= 0, newrow[np.maximum(pull, 0)], -1).astype(np.int32)
    push = wl.push_idx[keep].copy()
    Y = wl.Y
    if wl.loss == W.LOSS_L2:
        yrows = push[push >= 0]
        newy = -np.ones(max(wl.n_y, 1), dtype=np.int64)
        newy[yrows] = np.arange(yrows.size)
        push = np.where(push >= 0, newy[np.maximum(push, 0)], -1).astype(np.int32)
        Y = wl.Y[yrows]
    sizes = [wl.tree_offsets[k + 1] - wl.tree_offsets[k] for k in trees]
    offs = np.zeros(len(trees) + 1, dtype=np.int64)
    offs[1:] = np.cumsum(sizes)
    return W.Workload(name=wl.name + "_subset", cell=wl.cell, prec=wl.prec, loss=wl.loss,
                      N=wl.N, D=wl.D, H=wl.H, C=wl.C, child=child, parent=parent,
                      pull_idx=pull, push_idx=push, X=wl.X[rows], Y=Y, Wx=wl.Wx, U=wl.U,
                      b=wl.b, Ws=wl.Ws, bs=wl.bs, tree_offsets=offs)
