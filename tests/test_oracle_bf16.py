"""Pin of the oracle's bf16 emulation: which operands it rounds.

The bf16 path rounds the operands of every matrix product to bf16 (nearest
even) and accumulates the rest exactly (the reading of the bf16 MFMA configs:
forward x, W_x, h~ = sum_k h_k, h_k and U; backward the pre-activation
gradients with U and W_x; the lazy products h~, h_k, x and the gradients),
while states, gates, the loss head and the bias sums stay unrounded.

Here the same models are written independently in torch fp64: the forward per
vertex in topological order, the backward by autograd.  Every matrix product
goes through one autograd function whose forward multiplies bf16-rounded
operands and whose backward multiplies bf16-rounded incoming gradients by
bf16-rounded operands -- the rounding rule stated once, applied by autograd
at every product of both passes (the rounding helper itself is checked
against torch's float32 -> bfloat16 conversion).  A rounding point missing or added on either side (for example h~
rounded per child before the sum, or the summed forget-gate gradient of W_x
rounded per child) moves results by about 2^-9 relative; the comparison
holds to 1e-12.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_1712_04048_amd import workloads as W


def _rb(t):
    """fp64 -> nearest bf16 (8 significant bits, ties to even), directly:
    a detour through float32 could round twice.  The helper agrees with
    torch's float32 -> bfloat16 conversion on float32 inputs (checked in
    test_rb_matches_torch_conversion)."""
    m, e = torch.frexp(t)
    return torch.ldexp(torch.round(m * 256.0) / 256.0, e)


def test_rb_matches_torch_conversion():
    rng = np.random.Generator(np.random.PCG64(44))
    x = torch.from_numpy((rng.standard_normal(5000) * 10.0 ** rng.integers(-5, 5, 5000))
                         .astype(np.float32))
    x = torch.cat([x, torch.tensor([1 + 2 ** -8, 1 + 3 * 2 ** -8, -(1 + 2 ** -8), 0.0])])
    assert torch.equal(_rb(x.double()), x.to(torch.bfloat16).double())


class _BfMatmul(torch.autograd.Function):
    @staticmethod
    def forward(ctx, a, b):
        ctx.save_for_backward(a, b)
        return _rb(a) @ _rb(b)

    @staticmethod
    def backward(ctx, g):
        a, b = ctx.saved_tensors
        return _rb(g) @ _rb(b).T, _rb(a).T @ _rb(g)


def _mm(a, b):
    return _BfMatmul.apply(a.reshape(1, -1), b).reshape(-1)


def _topo(wl):
    order, seen = [], set()

    def visit(v):
        if v in seen:
            return
        seen.add(v)
        for c in wl.child[v]:
            if c >= 0:
                visit(int(c))
        order.append(v)

    for v in range(wl.V):
        visit(v)
    return order


def _torch_treelstm(wl):
    H, D = wl.H, wl.D
    t = lambda a: torch.from_numpy(np.asarray(a, dtype=np.float64)).requires_grad_(True)
    Wx, U, b, Ws, bs, X = t(wl.Wx), t(wl.U), t(wl.b), t(wl.Ws), t(wl.bs), t(wl.X)
    h, c = {}, {}
    for v in _topo(wl):
        kids = [int(k) for k in wl.child[v] if k >= 0]
        row = int(wl.pull_idx[v])
        xw = b + (_mm(X[row], Wx) if row >= 0 else 0.0)
        a = xw.clone() if not kids else None
        if kids:
            hs = sum(h[k] for k in kids)
            U_iou = torch.cat([U[:, 0:H], U[:, 2 * H:4 * H]], dim=1)
            a_iou = torch.cat([xw[0:H], xw[2 * H:4 * H]]) + _mm(hs, U_iou)
            i, o, u = torch.sigmoid(a_iou[:H]), torch.sigmoid(a_iou[H:2 * H]), torch.tanh(a_iou[2 * H:])
            cv = i * u
            for k in kids:
                f = torch.sigmoid(xw[H:2 * H] + _mm(h[k], U[:, H:2 * H]))
                cv = cv + f * c[k]
        else:
            i, o, u = torch.sigmoid(a[:H]), torch.sigmoid(a[2 * H:3 * H]), torch.tanh(a[3 * H:])
            cv = i * u
        c[v] = cv
        h[v] = o * torch.tanh(cv)
    lab = wl.push_idx
    sel = [v for v in range(wl.V) if lab[v] >= 0]
    Hm = torch.stack([h[v] for v in sel])
    z = Hm @ Ws + bs
    loss = torch.nn.functional.cross_entropy(z, torch.tensor(lab[sel].astype(np.int64)))
    loss.backward()
    res = dict(h=np.stack([h[v].detach().numpy() for v in range(wl.V)]),
               c=np.stack([c[v].detach().numpy() for v in range(wl.V)]), loss=loss.item(),
               dWx=Wx.grad.numpy(), dU=U.grad.numpy(), db=b.grad.numpy(), dWs=Ws.grad.numpy(),
               dbs=bs.grad.numpy(), dX=X.grad.numpy())
    return res


def _torch_treefc(wl):
    H = wl.H
    t = lambda a: torch.from_numpy(np.asarray(a, dtype=np.float64)).requires_grad_(True)
    Wt, b, X, Y = t(wl.U), t(wl.b), t(wl.X), torch.from_numpy(wl.Y.astype(np.float64))
    h = {}
    for v in _topo(wl):
        kids = [(k, int(c)) for k, c in enumerate(wl.child[v]) if c >= 0]
        if not kids:
            h[v] = X[int(wl.pull_idx[v])]
            continue
        z = b
        for k, cidx in kids:
            z = z + _mm(h[cidx], Wt[k * H:(k + 1) * H])
        h[v] = torch.tanh(z)
    sel = [v for v in range(wl.V) if wl.push_idx[v] >= 0]
    loss = sum(0.5 * ((h[v] - Y[int(wl.push_idx[v])]) ** 2).sum() for v in sel) / len(sel)
    loss.backward()
    return dict(h=np.stack([h[v].detach().numpy() for v in range(wl.V)]), loss=loss.item(),
                dU=Wt.grad.numpy(), db=b.grad.numpy(), dX=X.grad.numpy())


def _compare(got, want):
    for k, ref in want.items():
        if k == "loss":
            assert abs(got[k] - ref) <= 1e-12 * abs(ref), k
            continue
        scale = max(np.abs(ref).max(), 1e-300)
        err = np.abs(got[k] - ref).max() / scale
        assert err <= 1e-12, (k, err)


@pytest.mark.parametrize("inputs", ["leaves", "all"])
def test_bf16_rounding_points_treelstm(inputs):
    rng = np.random.Generator(np.random.PCG64(40 + (inputs == "all")))
    trees = [W.random_split_tree(L, rng) for L in (1, 2, 3, 6)] + [W.left_branching_tree(4)]
    trees.append([[-1, -1], [0, -1]])   # a unary vertex (slot 1 empty)
    wl = W.make_workload("bf16pin", trees, prec=W.PREC_BF16, N=2, D=5, H=6, C=4, sigma=0.5,
                         rng=rng, inputs=inputs, labels="all")
    wl.b[:] = (0.3 * rng.standard_normal(wl.b.shape)).astype(np.float32)
    got = oracle.run(wl, bf16=True)
    want = _torch_treelstm(wl)
    _compare(got, want)
    # and the rounding is visible: the plain fp64 oracle differs well above 1e-12
    plain = oracle.run(wl, bf16=False)
    assert np.abs(plain["dU"] - got["dU"]).max() > 1e-6 * np.abs(got["dU"]).max()


def test_bf16_rounding_points_chain():
    rng = np.random.Generator(np.random.PCG64(42))
    wl = W.make_workload("bf16chain", [W.chain(5), W.chain(1), W.chain(3)], prec=W.PREC_BF16,
                         N=1, D=4, H=5, C=3, sigma=0.5, rng=rng, inputs="all", labels="all")
    _compare(oracle.run(wl, bf16=True), _torch_treelstm(wl))


def test_bf16_rounding_points_treefc():
    rng = np.random.Generator(np.random.PCG64(43))
    trees = [W.random_split_tree(5, rng), W.complete_tree(4)]
    wl = W.make_workload("bf16fc", trees, cell=W.CELL_TREE_FC, loss=W.LOSS_L2, N=2, H=6,
                         sigma=0.5, rng=rng, labels="all")
    wl.b[:] = (0.3 * rng.standard_normal(wl.b.shape)).astype(np.float32)
    _compare(oracle.run(wl, bf16=True), _torch_treefc(wl))
