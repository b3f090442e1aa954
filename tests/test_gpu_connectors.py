"""GPU parity of the external connectors (push/pull to operators outside the
vertex function, Section 3.1; the multi-layer and LM models of Section 5),
through the C ABI, against the same compositions of the oracle.

* Stacked layers: layer 2 pulls layer 1's pushed states (its h_out, on the
  device, no copy) as inputs; layer 1 has no loss head and receives layer
  2's input gradient as the external gradient of its pushed states.
* Encoder-decoder: a Tree-LSTM encoder whose roots feed the first vertex of
  chain decoders, with a 40-class softmax at every decoder vertex (the
  large-vocabulary head).
* A Var-LSTM language model: a 4096-word softmax at every vertex.
fp32 outputs meet parity.check_fp32 (oracle fp64 and fp32 builds composed
the same way).
"""
import numpy as np
import pytest
import torch

import oracle
from parity import check_fp32
from paper_1712_04048_amd import binding as B
from paper_1712_04048_amd import workloads as W
from paper_1712_04048_amd.runner import Batch

pytestmark = pytest.mark.gpu

KEYS = ["h", "c", "loss", "dWx", "dU", "db", "dWs", "dbs", "dX"]


@pytest.fixture(scope="module")
def ctx():
    c = B.Context(0)
    yield c
    c.close()


def _oracle_stack(l1, l2, rows2, precision):
    """Oracle composition: forward 1, inputs of 2 = the pushed states of the
    vertices listed by rows2 (row r of X2 = h1[rows2[r]]), forward + backward
    2, backward 1 with the gradient sent back through the connector."""
    r1 = oracle.run(l1, backward=False, precision=precision)
    X2 = r1["h"][rows2]
    r2 = oracle.run(l2, X=X2, precision=precision)
    ext = np.zeros_like(r1["h"])
    np.add.at(ext, rows2, r2["dX"])
    r1b = oracle.run(l1, dH_ext=ext, precision=precision)
    return r1b, r2


def _gpu_stack(ctx, l1, l2, rows2):
    b1 = Batch(l1, ctx)
    b1.schedule()
    b1.alloc()
    b1.forward()
    b2 = Batch(l2, ctx)
    rows = torch.from_numpy(np.asarray(rows2, dtype=np.int64)).to(ctx.torch_device)
    b2.X = b1.h.index_select(0, rows).contiguous()
    got2 = b2.run()
    ext = torch.zeros_like(b1.h)
    ext.index_add_(0, rows, b2.grads["dX"])
    b1.dH_ext = ext
    b1.backward()
    ctx.sync()
    return b1.results(), got2


def _check(got, ref64, ref32, label):
    return check_fp32(got, ref64, ref32, [k for k in KEYS if k in ref64], label)


def test_stacked_two_layer_lstm(ctx):
    rng = np.random.Generator(np.random.PCG64(70))
    trees = [W.chain(int(n)) for n in rng.integers(5, 40, size=16)]
    l1 = W.make_workload("layer1", trees, N=1, D=64, H=256, loss=W.LOSS_NONE, sigma=0.1,
                         rng=rng, inputs="all")
    l2 = W.make_workload("layer2", trees, N=1, D=256, H=256, C=5, sigma=0.1, rng=rng,
                         inputs="all", labels="all")
    rows2 = np.argsort(l2.pull_idx)          # row r of X2 = h1 of the vertex pulling row r
    assert np.array_equal(l2.pull_idx[rows2], np.arange(l2.n_x))
    g1, g2 = _gpu_stack(ctx, l1, l2, rows2)
    a64, b64 = _oracle_stack(l1, l2, rows2, "f64")
    a32, b32 = _oracle_stack(l1, l2, rows2, "f32")
    _check(g2, b64, b32, "stack_layer2")
    _check(g1, a64, a32, "stack_layer1")


def test_tree_encoder_chain_decoder_large_vocab(ctx):
    rng = np.random.Generator(np.random.PCG64(71))
    K = 12
    enc = W.make_workload("encoder", [W.random_split_tree(int(L), rng)
                                      for L in rng.integers(2, 20, size=K)],
                          N=2, D=32, H=128, loss=W.LOSS_NONE, sigma=0.2, rng=rng)
    dec = W.make_workload("decoder", [W.chain(int(n)) for n in rng.integers(3, 15, size=K)],
                          N=1, D=128, H=128, C=40, sigma=0.2, rng=rng, inputs="none",
                          labels="all")
    # the first vertex of decoder k pulls the root state of encoder k
    first = np.array([int(dec.tree_offsets[k]) for k in range(K)])
    dec.pull_idx[first] = np.arange(K, dtype=np.int32)
    dec.X = np.zeros((K, 128), dtype=np.float32)
    roots = np.array([int(enc.tree_offsets[k + 1]) - 1 for k in range(K)])
    assert np.all(enc.parent[roots] < 0)
    g1, g2 = _gpu_stack(ctx, enc, dec, roots)
    a64, b64 = _oracle_stack(enc, dec, roots, "f64")
    a32, b32 = _oracle_stack(enc, dec, roots, "f32")
    _check(g2, b64, b32, "decoder_c40")
    _check(g1, a64, a32, "encoder")


def test_varlstm_language_model_softmax(ctx):
    rng = np.random.Generator(np.random.PCG64(72))
    wl = W.make_workload("lm_c4096", [W.chain(int(n)) for n in rng.integers(10, 60, size=6)],
                         N=1, D=64, H=256, C=4096, sigma=0.05, rng=rng, inputs="all",
                         labels="all")
    got = Batch(wl, ctx).run()
    _check(got, oracle.run(wl), oracle.run(wl, precision="f32"), "varlstm_lm_c4096")
    b = Batch(wl, ctx)
    train = b.run(backward=False)
    b.loss.fill_(float("nan"))
    assert b.run_infer()["loss"] == train["loss"]


def test_no_loss_head_with_external_gradient_only(ctx):
    rng = np.random.Generator(np.random.PCG64(73))
    trees = [W.random_split_tree(int(L), rng) for L in rng.integers(1, 20, size=20)]
    wl = W.make_workload("ext_only", trees, N=2, D=16, H=128, loss=W.LOSS_NONE, sigma=0.2,
                         rng=rng, inputs="all")
    G = (0.01 * rng.standard_normal((wl.V, wl.H))).astype(np.float32)
    b = Batch(wl, ctx)
    b.schedule()
    b.alloc()
    b.dH_ext = torch.from_numpy(G).to(ctx.torch_device)
    got = b.run()
    assert got["loss"] == 0.0
    _check(got, oracle.run(wl, dH_ext=G), oracle.run(wl, dH_ext=G, precision="f32"),
           "ext_only")
    # and without it every gradient is zero
    b.dH_ext = None
    got0 = b.run()
    for k in ("dWx", "dU", "db", "dX"):
        assert np.all(got0[k] == 0.0), k


def test_large_vocab_head_refuses_unaligned_class_count(ctx):
    rng = np.random.Generator(np.random.PCG64(74))
    wl = W.make_workload("c41", [W.chain(5)], N=1, D=8, H=64, C=41, rng=rng, inputs="all",
                         labels="all")
    with pytest.raises(B.CavsError) as e:
        Batch(wl, ctx).run()
    assert e.value.status == B.ERR_UNSUPPORTED
