"""The XCD-local small-level loop (forced on with CAVS_XCD_LOOP=1, off with
=0; by default taken only at H = 512 with a long suffix of small levels): the levels of at most
256 positions near the roots run in one launch per direction, each XCD
taking the tops of its own trees, with barriers among that XCD's
workgroups only.  Its level products are the per-level split-K tiles (with
the weight columns resident in LDS at H = 512), so the fp32 outputs must
agree with the per-level launches to rounding, and meet the oracle bar.
bf16 levels of 64 positions or more take another split of the contraction
in the per-level launches, so there both sides are held to the oracle.
"""
import numpy as np
import pytest

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


def _cases():
    rng = np.random.Generator(np.random.PCG64(80))
    out = {
        "sst_full": lambda: W.config_treelstm_sst(0),
        "sst_reduced": lambda: W.config_treelstm_sst(1, K=24),
        "chains": lambda: W.config_varlstm(1, K=16),
        "bf16_reduced": lambda: W.config_treelstm_deep_bf16(1, K=8, D=300, H=1024, lo=8, hi=40),
    }
    trees = [W.random_split_tree(int(L), rng) for L in rng.integers(1, 30, size=60)]
    trees += [[[-1, -1], [0, -1], [-1, -1], [1, 2]]] * 9 + [W.chain(1)] * 5
    out["mixed_unary"] = lambda: W.make_workload("mixed_unary", trees, N=2, D=16, H=512, C=5,
                                                 sigma=0.2, rng=rng, labels="all")
    # one tree only: seven of the eight XCDs own no position at any level
    out["one_tree"] = lambda: W.make_workload("one_tree", [W.left_branching_tree(20)], N=2,
                                              D=16, H=512, C=5, sigma=0.2, rng=rng,
                                              labels="all")
    return out


CASES = _cases()


@pytest.mark.parametrize("case", sorted(CASES))
def test_xcd_loop_equals_per_level_launches(ctx, monkeypatch, case):
    wl = CASES[case]()
    print("xcd loop case %s V=%d H=%d" % (case, wl.V, wl.H), flush=True)
    monkeypatch.setenv("CAVS_XCD_LOOP", "0")
    base = Batch(wl, ctx).run()
    monkeypatch.setenv("CAVS_XCD_LOOP", "1")
    got = Batch(wl, ctx).run()
    ctx.sync()
    if wl.prec == W.PREC_BF16:
        # From 64 positions the per-level bf16 products give each workgroup
        # two row tiles and split the contraction over four wavefronts (the
        # loop: one row tile, eight), so their sums round in another order
        # and the bf16 rounding of the states carries that on through the
        # levels.  Both are held to the oracle that rounds the same operands
        # (normwise, as in the bf16 parity tests).
        from parity import check
        want = oracle_sharded(wl, bf16=True)
        check(base, want, ALL_KEYS, 2e-2, "xcd_" + case + "_off", floor=1.0)
        check(got, want, ALL_KEYS, 2e-2, "xcd_" + case + "_on", floor=1.0)
        return
    for k in base:
        a, b = np.asarray(got[k], np.float64), np.asarray(base[k], np.float64)
        scale = max(float(np.max(np.abs(b))), 1e-30)
        assert float(np.max(np.abs(a - b))) <= 1e-5 * scale, (case, k)
    if wl.V < 20000:
        check_fp32(got, oracle_sharded(wl), oracle_sharded(wl, precision="f32"), ALL_KEYS,
                   "xcd_" + case)


def test_xcd_loop_parity_with_oracle(ctx, monkeypatch):
    monkeypatch.setenv("CAVS_XCD_LOOP", "1")
    wl = W.config_treelstm_sst(2, K=32)
    got = Batch(wl, ctx).run()
    ctx.sync()
    check_fp32(got, oracle_sharded(wl), oracle_sharded(wl, precision="f32"), ALL_KEYS,
               "xcd_loop_sst")


def test_xcd_barrier_timeout_reaches_the_caller(ctx, monkeypatch):
    """The XCD loop's barriers are bounded waits.  With the failure hook set
    to give up at once, the workgroups that would wait record the error and
    leave the loop (every later wait sees the flag and ends too); cavs_sync
    reports it, and the next run without the hook is clean."""
    wl = W.config_varlstm(2, K=12)
    monkeypatch.setenv("CAVS_XCD_LOOP", "1")
    monkeypatch.setenv("CAVS_PERSIST_SPIN", "-1")
    print("xcd barrier timeout V=%d" % wl.V, flush=True)
    with pytest.raises(B.CavsError) as e:
        Batch(wl, ctx).run()
    assert e.value.status == B.ERR_HIP
    assert "grid barrier" in str(e.value)
    monkeypatch.delenv("CAVS_PERSIST_SPIN")
    got = Batch(wl, ctx).run()
    ctx.sync()
    check_fp32(got, oracle_sharded(wl), oracle_sharded(wl, precision="f32"), ALL_KEYS,
               "xcd_after_timeout")


def test_xcd_loop_bf16_at_h512(ctx, monkeypatch):
    """bf16 products at H = 512 take the weight-stationary loop with the
    rounded weights in LDS.  Loop on and off, each against the oracle that
    rounds the same operands (normwise through the left-branching half,
    whose deep chains move bf16 rounding points; see the bf16 parity tests)."""
    from parity import check, oracle_sharded as osh
    wl = W.config_treelstm_deep_bf16(3, K=8, D=300, H=512, lo=8, hi=40)
    want = osh(wl, bf16=True)
    for mode in ("1", "0"):
        monkeypatch.setenv("CAVS_XCD_LOOP", mode)
        print("xcd loop bf16 H=512 V=%d mode %s" % (wl.V, mode), flush=True)
        got = Batch(wl, ctx).run()
        ctx.sync()
        check(got, want, ALL_KEYS, 2e-2, "xcd_bf16_h512_" + mode, floor=1.0)
