"""Host-side logic of bench.py (no GPU): the one-GPU guard and the
algorithmic-FLOP bookkeeping behind the roofline entry."""
import os
import subprocess
import sys

import numpy as np

import bench
import oracle
from paper_1712_04048_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=60)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_step_flops_match_the_closed_form():
    """Summed over one step's launches (forward and backward level products,
    the pull, dX and the three lazy products), the per-launch costs give
    30 H^2 per binary internal vertex plus 18 D H per pulled leaf: three times
    the forward's 10 H^2 and 6 D H."""
    wl = W.config_treelstm_sst(0, K=24)
    s = oracle.schedule(wl.child, wl.parent, wl.pull_idx, wl.push_idx)
    nc = (s["child_pos"] >= 0).sum(axis=1)
    lo = s["level_offsets"]
    n_pull = int((wl.pull_idx >= 0).sum())
    names = ["k_pull_tile<3, 64, 2>", "k_dx_tile<32, 64, 3>", "k_tn_dl<LdDUiou, 128, 256, 2>",
             "k_tn_dl<LdDUf, 128, 128, 4>", "k_tn_dl<LdDWx, 64, 256, 3>"]
    total = sum(bench.launch_cost(wl, nc, k, 0, wl.V, n_pull, False)[0] for k in names)
    for t in range(1, len(lo) - 1):
        rows = int(lo[t + 1] - lo[t])
        for k in ("k_lstm_fwd_tile<2, false, 32, 32, 2>", "k_lstm_bwd_level_sk<2, false, 1, 8>"):
            total += bench.launch_cost(wl, nc, k, int(lo[t]), rows, n_pull, False)[0]
    v_int = int((nc > 0).sum())
    assert np.all(nc[nc > 0] == 2) and n_pull == wl.V - v_int
    H, D = wl.H, wl.D
    assert total == 30.0 * H * H * v_int + 18.0 * D * H * n_pull


def test_grouped_and_loop_launches_cost_what_their_parts_do():
    """The grouped lazy launch (dU_f with dW_x) costs the sum of the two
    products, and the XCD loop kernels cost what per-level launches over the
    same rows would."""
    wl = W.config_treelstm_sst(0, K=24)
    s = oracle.schedule(wl.child, wl.parent, wl.pull_idx, wl.push_idx)
    nc = (s["child_pos"] >= 0).sum(axis=1)
    lo = s["level_offsets"]
    n_pull = int((wl.pull_idx >= 0).sum())
    cost = lambda k, r0=0, r=wl.V: bench.launch_cost(wl, nc, k, r0, r, n_pull, False)[0]
    assert cost("k_tn_group<dUf, dWx64>") == (cost("k_tn_dl<LdDUf, 128, 128, 4>") +
                                              cost("k_tn_dl<LdDWx, 64, 256, 3>")) > 0
    t0 = len(lo) - 4
    per_level = sum(cost("k_lstm_fwd_level_sk<2, false, 1, 8>", int(lo[t]), int(lo[t + 1] - lo[t]))
                    for t in range(t0, len(lo) - 1))
    assert cost("k_lstm_fwd_xcd_ws<2, false, 8>", int(lo[t0]), wl.V - int(lo[t0])) == per_level > 0
    assert cost("k_lstm_bwd_xcd_ws<2, false, 8>", int(lo[t0]), wl.V - int(lo[t0])) == per_level
