"""Device-side driver for one batch: uploads a workload, schedules it and runs
forward + backward through the C ABI.  Used by the tests, the smoke check and
the benchmark; it only allocates tensors and calls the binding."""
from __future__ import annotations

from typing import Optional

import numpy as np
import torch

from . import binding as B
from .workloads import Workload


class Batch:
    def __init__(self, wl: Workload, ctx: Optional[B.Context] = None, device: int = 0):
        self.wl = wl
        self.ctx = ctx if ctx is not None else B.Context(device)
        dev = self.ctx.torch_device
        self.dev = dev

        def i32(a):
            return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(dev)

        def f32(a):
            if a is None or a.size == 0:
                return None
            return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev)

        self.child = i32(wl.child.reshape(wl.V, wl.N))
        # graph inputs pass no parent array
        self.parent = None if getattr(wl, "dag", False) else i32(wl.parent)
        self.pull_idx = i32(wl.pull_idx)
        self.push_idx = i32(wl.push_idx)
        self.X = f32(wl.X)
        self.Y = f32(wl.Y) if wl.loss == B.LOSS_L2 else None
        self.params = B.Params(cell=wl.cell, prec=wl.prec, loss=wl.loss, D=wl.D, H=wl.H, N=wl.N,
                               C=wl.C if wl.loss == B.LOSS_CE else 0,
                               Wx=f32(wl.Wx) if wl.cell == B.TREE_LSTM else None,
                               U=f32(wl.U), b=f32(wl.b),
                               Ws=f32(wl.Ws) if wl.loss == B.LOSS_CE else None,
                               bs=f32(wl.bs) if wl.loss == B.LOSS_CE else None)
        self.dH_ext: Optional[torch.Tensor] = None   # [V, H] external gradient of h_out
        self.sched: Optional[B.Schedule] = None
        self.ws = None
        self.ws_infer = None

    def schedule(self) -> B.Schedule:
        """cavs_schedule; reuses the schedule buffers from an earlier call."""
        wl = self.wl
        if self.sched is None:
            self.sched = B.alloc_schedule(self.ctx, wl.V, wl.N, wl.n_x)
        B.run_schedule(self.ctx, self.sched, self.child, self.parent, self.pull_idx,
                       self.push_idx, n_x=wl.n_x, n_push=wl.n_push)
        return self.sched

    def alloc(self):
        wl, dev = self.wl, self.dev
        nbytes = B.workspace_bytes(self.params, self.sched)
        self.ws = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=dev)
        f = dict(dtype=torch.float32, device=dev)
        self.h = torch.empty(wl.V, wl.H, **f)
        self.c = torch.empty(wl.V, wl.H, **f) if wl.cell == B.TREE_LSTM else None
        self.loss = torch.empty(1, **f)
        H, D, C = wl.H, wl.D, wl.C
        g = {}
        if wl.cell == B.TREE_LSTM:
            g["dWx"] = torch.empty(D, 4 * H, **f)
            g["dU"] = torch.empty(H, 4 * H, **f)
            g["db"] = torch.empty(4 * H, **f)
        else:
            g["dU"] = torch.empty(wl.N * H, H, **f)
            g["db"] = torch.empty(H, **f)
        if wl.loss == B.LOSS_CE:
            g["dWs"] = torch.empty(H, C, **f)
            g["dbs"] = torch.empty(C, **f)
        g["dX"] = torch.empty(max(wl.n_x, 0), D, **f)
        self.grads = g

    def forward(self):
        B.forward(self.ctx, self.params, self.sched, self.X, self.Y, self.ws, self.h, self.c,
                  self.loss)

    def backward(self):
        B.backward(self.ctx, self.params, self.sched, self.X, self.Y, self.ws, self.grads,
                   self.dH_ext)

    def infer(self):
        """cavs_infer into the same h / c / loss outputs, with its own smaller workspace."""
        if self.ws_infer is None:
            nbytes = B.infer_workspace_bytes(self.params, self.sched)
            self.ws_infer = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=self.dev)
        B.infer(self.ctx, self.params, self.sched, self.X, self.Y, self.ws_infer, self.h,
                self.c, self.loss)

    def run_infer(self) -> dict:
        """Schedule (if needed), cavs_infer, and the outputs as float64 numpy arrays."""
        if self.sched is None:
            self.schedule()
        if self.ws is None:
            self.alloc()
        self.infer()
        self.ctx.sync()
        return self.results(backward=False)

    def step(self):
        """One pass of the whole path: schedule, forward, backward (async tail)."""
        self.schedule()
        self.forward()
        self.backward()

    def run(self, backward: bool = True) -> dict:
        if self.sched is None:
            self.schedule()
        if self.ws is None:
            self.alloc()
        self.forward()
        if backward:
            self.backward()
        self.ctx.sync()
        return self.results(backward)

    def results(self, backward: bool = True) -> dict:
        r = dict(h=self.h.double().cpu().numpy(), loss=float(self.loss.item()))
        if self.c is not None:
            r["c"] = self.c.double().cpu().numpy()
        if backward:
            for k, v in self.grads.items():
                r[k] = v.double().cpu().numpy()
        return r
