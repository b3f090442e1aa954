"""Thin ctypes binding of libcavs.so (see include/cavs.h).

Argument marshalling only: every step of the schedule, forward and backward
runs in the library's HIP kernels.  PyTorch supplies device memory and the
stream.  The library must be built (``python -m paper_1712_04048_amd.build``);
loading fails loudly otherwise -- there is no fallback path.
"""
from __future__ import annotations

import ctypes as ct
import os
from dataclasses import dataclass
from typing import Optional

import numpy as np
import torch

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libcavs.so")

OK = 0
ERR_ARG = -1
ERR_RANGE = -2
ERR_MULTIPARENT = -3
ERR_CYCLE = -4
ERR_MISMATCH = -5
ERR_WORKSPACE = -6
ERR_HIP = -7
ERR_UNSUPPORTED = -8
ERR_DUP_PULL = -9

TREE_LSTM = 0
TREE_FC = 1
FP32 = 0
BF16 = 1
LOSS_CE = 0
LOSS_L2 = 1
LOSS_NONE = 2

_i32 = ct.c_int32
_vp = ct.c_void_p


class cavs_graphs(ct.Structure):
    _fields_ = [("V", _i32), ("N", _i32), ("n_x", _i32), ("n_push", _i32),
                ("child", _vp), ("parent", _vp), ("pull_idx", _vp), ("push_idx", _vp)]


class cavs_sched(ct.Structure):
    _fields_ = [("T", _i32), ("V", _i32), ("N", _i32), ("n_x", _i32), ("n_push", _i32),
                ("n_pull", _i32), ("n_labelled", _i32), ("n_leaf_noinput", _i32),
                ("n_inner_input", _i32),
                ("level", _vp), ("order", _vp), ("pos", _vp), ("child_pos", _vp),
                ("parent_pos", _vp), ("pull_pos", _vp), ("push_pos", _vp), ("pull_list", _vp),
                ("level_offsets", _vp), ("level_offsets_host", _vp), ("dag", _i32),
                ("in_offsets", _vp), ("in_edges", _vp)]


class cavs_params(ct.Structure):
    _fields_ = [("cell", _i32), ("prec", _i32), ("loss", _i32), ("D", _i32), ("H", _i32),
                ("N", _i32), ("C", _i32),
                ("Wx", _vp), ("U", _vp), ("b", _vp), ("Ws", _vp), ("bs", _vp)]


class cavs_inputs(ct.Structure):
    _fields_ = [("X", _vp), ("Y", _vp), ("n_y", _i32), ("dH_ext", _vp)]


class cavs_grads(ct.Structure):
    _fields_ = [("dWx", _vp), ("dU", _vp), ("db", _vp), ("dWs", _vp), ("dbs", _vp), ("dX", _vp)]


class cavs_launch_time(ct.Structure):
    _fields_ = [("name", ct.c_char * 96), ("row0", _i32), ("rows", _i32), ("ms", ct.c_double)]


EXPORTS = ["cavs_create", "cavs_set_stream", "cavs_destroy", "cavs_last_error", "cavs_sync",
           "cavs_schedule_workspace_bytes", "cavs_schedule", "cavs_schedule_static",
           "cavs_workspace_bytes",
           "cavs_forward", "cavs_backward", "cavs_infer_workspace_bytes", "cavs_infer",
           "cavs_timing_enable", "cavs_timing_read"]

_lib = None


def lib():
    """Loads libcavs.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libcavs.so is not built: run `python -m paper_1712_04048_amd.build`")
        L = ct.CDLL(LIB_PATH)
        L.cavs_create.restype = _i32
        L.cavs_create.argtypes = [ct.POINTER(_vp), _i32, _vp]
        L.cavs_set_stream.restype = _i32
        L.cavs_set_stream.argtypes = [_vp, _vp]
        L.cavs_destroy.restype = None
        L.cavs_destroy.argtypes = [_vp]
        L.cavs_last_error.restype = ct.c_char_p
        L.cavs_last_error.argtypes = [_vp]
        L.cavs_sync.restype = _i32
        L.cavs_sync.argtypes = [_vp]
        L.cavs_schedule_workspace_bytes.restype = ct.c_size_t
        L.cavs_schedule_workspace_bytes.argtypes = [_i32, _i32, _i32]
        L.cavs_schedule.restype = _i32
        L.cavs_schedule.argtypes = [_vp, ct.POINTER(cavs_graphs), ct.POINTER(cavs_sched), _vp,
                                    ct.c_size_t]
        L.cavs_schedule_static.restype = _i32
        L.cavs_schedule_static.argtypes = [_vp, ct.POINTER(cavs_graphs), ct.POINTER(cavs_sched)]
        L.cavs_workspace_bytes.restype = ct.c_size_t
        L.cavs_workspace_bytes.argtypes = [ct.POINTER(cavs_params), ct.POINTER(cavs_sched)]
        L.cavs_forward.restype = _i32
        L.cavs_forward.argtypes = [_vp, ct.POINTER(cavs_params), ct.POINTER(cavs_sched),
                                   ct.POINTER(cavs_inputs), _vp, _vp, _vp, _vp, ct.c_size_t]
        L.cavs_backward.restype = _i32
        L.cavs_backward.argtypes = [_vp, ct.POINTER(cavs_params), ct.POINTER(cavs_sched),
                                    ct.POINTER(cavs_inputs), _vp, ct.c_size_t,
                                    ct.POINTER(cavs_grads)]
        L.cavs_infer_workspace_bytes.restype = ct.c_size_t
        L.cavs_infer_workspace_bytes.argtypes = [ct.POINTER(cavs_params), ct.POINTER(cavs_sched)]
        L.cavs_infer.restype = _i32
        L.cavs_infer.argtypes = L.cavs_forward.argtypes
        L.cavs_timing_enable.restype = _i32
        L.cavs_timing_enable.argtypes = [_vp, _i32]
        L.cavs_timing_read.restype = _i32
        L.cavs_timing_read.argtypes = [_vp, ct.POINTER(cavs_launch_time), _i32]
        _lib = L
    return _lib


class CavsError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__("cavs status %d: %s" % (status, msg))
        self.status = status


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    if t is None:
        return None
    assert t.is_contiguous()
    return t.data_ptr()


class Context:
    """A library context bound to one device and the current torch stream."""

    def __init__(self, device: int = 0, stream: Optional[torch.cuda.Stream] = None):
        self.device = device
        self.torch_device = torch.device("cuda", device)
        s = stream if stream is not None else torch.cuda.current_stream(self.torch_device)
        self._h = _vp()
        st = lib().cavs_create(ct.byref(self._h), device, s.cuda_stream)
        if st != OK:
            raise CavsError(st, "cavs_create failed")

    def close(self):
        if self._h:
            lib().cavs_destroy(self._h)
            self._h = _vp()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def check(self, st: int):
        if st != OK:
            raise CavsError(st, lib().cavs_last_error(self._h).decode())

    def sync(self):
        """cavs_sync: waits for the context's stream; raises on a kernel-recorded error."""
        self.check(lib().cavs_sync(self._h))

    def set_stream(self, stream: torch.cuda.Stream):
        self.check(lib().cavs_set_stream(self._h, stream.cuda_stream))

    def timing(self, on: bool):
        """Per-launch HIP-event timing of every library kernel (instrumentation)."""
        self.check(lib().cavs_timing_enable(self._h, int(bool(on))))

    def timing_read(self) -> list:
        """[(kernel name, row0, rows, ms)] per launch since the last read; synchronises."""
        cap = 1 << 16
        buf = (cavs_launch_time * cap)()
        n = lib().cavs_timing_read(self._h, buf, cap)
        if n < 0:
            self.check(n)
        return [(buf[i].name.decode(), int(buf[i].row0), int(buf[i].rows), float(buf[i].ms))
                for i in range(min(n, cap))]


@dataclass
class Schedule:
    """Schedule outputs (device tensors, host counts and offsets) plus the
    schedule workspace, reusable across batches of the same size."""
    raw: cavs_sched
    tensors: dict
    level_offsets_host: np.ndarray
    ws: torch.Tensor

    @property
    def T(self) -> int:
        return int(self.raw.T)

    def host(self) -> dict:
        d = {k: v.cpu().numpy() for k, v in self.tensors.items()
             if k not in ("in_offsets", "in_edges")}
        if self.raw.dag:
            d["in_offsets"] = self.tensors["in_offsets"].cpu().numpy()
            d["in_edges"] = self.tensors["in_edges"].cpu().numpy()
        d["level_offsets"] = d["level_offsets"][: self.T + 1]
        d["pull_list"] = d["pull_list"][: self.raw.n_pull]
        d["child_pos"] = d["child_pos"].reshape(-1, self.raw.N)
        d["T"] = self.T
        for k in ("n_pull", "n_labelled", "n_leaf_noinput", "n_inner_input"):
            d[k] = int(getattr(self.raw, k))
        return d


def alloc_schedule(ctx: Context, V: int, N: int, n_x: int) -> Schedule:
    """Allocates the schedule's output arrays and workspace for V vertices."""
    dev = ctx.torch_device
    i32 = dict(dtype=torch.int32, device=dev)
    t = dict(level=torch.empty(V, **i32), order=torch.empty(V, **i32), pos=torch.empty(V, **i32),
             child_pos=torch.empty(V * N, **i32), parent_pos=torch.empty(V, **i32),
             pull_pos=torch.empty(V, **i32), push_pos=torch.empty(V, **i32),
             pull_list=torch.empty(V, **i32), level_offsets=torch.empty(V + 1, **i32),
             in_offsets=torch.empty(V + 1, **i32), in_edges=torch.empty(V * N, **i32))
    host_off = np.zeros(V + 1, dtype=np.int32)
    s = cavs_sched()
    for k, v in t.items():
        setattr(s, k, v.data_ptr() if V > 0 else None)
    s.level_offsets_host = host_off.ctypes.data
    nbytes = lib().cavs_schedule_workspace_bytes(V, N, int(n_x))
    ws = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=dev)
    return Schedule(raw=s, tensors=t, level_offsets_host=host_off, ws=ws)


def run_schedule(ctx: Context, sched: Schedule, child: torch.Tensor,
                 parent: Optional[torch.Tensor],
                 pull_idx: Optional[torch.Tensor] = None,
                 push_idx: Optional[torch.Tensor] = None, n_x: int = 0, n_push: int = 0):
    """cavs_schedule into a previously allocated Schedule (one synchronisation).
    parent=None: graph inputs (a vertex may be read by several vertices)."""
    V = int(child.shape[0])
    N = int(child.shape[1]) if child.dim() == 2 else 1
    g = cavs_graphs(V, N, int(n_x), int(n_push), _ptr(child), _ptr(parent), _ptr(pull_idx),
                    _ptr(push_idx))
    nbytes = sched.ws.numel()
    ctx.check(lib().cavs_schedule(ctx._h, ct.byref(g), ct.byref(sched.raw),
                                  sched.ws.data_ptr(), nbytes))
    return sched


SCHEDULE_STATIC_BYTES = 4 << 20   # CAVS_SCHEDULE_STATIC_BYTES


def run_schedule_static(ctx: Context, sched: Schedule, child: torch.Tensor,
                        parent: Optional[torch.Tensor],
                        pull_idx: Optional[torch.Tensor] = None,
                        push_idx: Optional[torch.Tensor] = None, n_x: int = 0, n_push: int = 0):
    """cavs_schedule_static into a previously allocated Schedule: the
    scheduler's scratch comes from the library's static device array, so
    ``sched.ws`` is not used."""
    V = int(child.shape[0])
    N = int(child.shape[1]) if child.dim() == 2 else 1
    g = cavs_graphs(V, N, int(n_x), int(n_push), _ptr(child), _ptr(parent), _ptr(pull_idx),
                    _ptr(push_idx))
    ctx.check(lib().cavs_schedule_static(ctx._h, ct.byref(g), ct.byref(sched.raw)))
    return sched


def schedule(ctx: Context, child: torch.Tensor, parent: Optional[torch.Tensor],
             pull_idx: Optional[torch.Tensor] = None, push_idx: Optional[torch.Tensor] = None,
             n_x: int = 0, n_push: int = 0) -> Schedule:
    """cavs_schedule: int32 device tensors child [V, N], parent [V] (None for
    graph inputs), ..."""
    V = int(child.shape[0])
    N = int(child.shape[1]) if child.dim() == 2 else 1
    sched = alloc_schedule(ctx, V, N, n_x)
    return run_schedule(ctx, sched, child, parent, pull_idx, push_idx, n_x, n_push)


@dataclass
class Params:
    cell: int
    prec: int
    loss: int
    D: int
    H: int
    N: int
    C: int
    Wx: Optional[torch.Tensor]
    U: torch.Tensor
    b: torch.Tensor
    Ws: Optional[torch.Tensor]
    bs: Optional[torch.Tensor]

    def raw(self) -> cavs_params:
        return cavs_params(self.cell, self.prec, self.loss, self.D, self.H, self.N, self.C,
                           _ptr(self.Wx), _ptr(self.U), _ptr(self.b), _ptr(self.Ws),
                           _ptr(self.bs))


def workspace_bytes(params: Params, sched: Schedule) -> int:
    p = params.raw()
    return int(lib().cavs_workspace_bytes(ct.byref(p), ct.byref(sched.raw)))


def forward(ctx: Context, params: Params, sched: Schedule, X: Optional[torch.Tensor],
            Y: Optional[torch.Tensor], ws: torch.Tensor, h_out: torch.Tensor,
            c_out: Optional[torch.Tensor], loss_out: torch.Tensor) -> None:
    """cavs_forward (asynchronous on the context's stream)."""
    p = params.raw()
    inp = cavs_inputs(_ptr(X), _ptr(Y), int(Y.shape[0]) if Y is not None else 0)
    ctx.check(lib().cavs_forward(ctx._h, ct.byref(p), ct.byref(sched.raw), ct.byref(inp),
                                 _ptr(h_out), _ptr(c_out), _ptr(loss_out), ws.data_ptr(),
                                 ws.numel()))


def infer_workspace_bytes(params: Params, sched: Schedule) -> int:
    p = params.raw()
    return int(lib().cavs_infer_workspace_bytes(ct.byref(p), ct.byref(sched.raw)))


def infer(ctx: Context, params: Params, sched: Schedule, X: Optional[torch.Tensor],
          Y: Optional[torch.Tensor], ws: torch.Tensor, h_out: torch.Tensor,
          c_out: Optional[torch.Tensor], loss_out: torch.Tensor) -> None:
    """cavs_infer (asynchronous on the context's stream)."""
    p = params.raw()
    inp = cavs_inputs(_ptr(X), _ptr(Y), int(Y.shape[0]) if Y is not None else 0)
    ctx.check(lib().cavs_infer(ctx._h, ct.byref(p), ct.byref(sched.raw), ct.byref(inp),
                               _ptr(h_out), _ptr(c_out), _ptr(loss_out), ws.data_ptr(),
                               ws.numel()))


def backward(ctx: Context, params: Params, sched: Schedule, X: Optional[torch.Tensor],
             Y: Optional[torch.Tensor], ws: torch.Tensor, grads: dict,
             dH_ext: Optional[torch.Tensor] = None) -> None:
    """cavs_backward (asynchronous); ``grads`` holds dWx, dU, db, dWs, dbs, dX
    tensors; ``dH_ext`` [V, H] (vertex-id rows) is an external gradient of the
    pushed states."""
    p = params.raw()
    inp = cavs_inputs(_ptr(X), _ptr(Y), int(Y.shape[0]) if Y is not None else 0,
                      _ptr(dH_ext))
    g = cavs_grads(*[_ptr(grads.get(k)) for k in ("dWx", "dU", "db", "dWs", "dbs", "dX")])
    ctx.check(lib().cavs_backward(ctx._h, ct.byref(p), ct.byref(sched.raw), ct.byref(inp),
                                  ws.data_ptr(), ws.numel(), ct.byref(g)))
