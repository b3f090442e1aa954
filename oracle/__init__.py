"""CPU oracle for the Cavs vertex-function forward/backward (arXiv 1712.04048).

TEST INFRASTRUCTURE ONLY: imported by the tests, by ``__graft_entry__.smoke``
and by the CPU-baseline leg of ``bench.py``; the product path never imports or
calls it.  The arithmetic lives in ``oracle.c`` (plain C); this module only
compiles it with gcc -- once in fp64 (``liboracle.so``, the parity reference)
and once in fp32 (``liboracle_f32.so``, the same definitions evaluated in
float) -- loads it with ctypes and marshals numpy arrays.

Results are returned indexed by vertex id.  Gate arrays use the oracle's own
per-vertex layout [i | o | u | f_0 .. f_{N-1}], each H wide.
"""
from __future__ import annotations

import ctypes as ct
import os
import subprocess
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIBS = {"f64": os.path.join(_HERE, "liboracle.so"),
         "f32": os.path.join(_HERE, "liboracle_f32.so")}
_LIB = _LIBS["f64"]

OK = 0
ERR_ARG = -1
ERR_RANGE = -2
ERR_MULTIPARENT = -3
ERR_CYCLE = -4
ERR_MISMATCH = -5
ERR_DUP_PULL = -9

LOSS_CE = 0
LOSS_L2 = 1
LOSS_NONE = 2


def build(force: bool = False, precision: str = "f64") -> str:
    """Compile oracle.c into liboracle.so (fp64) or liboracle_f32.so (fp32):
    gcc -O2, no fast-math, no FMA contraction (each product and sum rounds
    on its own, as the source reads)."""
    path = _LIBS[precision]
    if force or not os.path.exists(path) or os.path.getmtime(path) < os.path.getmtime(_SRC):
        tmp = path + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-std=c99", "-ffp-contract=off", "-D_DEFAULT_SOURCE", "-shared",
               "-fPIC", _SRC, "-o", tmp, "-lm"]
        if precision == "f32":
            cmd.insert(1, "-DORC_FLOAT")
        subprocess.check_call(cmd)
        os.replace(tmp, path)
    return path


def build_all(force: bool = False) -> None:
    for p in _LIBS:
        build(force, p)


_libs = {}


def lib(precision: str = "f64"):
    if precision not in _libs:
        L = ct.CDLL(build(precision=precision))
        i32p = ct.POINTER(ct.c_int)
        f64p = ct.POINTER(ct.c_double) if precision == "f64" else ct.POINTER(ct.c_float)
        freal = ct.c_double if precision == "f64" else ct.c_float
        L.orc_real_bytes.restype = ct.c_int
        assert L.orc_real_bytes() == (8 if precision == "f64" else 4)
        _lib = L
        _lib.orc_validate.restype = ct.c_int
        _lib.orc_validate.argtypes = [ct.c_int, ct.c_int, i32p, i32p, i32p, ct.c_int, i32p, ct.c_int]
        _lib.orc_levels_recursive.restype = ct.c_int
        _lib.orc_levels_recursive.argtypes = [ct.c_int, ct.c_int, i32p, i32p]
        _lib.orc_levels_frontier.restype = ct.c_int
        _lib.orc_levels_frontier.argtypes = [ct.c_int, ct.c_int, i32p, i32p]
        _lib.orc_schedule.restype = ct.c_int
        _lib.orc_schedule.argtypes = [ct.c_int, ct.c_int, i32p, i32p, i32p, i32p, ct.c_int] + [i32p] * 10
        _lib.orc_treelstm.restype = ct.c_int
        _lib.orc_treelstm.argtypes = ([ct.c_int] * 8 + [i32p] * 4 + [f64p] * 7 + [freal]
                                      + [f64p] * 5 + [ct.c_int] + [f64p] * 9)
        _lib.orc_treefc.restype = ct.c_int
        _lib.orc_treefc.argtypes = ([ct.c_int] * 7 + [i32p] * 4 + [f64p] * 6 + [freal]
                                    + [f64p] * 3 + [ct.c_int] + [f64p] * 8)
        _lib.orc_bf16_round.restype = ct.c_double
        _lib.orc_bf16_round.argtypes = [ct.c_double]
        _libs[precision] = L
    return _libs[precision]


def _i32(a):
    if a is None:
        return None, None
    a = np.ascontiguousarray(np.asarray(a, dtype=np.int32))
    return a, a.ctypes.data_as(ct.POINTER(ct.c_int))


def _real(a, dtype=np.float64):
    if a is None:
        return None, None
    a = np.ascontiguousarray(np.asarray(a, dtype=dtype))
    ct_t = ct.c_double if dtype == np.float64 else ct.c_float
    return a, a.ctypes.data_as(ct.POINTER(ct_t))


def _f64(a):
    return _real(a, np.float64)


def _out(shape, dtype=np.float64):
    a = np.zeros(shape, dtype=dtype)
    ct_t = ct.c_double if dtype == np.float64 else ct.c_float
    return a, a.ctypes.data_as(ct.POINTER(ct_t))


def validate(child, parent, pull_idx=None, n_x=0, push_idx=None, n_push=0) -> int:
    """Validation status; parent=None declares graph (DAG) inputs."""
    child = np.asarray(child, dtype=np.int32)
    if child.ndim == 1:
        child = child.reshape(-1, 1)
    V, N = child.shape
    c, cp = _i32(child)
    p, pp = _i32(parent)
    pl, plp = _i32(pull_idx)
    ps, psp = _i32(push_idx)
    return lib().orc_validate(V, N, cp, pp, plp, int(n_x), psp, int(n_push))


def levels(child, mode: str = "recursive"):
    child = np.asarray(child, dtype=np.int32)
    V, N = child.shape
    c, cp = _i32(child)
    lev = np.zeros(V, dtype=np.int32)
    _, lp = _i32(lev)
    lp = lev.ctypes.data_as(ct.POINTER(ct.c_int))
    fn = lib().orc_levels_recursive if mode == "recursive" else lib().orc_levels_frontier
    T = fn(V, N, cp, lp)
    return T, lev


def schedule(child, parent, pull_idx=None, push_idx=None, mode: int = 0) -> dict:
    """Level-major layout; keys mirror the library's schedule outputs.
    parent=None declares graph (DAG) inputs (parent_pos is -1 throughout)."""
    child = np.asarray(child, dtype=np.int32)
    V, N = child.shape
    c, cp = _i32(child)
    p, pp = _i32(parent)
    pl, plp = _i32(pull_idx)
    ps, psp = _i32(push_idx)
    outs = {k: np.zeros(n, dtype=np.int32) for k, n in
            [("level", V), ("order", V), ("pos", V), ("child_pos", V * N), ("parent_pos", V),
             ("pull_pos", V), ("push_pos", V), ("level_offsets", V + 1), ("pull_list", V)]}
    n_pull = ct.c_int(0)
    ptrs = [outs[k].ctypes.data_as(ct.POINTER(ct.c_int)) for k in
            ["level", "order", "pos", "child_pos", "parent_pos", "pull_pos", "push_pos",
             "level_offsets", "pull_list"]]
    T = lib().orc_schedule(V, N, cp, pp, plp, psp, int(mode), *ptrs, ct.byref(n_pull))
    if T < 0:
        raise ValueError("oracle schedule failed: %d" % T)
    outs["T"] = T
    outs["level_offsets"] = outs["level_offsets"][: T + 1].copy()
    outs["n_pull"] = int(n_pull.value)
    outs["pull_list"] = outs["pull_list"][: n_pull.value].copy()
    outs["child_pos"] = outs["child_pos"].reshape(V, N)
    return outs


def bf16_round(x: float) -> float:
    return lib().orc_bf16_round(float(x))


def run(wl, *, order_mode: int = 0, bf16: Optional[bool] = None, backward: bool = True,
        denom: float = 0.0, params: Optional[dict] = None, X=None, Y=None,
        precision: str = "f64", dH_ext=None) -> dict:
    """Forward (+ loss) and optionally backward of ``wl``.

    ``precision`` "f64" (the parity reference) or "f32" (the same definitions
    evaluated in fp32).  ``params`` may override any of Wx, U, b, Ws, bs (e.g.
    for finite differences); X/Y likewise.  ``bf16`` defaults to the
    workload's precision.  ``dH_ext`` [V, H] (vertex-id rows) is the gradient
    of the pushed states from an external consumer, added to every dL/dh.
    Graph workloads (``wl.dag``) pass no parent array,
    so a vertex may be read by several vertices.  Returns a dict of float64
    arrays with h, c, gates, lossv, loss and, when ``backward``, dh, dc
    (total dL/dh_v, dL/dc_v per vertex), dWx, dU, db, dWs, dbs, dX.
    """
    L = lib(precision)
    dt = np.float64 if precision == "f64" else np.float32
    rl = lambda a: _real(a, dt)
    out = lambda shape: _out(shape, dt)
    from_wl = dict(Wx=wl.Wx, U=wl.U, b=wl.b, Ws=wl.Ws, bs=wl.bs)
    if params:
        from_wl.update(params)
    if bf16 is None:
        bf16 = wl.prec == 1
    V, N, D, H, C = wl.V, wl.N, wl.D, wl.H, wl.C
    Xa = wl.X if X is None else X
    Ya = wl.Y if Y is None else Y
    _, chp = _i32(wl.child.reshape(-1))
    ch_keep = _
    dag = bool(getattr(wl, "dag", False))
    par, parp = _i32(None if dag else wl.parent)
    pl, plp = _i32(wl.pull_idx)
    ps, psp = _i32(wl.push_idx)
    Xk, Xp = rl(Xa if Xa.size else np.zeros(1))
    Yk, Yp = rl(Ya if Ya.size else np.zeros(1))
    Wk, Wp = rl(from_wl["Wx"] if from_wl["Wx"].size else np.zeros(1))
    Uk, Up = rl(from_wl["U"])
    bk, bp = rl(from_wl["b"])
    Wsk, Wsp = rl(from_wl["Ws"] if from_wl["Ws"].size else np.zeros(1))
    bsk, bsp = rl(from_wl["bs"] if from_wl["bs"].size else np.zeros(1))
    h, hp = out((V, H))
    lossv, lvp = out(V)
    ext, extp = rl(dH_ext) if dH_ext is not None else (None, None)
    loss = (ct.c_double if precision == "f64" else ct.c_float)(0.0)
    n_x = max(int(Xa.shape[0]), 1)
    res = dict()
    if wl.cell == 0:
        c, cp = out((V, H))
        gates, gp = out((V, (3 + N) * H))
        dh, dhp = out((V, H))
        dc, dcp = out((V, H))
        dWx, dWxp = out((D, 4 * H))
        dU, dUp = out((H, 4 * H))
        db, dbp = out(4 * H)
        dWs, dWsp = out((H, max(C, 1)))
        dbs, dbsp = out(max(C, 1))
        dX, dXp = out((n_x, D))
        st = L.orc_treelstm(V, N, D, H, C, wl.loss, int(bool(bf16)), int(order_mode),
                            chp, parp, plp, psp, Xp, Yp, Wp, Up, bp, Wsp, bsp,
                            float(denom), hp, cp, gp, lvp, ct.byref(loss), int(backward),
                            dhp, dcp, dWxp, dUp, dbp, dWsp, dbsp, dXp, extp)
        res.update(c=c, gates=gates)
        if backward:
            res.update(dh=dh, dc=dc, dWx=dWx, dU=dU, db=db, dX=dX[: Xa.shape[0]])
            if wl.loss == LOSS_CE:
                res.update(dWs=dWs[:, :C], dbs=dbs[:C])
    else:
        dh, dhp = out((V, H))
        dcs, dcsp = out((V, H))
        dW, dWp = out((N * H, H))
        db, dbp = out(H)
        dWs, dWsp = out((H, max(C, 1)))
        dbs, dbsp = out(max(C, 1))
        dX, dXp = out((n_x, H))
        st = L.orc_treefc(V, N, H, C, wl.loss, int(bool(bf16)), int(order_mode),
                          chp, parp, plp, psp, Xp, Yp, Up, bp, Wsp, bsp, float(denom),
                          hp, lvp, ct.byref(loss), int(backward), dhp, dcsp, dWp, dbp,
                          dWsp, dbsp, dXp, extp)
        if backward:
            res.update(dh=dh, dU=dW, db=db, dX=dX[: Xa.shape[0]])
            if wl.loss == LOSS_CE:
                res.update(dWs=dWs[:, :C], dbs=dbs[:C])
    del ch_keep, ext
    if st != OK:
        raise ValueError("oracle rejected the input: status %d" % st)
    res.update(h=h, lossv=lossv, loss=float(loss.value))
    if precision != "f64":
        res = {k: (v.astype(np.float64) if isinstance(v, np.ndarray) else v)
               for k, v in res.items()}
    return res
