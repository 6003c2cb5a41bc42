"""Oracle for the OmniMoE atomic-expert layer: TEST INFRASTRUCTURE ONLY.

A plain, slow, fp64 host implementation of the layer (``omnimoe_ref.cpp``) with a ctypes
wrapper. Only the tests, the smoke check and the benchmark's CPU-baseline leg may import it; the
GPU library never does. Arguments are numpy arrays; bf16 inputs must be widened to float32 first.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

BRUTE, CARTESIAN, LOGSOFTMAX_BRUTE = 0, 1, 2


class RefDesc(ctypes.Structure):
    _fields_ = [("T", ctypes.c_int64), ("d", ctypes.c_int32), ("n_rows", ctypes.c_int32),
                ("n_cols", ctypes.c_int32), ("d_key", ctypes.c_int32), ("H", ctypes.c_int32),
                ("K", ctypes.c_int32), ("act", ctypes.c_int32), ("query_mode", ctypes.c_int32),
                ("group_size", ctypes.c_int32)]


def build(verbose: bool = False) -> str:
    cmd = ["g++", "-O2", "-std=c++17", "-ffp-contract=off", "-fPIC", "-shared", "-pthread",
           os.path.join(_HERE, "omnimoe_ref.cpp"), "-o", _LIB_PATH]
    if verbose:
        print(" ".join(cmd))
    subprocess.check_call(cmd)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError(f"{_LIB_PATH} is not built; run __graft_entry__.build()")
        lib = ctypes.CDLL(_LIB_PATH)
        P = ctypes.c_void_p
        D = ctypes.POINTER(RefDesc)
        lib.omnimoe_ref_half_scores.argtypes = [D, P, P, P, P, P, ctypes.c_int]
        lib.omnimoe_ref_select.argtypes = [D, P, P, ctypes.c_int, P, P, P, P, ctypes.c_int]
        lib.omnimoe_ref_select_f32.argtypes = [D, P, ctypes.c_int, P, P, P, P, ctypes.c_int]
        lib.omnimoe_ref_schedule.argtypes = [D, P, P, P, P, P, P]
        lib.omnimoe_ref_expert_forward.argtypes = [D, P, P, P, P, P, ctypes.c_int, P,
                                                   ctypes.c_int]
        lib.omnimoe_ref_layer_forward.argtypes = [D, P, P, P, P, P, ctypes.c_int, P, P, P,
                                                  ctypes.c_int]
        lib.omnimoe_ref_route_dense.argtypes = [D, P, P, P, P, P, ctypes.c_int]
        lib.omnimoe_ref_select_dense_f32.argtypes = [D, P, P, P, ctypes.c_int]
        lib.omnimoe_ref_shared_mlp.argtypes = [D, ctypes.c_int32, P, P, P, P, ctypes.c_int]
        lib.omnimoe_ref_expert_backward.argtypes = [D, P, P, P, P, P, P, P, P, P, P, P, P, P,
                                                    ctypes.c_int]
        lib.omnimoe_ref_route_backward.argtypes = [D, P, P, P, P, P, P, P, P, ctypes.c_int]
        lib.omnimoe_ref_act_grad.argtypes = [ctypes.c_int, ctypes.c_double]
        lib.omnimoe_ref_act_grad.restype = ctypes.c_double
        lib.omnimoe_ref_act.argtypes = [ctypes.c_int, ctypes.c_double]
        lib.omnimoe_ref_act.restype = ctypes.c_double
        for f in ("half_scores", "select", "select_f32", "schedule", "expert_forward",
                  "layer_forward", "route_dense", "select_dense_f32", "shared_mlp",
                  "expert_backward", "route_backward"):
            getattr(lib, "omnimoe_ref_" + f).restype = ctypes.c_int
        _lib = lib
    return _lib


def default_threads() -> int:
    n = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else (os.cpu_count() or 1)
    return max(1, min(64, n))


def desc(w, T: Optional[int] = None, K: Optional[int] = None, H: Optional[int] = None,
         group_size: Optional[int] = None) -> RefDesc:
    """Descriptor from any object with the layer's shape attributes."""
    return RefDesc(
        T=int(w.T if T is None else T), d=int(w.d), n_rows=int(w.n_rows), n_cols=int(w.n_cols),
        d_key=int(w.d_key), H=int(w.H if H is None else H), K=int(w.K if K is None else K),
        act={"gelu": 0, "silu": 1}[getattr(w, "act", "gelu")],
        query_mode={"split": 0, "shared": 1}[getattr(w, "query_mode", "split")],
        group_size=int(group_size if group_size is not None else getattr(w, "group_size", 1)))


def _f32(a):
    a = np.ascontiguousarray(a, dtype=np.float32)
    return a, a.ctypes.data


def _check(rc, what):
    if rc != 0:
        raise ValueError(f"oracle {what} rejected its arguments (rc={rc})")


def half_scores(dsc: RefDesc, x, keys_row, keys_col, n_threads=None):
    """Row and column logits (Eq. 9): sr [T, H, n_rows], sc [T, H, n_cols] in fp64."""
    lib = _load()
    x, px = _f32(x)
    kr, pkr = _f32(keys_row)
    kc, pkc = _f32(keys_col)
    sr = np.empty((dsc.T, dsc.H, dsc.n_rows), np.float64)
    sc = np.empty((dsc.T, dsc.H, dsc.n_cols), np.float64)
    _check(lib.omnimoe_ref_half_scores(ctypes.byref(dsc), px, pkr, pkc, sr.ctypes.data,
                                       sc.ctypes.data, n_threads or default_threads()),
           "half_scores")
    return sr, sc


def select(dsc: RefDesc, sr, sc, method=CARTESIAN, n_threads=None):
    """(idx [T,H,K] int32, selected scores fp64, gates fp64, number of inexact candidate sums)."""
    lib = _load()
    sr = np.ascontiguousarray(sr, np.float64)
    sc = np.ascontiguousarray(sc, np.float64)
    shape = (dsc.T, dsc.H, dsc.K)
    idx = np.empty(shape, np.int32)
    sel = np.empty(shape, np.float64)
    g = np.empty(shape, np.float64)
    inexact = ctypes.c_int64(0)
    _check(lib.omnimoe_ref_select(ctypes.byref(dsc), sr.ctypes.data, sc.ctypes.data, method,
                                  idx.ctypes.data, sel.ctypes.data, g.ctypes.data,
                                  ctypes.addressof(inexact), n_threads or default_threads()),
           "select")
    return idx, sel, g, inexact.value


def select_f32(dsc: RefDesc, hs, method=CARTESIAN, n_threads=None):
    """Selection from float32 half-scores [T, H, n_rows + n_cols]."""
    lib = _load()
    hs, phs = _f32(hs)
    shape = (dsc.T, dsc.H, dsc.K)
    idx = np.empty(shape, np.int32)
    sel = np.empty(shape, np.float64)
    g = np.empty(shape, np.float64)
    inexact = ctypes.c_int64(0)
    _check(lib.omnimoe_ref_select_f32(ctypes.byref(dsc), phs, method, idx.ctypes.data,
                                      sel.ctypes.data, g.ctypes.data, ctypes.addressof(inexact),
                                      n_threads or default_threads()), "select_f32")
    return idx, sel, g, inexact.value


def schedule(dsc: RefDesc, idx):
    """(perm [M], active [n_active], active_offsets [n_active+1], dense_offsets [N+1])."""
    lib = _load()
    idx = np.ascontiguousarray(idx, np.int32)
    M = dsc.T * dsc.H * dsc.K
    N = dsc.n_rows * dsc.n_cols
    perm = np.empty(M, np.int32)
    active = np.empty(min(M, N) + 1, np.int32)
    off = np.empty(min(M, N) + 1, np.int32)
    dense = np.empty(N + 1, np.int32)
    na = ctypes.c_int32(0)
    _check(lib.omnimoe_ref_schedule(ctypes.byref(dsc), idx.ctypes.data, perm.ctypes.data,
                                    active.ctypes.data, off.ctypes.data, ctypes.addressof(na),
                                    dense.ctypes.data), "schedule")
    A = na.value
    return perm, active[:A].copy(), off[:A + 1].copy(), dense


def expert_forward(dsc: RefDesc, x, u, v, idx, gates, scheduled=True, n_threads=None):
    """Routed output y [T, d] in fp64."""
    lib = _load()
    x, px = _f32(x)
    u, pu = _f32(u)
    v, pv = _f32(v)
    idx = np.ascontiguousarray(idx, np.int32)
    gates = np.ascontiguousarray(gates, np.float64)
    y = np.empty((dsc.T, dsc.d), np.float64)
    _check(lib.omnimoe_ref_expert_forward(ctypes.byref(dsc), px, pu, pv, idx.ctypes.data,
                                          gates.ctypes.data, 1 if scheduled else 0,
                                          y.ctypes.data, n_threads or default_threads()),
           "expert_forward")
    return y


def layer_forward(dsc: RefDesc, x, keys_row, keys_col, u, v, method=CARTESIAN, n_threads=None):
    """(y [T, d] fp64, idx [T,H,K], gates [T,H,K] fp64)."""
    lib = _load()
    x, px = _f32(x)
    kr, pkr = _f32(keys_row)
    kc, pkc = _f32(keys_col)
    u, pu = _f32(u)
    v, pv = _f32(v)
    y = np.empty((dsc.T, dsc.d), np.float64)
    idx = np.empty((dsc.T, dsc.H, dsc.K), np.int32)
    g = np.empty((dsc.T, dsc.H, dsc.K), np.float64)
    _check(lib.omnimoe_ref_layer_forward(ctypes.byref(dsc), px, pkr, pkc, pu, pv, method,
                                         y.ctypes.data, idx.ctypes.data, g.ctypes.data,
                                         n_threads or default_threads()), "layer_forward")
    return y, idx, g


def route_dense(dsc: RefDesc, x, w_gate, with_logits=False, n_threads=None):
    """Dense router (the router ablation): (idx [T,H,K], gates fp64, logits [T,H,N] fp64 or
    None). w_gate is [H, N, d]."""
    lib = _load()
    x, px = _f32(x)
    wg, pwg = _f32(w_gate)
    N = dsc.n_rows * dsc.n_cols
    idx = np.empty((dsc.T, dsc.H, dsc.K), np.int32)
    g = np.empty((dsc.T, dsc.H, dsc.K), np.float64)
    L = np.empty((dsc.T, dsc.H, N), np.float64) if with_logits else None
    _check(lib.omnimoe_ref_route_dense(ctypes.byref(dsc), px, pwg, idx.ctypes.data, g.ctypes.data,
                                       None if L is None else L.ctypes.data,
                                       n_threads or default_threads()), "route_dense")
    return idx, g, L


def select_dense_f32(dsc: RefDesc, logits, n_threads=None):
    """The dense router's top-K and gates from float32 logits [T, H, N]."""
    lib = _load()
    L, pl = _f32(logits)
    idx = np.empty((dsc.T, dsc.H, dsc.K), np.int32)
    g = np.empty((dsc.T, dsc.H, dsc.K), np.float64)
    _check(lib.omnimoe_ref_select_dense_f32(ctypes.byref(dsc), pl, idx.ctypes.data,
                                            g.ctypes.data, n_threads or default_threads()),
           "select_dense_f32")
    return idx, g


def shared_mlp(dsc: RefDesc, x, w_gu, w_down, y=None, n_threads=None):
    """y + MLP(x) in fp64 (y = 0 when not given): the shared SwiGLU branch, w_gu [2 d_ff, d]
    (gate rows then up rows), w_down [d, d_ff]."""
    lib = _load()
    x, px = _f32(x)
    wgu, pgu = _f32(w_gu)
    wd, pwd = _f32(w_down)
    d_ff = wd.shape[1]
    assert wgu.shape == (2 * d_ff, dsc.d) and wd.shape == (dsc.d, d_ff)
    out = np.zeros((dsc.T, dsc.d), np.float64) if y is None else np.array(y, np.float64)
    _check(lib.omnimoe_ref_shared_mlp(ctypes.byref(dsc), d_ff, px, pgu, pwd, out.ctypes.data,
                                      n_threads or default_threads()), "shared_mlp")
    return out


def expert_backward(dsc: RefDesc, x, u, v, idx, gates, dy, n_threads=None):
    """Gradients of L = sum_t dy_t . y_t through the expert compute, fp64: a dict with dx [T, d],
    active [A], du_rows / dv_rows [A, d] (rows of the active experts, ascending id), dgates and
    dscores [T, H, K]."""
    lib = _load()
    x, px = _f32(x)
    u, pu = _f32(u)
    v, pv = _f32(v)
    idx = np.ascontiguousarray(idx, np.int32)
    gates = np.ascontiguousarray(gates, np.float64)
    dy = np.ascontiguousarray(dy, np.float64)
    T, D = dsc.T, dsc.d
    M = T * dsc.H * dsc.K
    cap = min(M, dsc.n_rows * dsc.n_cols)
    dx = np.empty((T, D), np.float64)
    du = np.empty((cap, D), np.float64)
    dv = np.empty((cap, D), np.float64)
    active = np.empty(cap, np.int32)
    na = np.zeros(1, np.int32)
    dg = np.empty((T, dsc.H, dsc.K), np.float64)
    ds = np.empty((T, dsc.H, dsc.K), np.float64)
    _check(lib.omnimoe_ref_expert_backward(
        ctypes.byref(dsc), px, pu, pv, idx.ctypes.data, gates.ctypes.data, dy.ctypes.data,
        dx.ctypes.data, du.ctypes.data, dv.ctypes.data, active.ctypes.data, na.ctypes.data,
        dg.ctypes.data, ds.ctypes.data, n_threads or default_threads()), "expert_backward")
    A = int(na[0])
    return {"dx": dx, "active": active[:A], "du_rows": du[:A], "dv_rows": dv[:A],
            "dgates": dg, "dscores": ds}


def route_backward(dsc: RefDesc, x, keys_row, keys_col, idx, dscores, dx=None, n_threads=None):
    """Router backward for fixed selections, fp64: (dx + router share, dkeys_row, dkeys_col)."""
    lib = _load()
    x, px = _f32(x)
    kr, pkr = _f32(keys_row)
    kc, pkc = _f32(keys_col)
    idx = np.ascontiguousarray(idx, np.int32)
    ds = np.ascontiguousarray(dscores, np.float64)
    out = np.zeros((dsc.T, dsc.d), np.float64) if dx is None else np.array(dx, np.float64)
    dkr = np.empty((dsc.H, dsc.n_rows, dsc.d_key), np.float64)
    dkc = np.empty((dsc.H, dsc.n_cols, dsc.d_key), np.float64)
    _check(lib.omnimoe_ref_route_backward(ctypes.byref(dsc), px, pkr, pkc, idx.ctypes.data,
                                          ds.ctypes.data, out.ctypes.data, dkr.ctypes.data,
                                          dkc.ctypes.data, n_threads or default_threads()),
           "route_backward")
    return out, dkr, dkc


def act_grad(kind: int, z: float) -> float:
    return _load().omnimoe_ref_act_grad(kind, float(z))


def act(kind: int, z: float) -> float:
    return _load().omnimoe_ref_act(kind, float(z))
