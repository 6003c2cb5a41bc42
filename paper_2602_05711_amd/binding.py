"""Python binding of libomnimoe.so (declared in include/omnimoe.h): argument marshalling only.

Every function has the name of the C entry point it calls and takes torch tensors on the GPU.
torch provides device memory and the stream (the current stream unless one is given); all of
the layer's work runs in the library's HIP kernels. There is no fallback: the functions raise
when the library is missing or a call fails.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libomnimoe.so")

OMNIMOE_F32, OMNIMOE_BF16 = 0, 1
OMNIMOE_ACT_GELU, OMNIMOE_ACT_SILU = 0, 1
OMNIMOE_QUERY_SPLIT, OMNIMOE_QUERY_SHARED = 0, 1
(STAGE_ROUTE, STAGE_SELECT, STAGE_SCHEDULE, STAGE_EXPERT, STAGE_LAYER, STAGE_ROUTE_DENSE,
 STAGE_EXPERT_BACKWARD, STAGE_ROUTE_BACKWARD, STAGE_EXPERT_GROUPED,
 STAGE_EXPERT_SCATTER, STAGE_EXPERT_GROUP_ROWS) = range(11)
KERNEL_NAMES = ("score", "select", "schedule", "expert_dot", "accumulate")

EXPORTED = (
    "omnimoe_workspace_size", "omnimoe_route", "omnimoe_select", "omnimoe_route_dense",
    "omnimoe_select_dense", "omnimoe_shared_mlp", "omnimoe_shared_mlp_workspace_size",
    "omnimoe_schedule",
    "omnimoe_expert_forward", "omnimoe_expert_forward_grouped",
    "omnimoe_expert_forward_scatter", "omnimoe_expert_forward_token_centric",
    "omnimoe_expert_forward_group_rows",
    "omnimoe_expert_backward",
    "omnimoe_route_backward",
    "omnimoe_layer_forward", "omnimoe_layer_forward_noalloc", "omnimoe_layer_path",
    "omnimoe_timer_create",
    "omnimoe_timer_destroy", "omnimoe_timer_read", "omnimoe_layer_forward_timed",
    "omnimoe_status_string",
)


class OmnimoeLayerDesc(ctypes.Structure):
    _fields_ = [("T", ctypes.c_int64), ("d", ctypes.c_int32), ("n_rows", ctypes.c_int32),
                ("n_cols", ctypes.c_int32), ("d_key", ctypes.c_int32), ("H", ctypes.c_int32),
                ("K", ctypes.c_int32), ("dtype", ctypes.c_int32), ("act", ctypes.c_int32),
                ("query_mode", ctypes.c_int32), ("group_size", ctypes.c_int32)]


class OmnimoeError(RuntimeError):
    def __init__(self, fn: str, status: int, text: str):
        super().__init__(f"{fn} failed: {text} (status {status})")
        self.status = status


_lib = None


def load_library():
    """Loads libomnimoe.so; raises when it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
    D = ctypes.POINTER(OmnimoeLayerDesc)
    sig = {
        "omnimoe_workspace_size": [D, I32, ctypes.POINTER(SZ)],
        "omnimoe_route": [D, P, P, P, P, P, P, P, SZ, P],
        "omnimoe_select": [D, P, P, P, P, SZ, P],
        "omnimoe_route_dense": [D, P, P, P, P, P, P, SZ, P],
        "omnimoe_select_dense": [D, P, P, P, P],
        "omnimoe_shared_mlp_workspace_size": [D, I32, ctypes.POINTER(SZ)],
        "omnimoe_shared_mlp": [D, I32, P, P, P, P, P, SZ, P],
        "omnimoe_schedule": [D, P, P, P, P, P, P, P, SZ, P],
        "omnimoe_expert_forward": [D, P, P, P, P, P, P, P, P, SZ, P],
        "omnimoe_expert_forward_grouped": [D, P, P, P, P, P, P, P, P, P, P, SZ, P],
        "omnimoe_expert_forward_scatter": [D, P, P, P, P, P, P, P, P, SZ, P],
        "omnimoe_expert_forward_group_rows": [D, P, P, P, P, P, P, P, P, P, P, SZ, P],
        "omnimoe_expert_forward_token_centric": [D, P, P, P, P, P, P, P],
        "omnimoe_expert_backward": [D, P, P, P, P, P, P, P, P, P, P, P, P, P, P, P, SZ, P],
        "omnimoe_route_backward": [D, P, P, P, P, P, P, P, P, P, SZ, P],
        "omnimoe_layer_forward": [D, P, P, P, P, P, P, P, P, P, SZ, P],
        "omnimoe_layer_forward_noalloc": [D, P, P, P, P, P, P, P, P, P],
        "omnimoe_layer_path": [D, ctypes.POINTER(I32)],
        "omnimoe_layer_forward_timed": [D, P, P, P, P, P, P, P, P, P, SZ, P, P],
        "omnimoe_timer_create": [I32, ctypes.POINTER(P)],
        "omnimoe_timer_destroy": [P],
        "omnimoe_timer_read": [P, ctypes.POINTER(ctypes.c_float), ctypes.POINTER(I32)],
    }
    for name, args in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = ctypes.c_int
    lib.omnimoe_status_string.argtypes = [I32]
    lib.omnimoe_status_string.restype = ctypes.c_char_p
    _lib = lib
    return lib


def _check(fn: str, status: int):
    if status != 0:
        text = load_library().omnimoe_status_string(status).decode()
        raise OmnimoeError(fn, status, text)


def make_desc(w, T: Optional[int] = None) -> OmnimoeLayerDesc:
    """Descriptor from an object with the layer's shape attributes (e.g. synth.Workload)."""
    return OmnimoeLayerDesc(
        T=int(w.T if T is None else T), d=int(w.d), n_rows=int(w.n_rows), n_cols=int(w.n_cols),
        d_key=int(w.d_key), H=int(w.H), K=int(w.K),
        dtype=OMNIMOE_BF16 if getattr(w, "dtype", "bf16") == "bf16" else OMNIMOE_F32,
        act={"gelu": OMNIMOE_ACT_GELU, "silu": OMNIMOE_ACT_SILU}[getattr(w, "act", "gelu")],
        query_mode={"split": OMNIMOE_QUERY_SPLIT,
                     "shared": OMNIMOE_QUERY_SHARED}[getattr(w, "query_mode", "split")],
        group_size=int(getattr(w, "group_size", 1)))


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def omnimoe_workspace_size(desc: OmnimoeLayerDesc, stage: int) -> int:
    n = ctypes.c_size_t(0)
    _check("omnimoe_workspace_size",
           load_library().omnimoe_workspace_size(ctypes.byref(desc), stage, ctypes.byref(n)))
    return n.value


def workspace(desc: OmnimoeLayerDesc, stage: int, device="cuda"):
    """A uint8 device tensor of the workspace size of `stage` (at least 256 bytes)."""
    import torch
    return torch.empty(max(256, omnimoe_workspace_size(desc, stage)), dtype=torch.uint8,
                       device=device)


def omnimoe_route(desc, x, keys_row, keys_col, idx, gates, half_scores=None, ws=None,
                  stream=None):
    if ws is None and half_scores is None:
        ws = workspace(desc, STAGE_ROUTE, x.device)
    _check("omnimoe_route", load_library().omnimoe_route(
        ctypes.byref(desc), _ptr(x), _ptr(keys_row), _ptr(keys_col), _ptr(idx), _ptr(gates),
        _ptr(half_scores), _ptr(ws), 0 if ws is None else ws.numel(), _stream(stream)))


def omnimoe_select(desc, half_scores, idx, gates, stream=None):
    _check("omnimoe_select", load_library().omnimoe_select(
        ctypes.byref(desc), _ptr(half_scores), _ptr(idx), _ptr(gates), None, 0, _stream(stream)))


def omnimoe_route_dense(desc, x, w_gate, idx, gates, logits=None, ws=None, stream=None):
    if ws is None and logits is None:
        ws = workspace(desc, STAGE_ROUTE_DENSE, x.device)
    _check("omnimoe_route_dense", load_library().omnimoe_route_dense(
        ctypes.byref(desc), _ptr(x), _ptr(w_gate), _ptr(idx), _ptr(gates), _ptr(logits),
        _ptr(ws), 0 if ws is None else ws.numel(), _stream(stream)))


def omnimoe_select_dense(desc, logits, idx, gates, stream=None):
    _check("omnimoe_select_dense", load_library().omnimoe_select_dense(
        ctypes.byref(desc), _ptr(logits), _ptr(idx), _ptr(gates), _stream(stream)))


def omnimoe_shared_mlp_workspace_size(desc, d_ff: int) -> int:
    n = ctypes.c_size_t(0)
    _check("omnimoe_shared_mlp_workspace_size", load_library().omnimoe_shared_mlp_workspace_size(
        ctypes.byref(desc), d_ff, ctypes.byref(n)))
    return n.value


def omnimoe_shared_mlp(desc, d_ff, x, w_gu, w_down, y, ws=None, stream=None):
    """y += MLP(x), the shared SwiGLU branch."""
    import torch
    if ws is None:
        ws = torch.empty(max(256, omnimoe_shared_mlp_workspace_size(desc, d_ff)),
                         dtype=torch.uint8, device=x.device)
    _check("omnimoe_shared_mlp", load_library().omnimoe_shared_mlp(
        ctypes.byref(desc), d_ff, _ptr(x), _ptr(w_gu), _ptr(w_down), _ptr(y), _ptr(ws),
        ws.numel(), _stream(stream)))


def omnimoe_schedule(desc, idx, perm, active, active_offsets, n_active, dense_offsets=None,
                     ws=None, stream=None):
    if ws is None:
        ws = workspace(desc, STAGE_SCHEDULE, idx.device)
    _check("omnimoe_schedule", load_library().omnimoe_schedule(
        ctypes.byref(desc), _ptr(idx), _ptr(perm), _ptr(active), _ptr(active_offsets),
        _ptr(n_active), _ptr(dense_offsets), _ptr(ws), ws.numel(), _stream(stream)))


def omnimoe_expert_forward(desc, x, u, v, idx, gates, perm, y, ws=None, stream=None):
    if ws is None:
        ws = workspace(desc, STAGE_EXPERT, x.device)
    _check("omnimoe_expert_forward", load_library().omnimoe_expert_forward(
        ctypes.byref(desc), _ptr(x), _ptr(u), _ptr(v), _ptr(idx), _ptr(gates), _ptr(perm),
        _ptr(y), _ptr(ws), ws.numel(), _stream(stream)))


def omnimoe_expert_forward_grouped(desc, x, u, v, idx, gates, perm, active, n_active, y, ws=None,
                                   stream=None):
    if ws is None:
        ws = workspace(desc, STAGE_EXPERT_GROUPED, x.device)
    _check("omnimoe_expert_forward_grouped", load_library().omnimoe_expert_forward_grouped(
        ctypes.byref(desc), _ptr(x), _ptr(u), _ptr(v), _ptr(idx), _ptr(gates), _ptr(perm),
        _ptr(active), _ptr(n_active), _ptr(y), _ptr(ws), ws.numel(), _stream(stream)))


def omnimoe_expert_forward_group_rows(desc, x, u, v, idx, gates, perm, active, n_active, y,
                                     ws=None, stream=None):
    if ws is None:
        ws = workspace(desc, STAGE_EXPERT_GROUP_ROWS, x.device)
    _check("omnimoe_expert_forward_group_rows", load_library().omnimoe_expert_forward_group_rows(
        ctypes.byref(desc), _ptr(x), _ptr(u), _ptr(v), _ptr(idx), _ptr(gates), _ptr(perm),
        _ptr(active), _ptr(n_active), _ptr(y), _ptr(ws), ws.numel(), _stream(stream)))


def omnimoe_expert_forward_scatter(desc, x, u, v, idx, gates, perm, y, ws=None, stream=None):
    if ws is None:
        ws = workspace(desc, STAGE_EXPERT_SCATTER, x.device)
    _check("omnimoe_expert_forward_scatter", load_library().omnimoe_expert_forward_scatter(
        ctypes.byref(desc), _ptr(x), _ptr(u), _ptr(v), _ptr(idx), _ptr(gates), _ptr(perm),
        _ptr(y), _ptr(ws), ws.numel(), _stream(stream)))


def omnimoe_expert_forward_token_centric(desc, x, u, v, idx, gates, y, stream=None):
    _check("omnimoe_expert_forward_token_centric",
           load_library().omnimoe_expert_forward_token_centric(
               ctypes.byref(desc), _ptr(x), _ptr(u), _ptr(v), _ptr(idx), _ptr(gates), _ptr(y),
               _stream(stream)))


def omnimoe_expert_backward(desc, x, u, v, idx, gates, perm, active_offsets, n_active, dy, dx,
                            du_rows, dv_rows, dgates, dscores, ws=None, stream=None):
    if ws is None:
        ws = workspace(desc, STAGE_EXPERT_BACKWARD, x.device)
    _check("omnimoe_expert_backward", load_library().omnimoe_expert_backward(
        ctypes.byref(desc), _ptr(x), _ptr(u), _ptr(v), _ptr(idx), _ptr(gates), _ptr(perm),
        _ptr(active_offsets), _ptr(n_active), _ptr(dy), _ptr(dx), _ptr(du_rows), _ptr(dv_rows),
        _ptr(dgates), _ptr(dscores), _ptr(ws), ws.numel(), _stream(stream)))


def omnimoe_route_backward(desc, x, keys_row, keys_col, idx, dscores, dx, dkeys_row, dkeys_col,
                           ws=None, stream=None):
    if ws is None:
        ws = workspace(desc, STAGE_ROUTE_BACKWARD, x.device)
    _check("omnimoe_route_backward", load_library().omnimoe_route_backward(
        ctypes.byref(desc), _ptr(x), _ptr(keys_row), _ptr(keys_col), _ptr(idx), _ptr(dscores),
        _ptr(dx), _ptr(dkeys_row), _ptr(dkeys_col), _ptr(ws), ws.numel(), _stream(stream)))


def omnimoe_layer_forward(desc, x, keys_row, keys_col, u, v, y, idx_out=None, gates_out=None,
                          ws=None, stream=None):
    if ws is None:
        ws = workspace(desc, STAGE_LAYER, x.device)
    _check("omnimoe_layer_forward", load_library().omnimoe_layer_forward(
        ctypes.byref(desc), _ptr(x), _ptr(keys_row), _ptr(keys_col), _ptr(u), _ptr(v), _ptr(y),
        _ptr(idx_out), _ptr(gates_out), _ptr(ws), ws.numel(), _stream(stream)))


NOALLOC_SCRATCH_BYTES = 64 * 1024 * 1024  # OMNIMOE_NOALLOC_SCRATCH_BYTES

# omnimoe_path_flag
PATH_SCHEDULE, PATH_GROUPED, PATH_SELECT_DOT, PATH_DENSE_SUM, PATH_DENSE_DOT = 1, 2, 4, 8, 16


def omnimoe_layer_path(desc):
    """The omnimoe_path_flag bits of the kernels omnimoe_layer_forward runs for desc."""
    out = ctypes.c_int32(0)
    _check("omnimoe_layer_path", load_library().omnimoe_layer_path(ctypes.byref(desc),
                                                                    ctypes.byref(out)))
    return out.value


def omnimoe_layer_forward_noalloc(desc, x, keys_row, keys_col, u, v, y, idx_out=None,
                                  gates_out=None, stream=None):
    _check("omnimoe_layer_forward_noalloc", load_library().omnimoe_layer_forward_noalloc(
        ctypes.byref(desc), _ptr(x), _ptr(keys_row), _ptr(keys_col), _ptr(u), _ptr(v), _ptr(y),
        _ptr(idx_out), _ptr(gates_out), _stream(stream)))


class Timer:
    """omnimoe_timer_*: per-kernel-group HIP event timing of omnimoe_layer_forward_timed."""

    def __init__(self, capacity: int):
        self._h = ctypes.c_void_p()
        _check("omnimoe_timer_create",
               load_library().omnimoe_timer_create(capacity, ctypes.byref(self._h)))

    def layer_forward(self, desc, x, keys_row, keys_col, u, v, y, ws, idx_out=None,
                      gates_out=None, stream=None):
        _check("omnimoe_layer_forward_timed", load_library().omnimoe_layer_forward_timed(
            ctypes.byref(desc), _ptr(x), _ptr(keys_row), _ptr(keys_col), _ptr(u), _ptr(v),
            _ptr(y), _ptr(idx_out), _ptr(gates_out), _ptr(ws), ws.numel(), _stream(stream),
            self._h))

    def read(self):
        """({kernel group: summed ms}, number of calls); clears the timer."""
        ms = (ctypes.c_float * len(KERNEL_NAMES))()
        n = ctypes.c_int32(0)
        _check("omnimoe_timer_read", load_library().omnimoe_timer_read(self._h, ms,
                                                                        ctypes.byref(n)))
        return dict(zip(KERNEL_NAMES, list(ms))), n.value

    def close(self):
        if self._h:
            load_library().omnimoe_timer_destroy(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
