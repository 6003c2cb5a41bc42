"""Seeded synthetic inputs for the atomic-expert layer (shared by the GPU path and the oracle).

The module draws numbers only; it holds none of the layer's arithmetic. The C generator
(``synth.c``) is counter based: element ``c`` of tensor ``stream`` under ``seed`` is a function
of ``(seed, stream, c)`` alone, so a token subsample or a set of expert rows can be drawn without
drawing the whole tensor.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass, replace
from typing import Dict, Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libsynth.so")
_lib = None

# Tensor streams under one seed.
STREAM_X, STREAM_KEYS_ROW, STREAM_KEYS_COL, STREAM_U, STREAM_V = 1, 2, 3, 4, 5
STREAM_PERM_ROW, STREAM_PERM_COL = 6, 7
STREAM_GATE = 8
STREAM_MLP_GU, STREAM_MLP_DOWN = 9, 10


def build(verbose: bool = False) -> str:
    """Compile ``synth.c`` into ``libsynth.so`` next to it."""
    import subprocess
    cmd = ["gcc", "-O2", "-std=c99", "-fPIC", "-shared", "-pthread",
           os.path.join(_HERE, "synth.c"), "-o", _LIB_PATH]
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
        lib.synth_fill_rows.restype = None
        lib.synth_fill_rows.argtypes = [
            ctypes.c_uint64, ctypes.c_uint32, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64,
            ctypes.c_int64, ctypes.c_void_p, ctypes.c_double, ctypes.c_int, ctypes.c_void_p,
            ctypes.c_int]
        lib.synth_stream_key.restype = ctypes.c_uint64
        lib.synth_stream_key.argtypes = [ctypes.c_uint64, ctypes.c_uint32]
        lib.synth_splitmix64_output.restype = ctypes.c_uint64
        lib.synth_splitmix64_output.argtypes = [ctypes.c_uint64, ctypes.c_uint64]
        _lib = lib
    return _lib


def default_threads() -> int:
    n = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else (os.cpu_count() or 1)
    return max(1, min(16, n))


def fill_rows(seed: int, stream: int, n_rows: int, row_len: int, scale: float, bf16: bool,
              rows: Optional[np.ndarray] = None, first_row: int = 0,
              row_scale: Optional[np.ndarray] = None, n_threads: Optional[int] = None) -> np.ndarray:
    """Draw ``n_rows`` x ``row_len`` values; bf16 results come back as uint16 bit patterns."""
    lib = _load()
    out = np.empty((n_rows, row_len), dtype=np.uint16 if bf16 else np.float32)
    rows_ptr = None
    if rows is not None:
        rows = np.ascontiguousarray(rows, dtype=np.int64)
        assert rows.shape == (n_rows,)
        rows_ptr = rows.ctypes.data
    rs_ptr = None
    if row_scale is not None:
        row_scale = np.ascontiguousarray(row_scale, dtype=np.float64)
        rs_ptr = row_scale.ctypes.data
    lib.synth_fill_rows(seed, stream, rows_ptr, first_row, n_rows, row_len, rs_ptr, float(scale),
                        1 if bf16 else 0, out.ctypes.data, n_threads or default_threads())
    return out


def bf16_bits_to_f32(a: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns (uint16) to float32."""
    out = np.empty(a.shape, np.uint32)
    np.left_shift(a, 16, out=out, dtype=np.uint32)
    return out.view(np.float32)


def as_f32(a: np.ndarray) -> np.ndarray:
    return bf16_bits_to_f32(a) if a.dtype == np.uint16 else np.ascontiguousarray(a, np.float32)


@dataclass(frozen=True)
class Workload:
    """Shapes and input recipe of one layer call.

    Sub-key tables are [H, n_rows, d_key] and [H, n_cols, d_key]; expert tables are [N, d] with
    N = n_rows * n_cols; x is [T, d]. ``skew_alpha`` > 0 scales sub-key row i of each half by
    c_i = ((pi(i) + 1) / n)^(-alpha), normalised to mean c^2 = 1, with pi a seeded permutation
    shared by all heads, which concentrates routing on a few experts.
    """
    name: str
    T: int
    d: int
    n_rows: int
    n_cols: int
    d_key: int
    H: int
    K: int
    dtype: str = "bf16"          # "f32" or "bf16"
    act: str = "gelu"            # "gelu" (erf form) or "silu"
    query_mode: str = "split"    # "split" or "shared"
    seed: int = 0
    skew_alpha: float = 0.0
    group_size: int = 1          # B of the schedule (active experts per execution group)

    @property
    def N(self) -> int:
        return self.n_rows * self.n_cols

    @property
    def M(self) -> int:
        return self.T * self.H * self.K

    @property
    def bf16(self) -> bool:
        return self.dtype == "bf16"

    @property
    def weight_scale(self) -> float:
        return 1.0 / float(np.sqrt(self.d))

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


# The layer shapes the implementation is checked and measured on.
WORKLOADS: Dict[str, Workload] = {
    # T=256, d=64, N=64^2, sub-keys 2 x 64 of dim 32, H=1, K=8, fp32.
    "tiny_f32": Workload("tiny_f32", T=256, d=64, n_rows=64, n_cols=64, d_key=32, H=1, K=8,
                         dtype="f32"),
    # T=4096, d=512, N=256^2, sub-keys 2 x 256 of dim 256, H=4, K=16, bf16.
    "small_bf16": Workload("small_bf16", T=4096, d=512, n_rows=256, n_cols=256, d_key=256, H=4,
                           K=16),
    # T=16384 (8 x 2048), d=2048, N=1024^2, sub-keys 2 x 1024 of dim 1024, H=8, K=16, bf16.
    "train_bf16": Workload("train_bf16", T=16384, d=2048, n_rows=1024, n_cols=1024, d_key=1024,
                           H=8, K=16),
    # As train_bf16, with sub-key rows scaled so that about 10% of the experts take about half
    # of the (token, expert) pairs: alpha = 0.080078125 routes 50.3% of the pairs to the top 10%
    # (tests/golden/calibrate_skew.py, result in tests/golden/skew_calibration.json).
    "skew_bf16": Workload("skew_bf16", T=16384, d=2048, n_rows=1024, n_cols=1024, d_key=1024,
                          H=8, K=16, skew_alpha=0.080078125),
    # One GPU's share of the training batch when tokens are split over eight GPUs with the
    # tables replicated (data-parallel): 2048 tokens against all 1024^2 experts.
    "dp8share_bf16": Workload("dp8share_bf16", T=2048, d=2048, n_rows=1024, n_cols=1024,
                              d_key=1024, H=8, K=16),
    # The paper's speed-benchmark configuration (Table A): d = 1024, N = 102,400 = 320^2, one
    # head, 4096 tokens, K = 512 and K = 4096 (reuse per active expert eta ~ 20 and ~ 160).
    "paper_k512_bf16": Workload("paper_k512_bf16", T=4096, d=1024, n_rows=320, n_cols=320,
                                d_key=512, H=1, K=512),
    "paper_k4096_bf16": Workload("paper_k4096_bf16", T=4096, d=1024, n_rows=320, n_cols=320,
                                 d_key=512, H=1, K=4096),
    # The paper's speed-benchmark sweeps (its benchmark table): the activated-expert budget
    # K = 512 .. 4096 at 1k tokens, and 1k .. 16k tokens at K = 512 (4k tokens is
    # paper_k512_bf16 above).
    "paper_t1k_k512_bf16": Workload("paper_t1k_k512_bf16", T=1024, d=1024, n_rows=320,
                                    n_cols=320, d_key=512, H=1, K=512),
    "paper_t1k_k1024_bf16": Workload("paper_t1k_k1024_bf16", T=1024, d=1024, n_rows=320,
                                     n_cols=320, d_key=512, H=1, K=1024),
    "paper_t1k_k2048_bf16": Workload("paper_t1k_k2048_bf16", T=1024, d=1024, n_rows=320,
                                     n_cols=320, d_key=512, H=1, K=2048),
    "paper_t1k_k4096_bf16": Workload("paper_t1k_k4096_bf16", T=1024, d=1024, n_rows=320,
                                     n_cols=320, d_key=512, H=1, K=4096),
    "paper_t2k_k512_bf16": Workload("paper_t2k_k512_bf16", T=2048, d=1024, n_rows=320,
                                    n_cols=320, d_key=512, H=1, K=512),
    "paper_t8k_k512_bf16": Workload("paper_t8k_k512_bf16", T=8192, d=1024, n_rows=320,
                                    n_cols=320, d_key=512, H=1, K=512),
    "paper_t16k_k512_bf16": Workload("paper_t16k_k512_bf16", T=16384, d=1024, n_rows=320,
                                     n_cols=320, d_key=512, H=1, K=512),
    # One decode step of a batch of 64, and a single token.
    "decode64_bf16": Workload("decode64_bf16", T=64, d=2048, n_rows=1024, n_cols=1024,
                              d_key=1024, H=8, K=16),
    "decode1_bf16": Workload("decode1_bf16", T=1, d=2048, n_rows=1024, n_cols=1024, d_key=1024,
                             H=8, K=16),
}


def seeded_permutation(seed: int, stream: int, n: int) -> np.ndarray:
    """pi with pi[i] = rank of the i-th SplitMix64 output of the stream among the n outputs."""
    lib = _load()
    key = lib.synth_stream_key(seed, stream)
    h = np.array([lib.synth_splitmix64_output(key, i + 1) for i in range(n)], dtype=np.uint64)
    order = np.argsort(h, kind="stable")
    pi = np.empty(n, dtype=np.int64)
    pi[order] = np.arange(n)
    return pi


def skew_row_scale(w: Workload, n: int, stream: int) -> Optional[np.ndarray]:
    """Per-row scale c_i of one sub-key half ([H * n] entries, the same for every head)."""
    if w.skew_alpha <= 0.0:
        return None
    pi = seeded_permutation(w.seed, stream, n)
    c = ((pi + 1.0) / n) ** (-w.skew_alpha)
    c = c / np.sqrt(np.mean(c * c))
    return np.tile(c, w.H)


def make_x(w: Workload, tokens: Optional[Sequence[int]] = None, n_threads=None) -> np.ndarray:
    if tokens is None:
        return fill_rows(w.seed, STREAM_X, w.T, w.d, 1.0, w.bf16, n_threads=n_threads)
    tok = np.asarray(tokens, dtype=np.int64)
    return fill_rows(w.seed, STREAM_X, len(tok), w.d, 1.0, w.bf16, rows=tok, n_threads=n_threads)


def make_keys(w: Workload, n_threads=None):
    """(keys_row [H, n_rows, d_key], keys_col [H, n_cols, d_key])."""
    kr = fill_rows(w.seed, STREAM_KEYS_ROW, w.H * w.n_rows, w.d_key, w.weight_scale, w.bf16,
                   row_scale=skew_row_scale(w, w.n_rows, STREAM_PERM_ROW), n_threads=n_threads)
    kc = fill_rows(w.seed, STREAM_KEYS_COL, w.H * w.n_cols, w.d_key, w.weight_scale, w.bf16,
                   row_scale=skew_row_scale(w, w.n_cols, STREAM_PERM_COL), n_threads=n_threads)
    return kr.reshape(w.H, w.n_rows, w.d_key), kc.reshape(w.H, w.n_cols, w.d_key)


def make_expert_rows(w: Workload, which: str, rows: Optional[Sequence[int]] = None,
                     n_threads=None) -> np.ndarray:
    """Rows of the down (``"u"``) or up (``"v"``) expert table; all N rows when rows is None."""
    stream = {"u": STREAM_U, "v": STREAM_V}[which]
    if rows is None:
        return fill_rows(w.seed, stream, w.N, w.d, w.weight_scale, w.bf16, n_threads=n_threads)
    r = np.asarray(rows, dtype=np.int64)
    return fill_rows(w.seed, stream, len(r), w.d, w.weight_scale, w.bf16, rows=r,
                     n_threads=n_threads)


def make_gate_table(w: Workload, n_threads=None) -> np.ndarray:
    """Gating vectors of a dense router over all N experts, [H, N, d] ~ N(0, 1/d)."""
    g = fill_rows(w.seed, STREAM_GATE, w.H * w.N, w.d, w.weight_scale, w.bf16,
                  n_threads=n_threads)
    return g.reshape(w.H, w.N, w.d)


def make_mlp_weights(w: Workload, d_ff: int, n_threads=None):
    """Shared SwiGLU branch: (w_gu [2 d_ff, d] ~ N(0, 1/d), w_down [d, d_ff] ~ N(0, 1/d_ff))."""
    gu = fill_rows(w.seed, STREAM_MLP_GU, 2 * d_ff, w.d, w.weight_scale, w.bf16,
                   n_threads=n_threads)
    down = fill_rows(w.seed, STREAM_MLP_DOWN, w.d, d_ff, 1.0 / float(np.sqrt(d_ff)), w.bf16,
                     n_threads=n_threads)
    return gu, down


def make_inputs(w: Workload, n_threads=None) -> Dict[str, np.ndarray]:
    """All tensors of one layer call, in the layer's storage dtype (bf16 as uint16 bits)."""
    kr, kc = make_keys(w, n_threads)
    return {
        "x": make_x(w, n_threads=n_threads),
        "keys_row": kr,
        "keys_col": kc,
        "u": make_expert_rows(w, "u", n_threads=n_threads),
        "v": make_expert_rows(w, "v", n_threads=n_threads),
    }
