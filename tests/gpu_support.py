"""Helpers for the GPU parity tests: upload seeded inputs, run the library, compare with the oracle."""
from __future__ import annotations

import numpy as np

import oracle
import synth

F32_TOL = 1e-5    # max relative error, fp32 layer
BF16_TOL = 2e-2   # max relative error, bf16 layer (fp32 accumulation)
GATE_TOL = 1e-5   # gates are computed in fp32 for both storage types


def tol(w):
    return BF16_TOL if w.bf16 else F32_TOL


def to_dev(a: np.ndarray):
    """numpy -> cuda tensor; uint16 arrays are bf16 bit patterns."""
    import torch
    if a.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda().view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def upload(inputs: dict) -> dict:
    return {k: to_dev(v) for k, v in inputs.items()}


def row_rel_err(got: np.ndarray, ref: np.ndarray) -> np.ndarray:
    """Per row: max |got - ref| / max(max |ref|, 1e-30)."""
    got = got.reshape(ref.shape[0], -1).astype(np.float64)
    ref = ref.reshape(ref.shape[0], -1)
    den = np.maximum(np.abs(ref).max(axis=1), 1e-30)
    return np.abs(got - ref).max(axis=1) / den


def higham_bound(xq: np.ndarray, keys: np.ndarray, u: float = 2.0 ** -23) -> np.ndarray:
    """2 gamma_n sum |x||k| bound on an fp32-accumulated dot of length n (Higham, Thm 3.1)."""
    n = xq.shape[-1]
    gamma = n * u / (1 - n * u)
    return 2 * gamma * np.einsum("tm,hjm->thj", np.abs(xq).astype(np.float64),
                                 np.abs(keys).astype(np.float64), optimize=True)


def grid_scores(sr_row, sc_row, ids, n_cols):
    ids = np.asarray(ids)
    return sr_row[ids // n_cols] + sc_row[ids % n_cols]


def certify_rows(w, sr, sc, delta):
    """Oracle top-(K+1) scores per (t, h) row; returns (certified mask, kth score, margin).

    A row is certified when every gap between consecutive scores among its top K+1 exceeds
    4 * delta (each half-logit is within delta, so a score is within 2 delta and a difference
    within 4 delta): then the GPU must reproduce the list exactly, order included.
    """
    dsc = oracle.desc(w, T=sr.shape[0], K=min(w.K + 1, w.N))
    _, sel, _, _ = oracle.select(dsc, sr, sc, oracle.CARTESIAN)
    gaps = -np.diff(sel, axis=-1)
    cert = gaps.min(axis=-1) > 4 * delta
    return cert, sel[..., w.K - 1]


def compare_routing(w, gpu_idx, ref_idx, sr, sc, delta):
    """Bit-exact idx on certified rows; on the others every GPU pick must score within
    4 delta of the K-th best. Returns the number of uncertified rows."""
    cert, kth = certify_rows(w, sr, sc, delta)
    g = gpu_idx.reshape(cert.shape + (w.K,))
    r = ref_idx.reshape(cert.shape + (w.K,))
    bad = cert & np.any(g != r, axis=-1)
    assert not bad.any(), f"{int(bad.sum())} certified rows differ, first at {np.argwhere(bad)[0]}"
    for t, h in np.argwhere(~cert):
        s = grid_scores(sr[t, h], sc[t, h], g[t, h], w.n_cols)
        assert np.all(s >= kth[t, h] - 4 * delta), (t, h)
        assert len(set(g[t, h].tolist())) == w.K
    return int((~cert).sum())
