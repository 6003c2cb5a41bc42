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


def backward_error_bounds(x, u, v, idx, g, dy, f_act, f_dact, dd_act_max=0.8,
                          unit=2.0 ** -23):
    """First-order bounds on the fp32 errors of the expert backward, element by element.

    h_p = x_t . u_e and da_p = dy_t . v_e are fp32 dot products of length d, each within
    2 gamma_d sum |.||.| (Higham, Thm 3.1); the errors propagate through a = g act(h),
    dh = da g act'(h) and dgates = da act(h) (|act''| <= dd_act_max), and the fp32 sums of dx,
    du, dv and of the softmax term each add gamma_n of their absolute terms. A small multiple
    of the unit roundoff covers each rounded product and activation. Returns arrays shaped like
    the outputs: dx [T, d], du / dv [A, d] over the active experts in ascending id order,
    dgates and dscores [T, H, K]. f_act and f_dact evaluate act and act' in fp64.
    """
    T, D = x.shape
    H, K = idx.shape[1], idx.shape[2]
    hk = H * K
    M = T * hk

    def gam(n):
        return n * unit / (1 - n * unit)

    ii = idx.reshape(-1).astype(np.int64)
    t = np.arange(M) // hk
    x64, u64, v64, dy64 = (np.asarray(a, np.float64) for a in (x, u, v, dy))
    gg = np.asarray(g, np.float64).reshape(-1)
    h = np.einsum("pd,pd->p", x64[t], u64[ii])
    da = np.einsum("pd,pd->p", dy64[t], v64[ii])
    bh = 2 * gam(D) * np.einsum("pd,pd->p", np.abs(x64[t]), np.abs(u64[ii]))
    bda = 2 * gam(D) * np.einsum("pd,pd->p", np.abs(dy64[t]), np.abs(v64[ii]))
    act, dact = f_act(h), f_dact(h)
    a, dh, dg = gg * act, da * gg * dact, da * act
    ba = np.abs(gg) * (np.abs(dact) + dd_act_max * bh) * bh + 8 * unit * np.abs(a)
    bdh = (np.abs(gg) * (np.abs(dact) * bda + np.abs(da) * dd_act_max * bh)
           + 8 * unit * np.abs(dh))
    bdg = (np.abs(act) * bda + np.abs(da) * (np.abs(dact) + dd_act_max * bh) * bh
           + 8 * unit * np.abs(dg))
    out = {}
    dx = np.zeros((T, D))
    for s_ in range(hk):
        p = np.arange(T) * hk + s_
        dx += bdh[p, None] * np.abs(u64[ii[p]]) + gam(hk) * np.abs(dh[p, None] * u64[ii[p]])
    out["dx"] = dx
    active = np.unique(ii)
    rows = np.searchsorted(active, ii)
    cnt = np.bincount(rows, minlength=active.size)
    ge = gam(np.maximum(cnt, 1))[:, None]
    for name, bterm, val, other in (("du", bdh, dh, x64[t]), ("dv", ba, a, dy64[t])):
        b = np.zeros((active.size, D))
        ab = np.zeros((active.size, D))
        np.add.at(b, rows, bterm[:, None] * np.abs(other))
        np.add.at(ab, rows, np.abs(val[:, None] * other))
        out[name] = b + ge * ab
    out["dgates"] = bdg.reshape(T, H, K)
    g3, dg3, bdg3 = gg.reshape(T, H, K), dg.reshape(T, H, K), bdg.reshape(T, H, K)
    srow = (np.abs(g3) * bdg3).sum(axis=-1, keepdims=True) + gam(K) * np.abs(g3 * dg3).sum(
        axis=-1, keepdims=True)
    ds = g3 * (dg3 - (g3 * dg3).sum(axis=-1, keepdims=True))
    out["dscores"] = np.abs(g3) * (bdg3 + srow) + 8 * unit * np.abs(ds)
    return out


def _act64(kind: int, h: np.ndarray) -> np.ndarray:
    from scipy.special import erfc
    if kind == 1:
        return h / (1.0 + np.exp(-h))
    return 0.5 * h * erfc(-h / np.sqrt(2.0))


def grouped_gap_bound(f, idx, g, d: int, act_kind: int) -> np.ndarray:
    """Element-wise bound on |y_a - y_b| for two expert computations that differ only in the
    order in which each x_t . u_e is summed in fp32 (per task, as in the scheduled kernel, or
    as dense tiles on the matrix cores): each dot lies within gamma_d sum |x u| of the exact
    value (Higham, Thm. 3.1), |act'| <= 1.13 for GELU (1.10 for SiLU), the activation and the
    gate multiply add a few ulp, and both results then go through the same fp32 slot-order sum
    of a * v, each within gamma_{n+1} sum |a| |v| of its exact value."""
    x, u, v = f["x"], f["u"], f["v"]
    T = x.shape[0]
    e = idx.reshape(T, -1)
    gg = np.abs(g.reshape(T, -1)).astype(np.float64)
    n = e.shape[1]

    def gam(k):
        return k * 2.0 ** -24 / (1 - k * 2.0 ** -24)

    out = np.empty((T, d))
    chunk = max(1, (1 << 23) // max(1, n * d))
    for t0 in range(0, T, chunk):
        xs = np.asarray(x[t0:t0 + chunk], dtype=np.float64)
        es, gs = e[t0:t0 + chunk], gg[t0:t0 + chunk]
        U = np.asarray(u[es], dtype=np.float64)
        h = np.einsum("cd,cnd->cn", xs, U, optimize=True)
        S = np.einsum("cd,cnd->cn", np.abs(xs), np.abs(U), optimize=True)
        del U
        a = gs * np.abs(_act64(act_kind, h))
        da = gs * 1.13 * 2 * gam(d) * S + 16 * 2.0 ** -24 * a
        V = np.abs(np.asarray(v[es], dtype=np.float64))
        out[t0:t0 + chunk] = np.einsum("cn,cnd->cd", da + 2.02 * gam(n + 1) * a, V,
                                       optimize=True)
    return out + 1e-30
