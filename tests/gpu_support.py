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


def certify_positions(w, sr, sc, delta):
    """Oracle top-K list per (t, h) row and which of its positions the GPU must reproduce.

    Each GPU half-logit lies within delta of the oracle's fp64 value, so each GPU cell score
    lies within 2 delta of its exact S and any comparison of two scores within 4 delta. A list
    position k is certified when the exact scores at ranks k - 1 and k + 1 (rank K included,
    the first cell outside the list) both differ from rank k's by more than 4 delta: every
    cell ranked above k then outscores it on the GPU too and every cell ranked below it scores
    less, so the GPU must put the oracle's cell k at position k. Returns (oracle idx [.., K],
    oracle scores of ranks 0..K [.., K + 1] (rank K is -inf when K = N), certified [.., K]).
    """
    K1 = min(w.K + 1, w.N)
    dsc = oracle.desc(w, T=sr.shape[0], K=K1)
    # (fp64 logits: their sums round at 1e-16 relative, far inside the 4 delta margins)
    ref1, sel1, _, _ = oracle.select(dsc, sr, sc, oracle.CARTESIAN)
    if K1 == w.K:  # every cell is selected: nothing follows rank K - 1
        sel1 = np.concatenate([sel1, np.full(sel1.shape[:-1] + (1,), -np.inf)], axis=-1)
    ref = ref1[..., :w.K]
    gap = sel1[..., :-1] - sel1[..., 1:]          # gap[k] = S_k - S_{k+1}, k < K
    inf = np.full(gap.shape[:-1] + (1,), np.inf)
    before = np.concatenate([inf, gap[..., :-1]], axis=-1)
    cert = (before > 4 * delta) & (gap > 4 * delta)
    return ref, sel1, cert


def compare_routing(w, gpu_idx, sr, sc, delta):
    """GPU routing [T, H, K] against the fp64 oracle on logits sr, sc (see certify_positions).

    * every certified position holds the oracle's cell (whole rows bit-exact when certified);
    * every row holds K distinct ids in [0, N);
    * every pick scores at least S_(K-1) - 4 delta (nothing from outside the near-tie band);
    * every cell of the oracle list scoring above S_(K-1) + 4 delta is picked (containment);
    * picks are in non-increasing exact score up to 4 delta (order).
    Returns (uncertified positions, rows with an uncertified position, total positions)."""
    ref, sel1, cert = certify_positions(w, sr, sc, delta)
    g = np.asarray(gpu_idx).reshape(ref.shape).astype(np.int64)
    bad = cert & (g != ref)
    assert not bad.any(), (f"{int(bad.sum())} certified positions differ, first at "
                           f"{np.argwhere(bad)[0].tolist()}")
    assert g.min() >= 0 and g.max() < w.N
    srt = np.sort(g, axis=-1)
    assert np.all(np.diff(srt, axis=-1) > 0), "a row repeats an id"
    s_g = np.take_along_axis(sr, g // w.n_cols, axis=-1) + np.take_along_axis(sc, g % w.n_cols,
                                                                            axis=-1)
    kth = sel1[..., w.K - 1:w.K]
    low = s_g < kth - 4 * delta
    assert not low.any(), f"pick below the near-tie band at {np.argwhere(low)[0].tolist()}"
    assert np.all(s_g[..., :-1] >= s_g[..., 1:] - 4 * delta), "picks out of order"
    # containment: oracle cells above the band must be picked (search in row-tagged sorted ids)
    rows = np.arange(g.shape[0] * g.shape[1], dtype=np.int64).reshape(g.shape[:2] + (1,))
    tagged = np.sort((rows * w.N + g).reshape(-1))
    need = sel1[..., :w.K] > kth + 4 * delta
    want = (rows * w.N + ref)[need]
    pos = np.searchsorted(tagged, want)
    hit = (pos < tagged.size) & (tagged[np.minimum(pos, tagged.size - 1)] == want)
    assert hit.all(), f"{int((~hit).sum())} cells above the near-tie band are missing"
    return int((~cert).sum()), int((~cert.all(axis=-1)).sum()), int(cert.size)


def gate_bound_check(gpu_g, sr, sc, gpu_idx, n_cols, delta, rtol):
    """GPU gates against the fp64 softmax of the exact scores of the GPU's own picks: each
    score is within 2 delta, so each log-gate within 4 delta, plus the fp32 rounding rtol."""
    g = np.asarray(gpu_idx).astype(np.int64)
    s = np.take_along_axis(sr, g // n_cols, axis=-1) + np.take_along_axis(sc, g % n_cols, axis=-1)
    e = np.exp(s - s.max(axis=-1, keepdims=True))
    ref = e / e.sum(axis=-1, keepdims=True)
    tolr = np.expm1(4 * delta) + rtol
    err = np.abs(gpu_g - ref)
    assert np.all(err <= tolr * ref + 1e-7), f"gate error {float((err / ref).max()):.3e}"
    return float((err / ref).max())


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
