"""The routing comparison the GPU parity tests use, exercised on the CPU.

A stand-in for the GPU rounds the oracle's fp64 logits to fp32 and selects on them (as the GPU
does on its own fp32 logits); that routing must pass. Planted mistakes in it (the best cell
dropped, two picks swapped, a pick from below the near-tie band, a repeated id) must fail.
"""
import numpy as np
import pytest

import oracle
import synth
from gpu_support import certify_positions, compare_routing, gate_bound_check


def _case(T=64, n=64, K=16, H=2, seed=0, ties=False):
    w = synth.Workload("chk", T=T, d=128, n_rows=n, n_cols=n, d_key=64, H=H, K=K)
    rng = np.random.default_rng(seed)
    if ties:  # integer logits: many exact ties in the grid
        sr = rng.integers(-4, 5, (T, H, n)).astype(np.float64)
        sc = rng.integers(-4, 5, (T, H, n)).astype(np.float64)
    else:
        sr = rng.standard_normal((T, H, n))
        sc = rng.standard_normal((T, H, n))
    hs = np.concatenate([sr, sc], axis=-1).astype(np.float32)
    delta = float(np.abs(hs.astype(np.float64) - np.concatenate([sr, sc], -1)).max())
    idx, _, g, _ = oracle.select_f32(oracle.desc(w), hs, oracle.CARTESIAN)
    return w, sr, sc, idx, g.astype(np.float32), max(delta, 1e-300)


@pytest.mark.parametrize("ties", [False, True])
@pytest.mark.parametrize("K", [1, 16, 200])
def test_fp32_routing_passes(K, ties):
    w, sr, sc, idx, g, delta = _case(K=K, ties=ties)
    unc, rows, npos = compare_routing(w, idx, sr, sc, delta)
    assert npos == w.T * w.H * K and 0 <= unc <= npos
    if not ties:
        assert unc < npos  # most positions are certified with Gaussian logits
    gate_bound_check(g, sr, sc, idx, w.n_cols, delta, 1e-5)


def test_certified_positions_of_a_hand_row():
    # one row, grid 1 x 5: scores 5, 4, 4, 2, 1 (ids 0..4); K = 3, delta tiny
    w = synth.Workload("hand", T=1, d=8, n_rows=1, n_cols=5, d_key=4, H=1, K=3)
    sr = np.zeros((1, 1, 1))
    sc = np.array([5.0, 4.0, 4.0, 2.0, 1.0]).reshape(1, 1, 5)
    ref, sel, cert = certify_positions(w, sr, sc, 1e-9)
    assert ref.reshape(-1).tolist() == [0, 1, 2]
    assert sel.reshape(-1).tolist() == [5.0, 4.0, 4.0, 2.0]
    assert cert.reshape(-1).tolist() == [True, False, False]
    # the tied pair may come in either order
    compare_routing(w, np.array([0, 2, 1]).reshape(1, 1, 3), sr, sc, 1e-9)
    with pytest.raises(AssertionError):
        compare_routing(w, np.array([1, 0, 2]).reshape(1, 1, 3), sr, sc, 1e-9)


def _plant(mut):
    w, sr, sc, idx, g, delta = _case(K=16)
    bad = idx.copy()
    mut(w, bad, sr, sc)
    with pytest.raises(AssertionError):
        compare_routing(w, bad, sr, sc, delta)


def test_dropped_best_cell_fails():
    def mut(w, b, sr, sc):  # replace row 0's best pick by an unpicked cell
        b[0, 0, 0] = next(e for e in range(w.N) if e not in set(b[0, 0].tolist()))
    _plant(mut)


def test_swapped_order_fails():
    def mut(w, b, sr, sc):
        b[3, 1, [0, 5]] = b[3, 1, [5, 0]]
    _plant(mut)


def test_pick_below_band_fails():
    def mut(w, b, sr, sc):  # last pick replaced by the row's worst cell
        s = sr[5, 0][:, None] + sc[5, 0][None, :]
        b[5, 0, -1] = int(np.argmin(s))
    _plant(mut)


def test_repeated_id_fails():
    def mut(w, b, sr, sc):
        b[7, 1, 9] = b[7, 1, 8]
    _plant(mut)


def test_gate_check_catches_wrong_gate():
    w, sr, sc, idx, g, delta = _case(K=16)
    g = g.copy()
    g[2, 0, 3] *= 1.001
    with pytest.raises(AssertionError):
        gate_bound_check(g, sr, sc, idx, w.n_cols, delta, 1e-5)
