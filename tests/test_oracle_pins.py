"""Pins of the oracle against facts fixed by the paper and by mathematics, not by the oracle itself.

Each test names the plausible mistake it would catch. Hand-worked fixtures live in tests/golden/.
"""
import json
import math
import os

import numpy as np
import pytest

import oracle
import synth

GELU, SILU = 0, 1


class Shape:
    def __init__(self, **kw):
        self.act = "gelu"
        self.query_mode = "split"
        self.group_size = 1
        self.__dict__.update(kw)


def _load(golden_dir, name):
    with open(os.path.join(golden_dir, name)) as f:
        return json.load(f)


# ---------------------------------------------------------------- input generator

def test_splitmix64_published_outputs():
    # First four outputs of SplitMix64 seeded with 0 (Steele, Lea, Flood 2014 reference code).
    lib = synth._load()
    want = [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F, 0xF88BB8A8724C81EC]
    assert [lib.synth_splitmix64_output(0, n) for n in range(1, 5)] == want


def test_synth_is_counter_based_and_normalish():
    w = synth.WORKLOADS["small_bf16"]
    full = synth.fill_rows(0, synth.STREAM_U, 64, 512, 1.0, False)
    rows = synth.fill_rows(0, synth.STREAM_U, 3, 512, 1.0, False, rows=np.array([5, 0, 63]))
    assert np.array_equal(rows, full[[5, 0, 63]])
    assert abs(full.mean()) < 0.02 and abs(full.std() - 1.0) < 0.02
    b = synth.fill_rows(0, synth.STREAM_U, 64, 512, 1.0, True)
    # bf16 bits are the round-to-nearest-even of the float draw
    f = synth.bf16_bits_to_f32(b)
    assert np.all(np.abs(f - full) <= np.abs(full) * 2.0 ** -8)
    x1 = synth.make_x(w.with_(T=8))
    x2 = synth.make_x(w, tokens=[3, 7])
    assert np.array_equal(x1[[3, 7]], x2)


def test_skew_scale_recipe(golden_dir):
    # Row scales: a power law in the seeded rank, normalised to mean square 1, same for every
    # head; the calibrated exponent is the one the workload table carries.
    w = synth.WORKLOADS["skew_bf16"]
    c = synth.skew_row_scale(w, w.n_rows, synth.STREAM_PERM_ROW)
    assert c.shape == (w.H * w.n_rows,)
    one = c[: w.n_rows]
    np.testing.assert_allclose(np.mean(one ** 2), 1.0, rtol=1e-12)
    assert np.array_equal(np.tile(one, w.H), c)
    pi = synth.seeded_permutation(w.seed, synth.STREAM_PERM_ROW, w.n_rows)
    assert np.array_equal(np.sort(pi), np.arange(w.n_rows))
    assert np.all(np.diff(one[np.argsort(pi)]) < 0)  # rank 0 is the hottest row
    cal = _load(golden_dir, "skew_calibration.json")
    assert cal["chosen"]["alpha"] == w.skew_alpha
    assert abs(cal["chosen"]["top10_share"] - 0.5) <= cal["tolerance"]
    assert synth.skew_row_scale(synth.WORKLOADS["train_bf16"], 1024, 6) is None


# ---------------------------------------------------------------- activation (Eq. 4)

def test_activation_values(golden_dir):
    g = _load(golden_dir, "activation_values.json")
    phi = {float(k): v for k, v in g["phi"].items()}
    for z, p in phi.items():
        assert oracle.act(GELU, z) == pytest.approx(z * p, rel=1e-15, abs=1e-16)
        assert oracle.act(GELU, -z) == pytest.approx(-z * (1.0 - p), rel=1e-13, abs=1e-16)
    assert oracle.act(GELU, 0.0) == 0.0
    for z in np.linspace(-6, 6, 49):
        assert oracle.act(GELU, z) - oracle.act(GELU, -z) == pytest.approx(z, abs=1e-15)
    assert oracle.act(SILU, 1.0) == pytest.approx(1.0 * g["logistic"]["1"], rel=1e-15)
    assert oracle.act(SILU, -2.0) == pytest.approx(-2.0 * g["logistic"]["-2"], rel=1e-15)


# ---------------------------------------------------------------- half-scores (Eq. 9)

@pytest.mark.parametrize("mode", ["split", "shared"])
def test_half_scores_are_matrix_products(mode):
    # Catches a dropped term, a wrong query offset and a transposed key operand.
    rng = np.random.default_rng(1)
    s = Shape(T=7, d=24, n_rows=5, n_cols=6, d_key=9, H=3, K=4, query_mode=mode)
    x = rng.standard_normal((s.T, s.d)).astype(np.float32)
    kr = rng.standard_normal((s.H, s.n_rows, s.d_key)).astype(np.float32)
    kc = rng.standard_normal((s.H, s.n_cols, s.d_key)).astype(np.float32)
    sr, sc = oracle.half_scores(oracle.desc(s), x, kr, kc)
    c0 = s.d_key if mode == "split" else 0
    xd = x.astype(np.float64)
    want_r = np.einsum("tm,him->thi", xd[:, :s.d_key], kr.astype(np.float64))
    want_c = np.einsum("tm,hjm->thj", xd[:, c0:c0 + s.d_key], kc.astype(np.float64))
    np.testing.assert_allclose(sr, want_r, rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(sc, want_c, rtol=1e-13, atol=1e-13)


# ---------------------------------------------------------------- router (Eq. 1, 2, 11)

@pytest.mark.parametrize("method", [oracle.BRUTE, oracle.CARTESIAN, oracle.LOGSOFTMAX_BRUTE])
def test_router_hand_examples(golden_dir, method):
    # Catches a transposed id map (j * n_rows + i), a reversed tie rule and unnormalised gates.
    for case in _load(golden_dir, "router_hand.json")["cases"]:
        s = Shape(T=1, **{k: case[k] for k in ("d", "n_rows", "n_cols", "d_key", "H", "K")})
        s.query_mode = case.get("query_mode", "split")
        dsc = oracle.desc(s)
        sr, sc = oracle.half_scores(dsc, np.array(case["x"], np.float32),
                                    np.array(case["keys_row"], np.float32),
                                    np.array(case["keys_col"], np.float32))
        if "sr" in case:
            assert sr.ravel().tolist() == case["sr"] and sc.ravel().tolist() == case["sc"]
        idx, sel, g, _ = oracle.select(dsc, sr, sc, method)
        want_idx = np.array(case["idx"]).reshape(s.H, s.K)
        assert np.array_equal(idx.reshape(s.H, s.K), want_idx), case["name"]
        ex = np.array(case["gate_exponents"], np.float64).reshape(s.H, s.K)
        want_g = np.exp(ex) / np.exp(ex).sum(axis=1, keepdims=True)
        np.testing.assert_allclose(g.reshape(s.H, s.K), want_g, rtol=1e-14)
        if method != oracle.LOGSOFTMAX_BRUTE:
            assert np.array_equal(sel.reshape(s.H, s.K),
                                  np.array(case["sel"], np.float64).reshape(s.H, s.K))


def _brute_topk_lexsort(S, K):
    """Top-K of a flat score vector by (S desc, id asc) with numpy's lexsort."""
    n = np.arange(S.size)
    order = np.lexsort((n, -S))
    return order[:K]


def test_cartesian_equals_bruteforce_on_tie_heavy_grids():
    # The Cartesian candidate set (a+1)(b+1) <= K must give exactly the brute-force top-K,
    # in the same order, including heavy ties (integer-valued logits).
    rng = np.random.default_rng(2)
    trials = 0
    for nr in range(1, 11):
        for nc in range(1, 11):
            N = nr * nc
            for K in sorted({k for k in (1, 2, 3, 5, 8, 13, N) if k <= N}):
                s = Shape(T=6, d=2, n_rows=nr, n_cols=nc, d_key=1, H=1, K=K)
                dsc = oracle.desc(s)
                sr = rng.integers(-2, 3, size=(6, 1, nr)).astype(np.float64)
                sc = rng.integers(-2, 3, size=(6, 1, nc)).astype(np.float64)
                i_b, s_b, g_b, _ = oracle.select(dsc, sr, sc, oracle.BRUTE, n_threads=1)
                i_c, s_c, g_c, inexact = oracle.select(dsc, sr, sc, oracle.CARTESIAN, n_threads=1)
                assert inexact == 0
                assert np.array_equal(i_b, i_c), (nr, nc, K)
                assert np.array_equal(g_b, g_c)
                for t in range(6):
                    S = (sr[t, 0][:, None] + sc[t, 0][None, :]).ravel()
                    assert np.array_equal(i_b[t, 0], _brute_topk_lexsort(S, K))
                trials += 1
    assert trials > 500


def test_cartesian_equals_bruteforce_float32_scores():
    rng = np.random.default_rng(3)
    s = Shape(T=200, d=2, n_rows=32, n_cols=16, d_key=1, H=2, K=24)
    dsc = oracle.desc(s)
    hs = rng.standard_normal((s.T, s.H, s.n_rows + s.n_cols)).astype(np.float32)
    i_b, _, g_b, _ = oracle.select_f32(dsc, hs, oracle.BRUTE)
    i_c, _, g_c, inexact = oracle.select_f32(dsc, hs, oracle.CARTESIAN)
    assert inexact == 0  # sums of two float32 values are exact in double
    assert np.array_equal(i_b, i_c)
    np.testing.assert_array_equal(g_b, g_c)


def test_single_row_grid_is_plain_topk_over_columns():
    # n_rows = 1: the grid is one row, so the router is an ordinary top-K of the column logits.
    rng = np.random.default_rng(4)
    s = Shape(T=50, d=2, n_rows=1, n_cols=40, d_key=1, H=1, K=11)
    dsc = oracle.desc(s)
    sr = np.zeros((50, 1, 1))
    sc = np.round(rng.standard_normal((50, 1, 40)), 1)  # rounded: ties are common
    idx, _, _, _ = oracle.select(dsc, sr, sc, oracle.CARTESIAN)
    for t in range(50):
        want = np.argsort(-sc[t, 0], kind="stable")[:11]
        assert np.array_equal(idx[t, 0], want)


def test_logsoftmax_does_not_change_selection_or_gates():
    # Eq. 10 subtracts a per-half constant: same set, same order, same gates (to rounding).
    rng = np.random.default_rng(5)
    s = Shape(T=64, d=2, n_rows=16, n_cols=16, d_key=1, H=2, K=16)
    dsc = oracle.desc(s)
    sr = rng.standard_normal((64, 2, 16)) * 3
    sc = rng.standard_normal((64, 2, 16)) * 3
    i_raw, _, g_raw, _ = oracle.select(dsc, sr, sc, oracle.BRUTE)
    i_lsm, _, g_lsm, _ = oracle.select(dsc, sr, sc, oracle.LOGSOFTMAX_BRUTE)
    assert np.array_equal(i_raw, i_lsm)
    np.testing.assert_allclose(g_raw, g_lsm, rtol=1e-12)


def test_gate_properties():
    rng = np.random.default_rng(6)
    s = Shape(T=100, d=2, n_rows=20, n_cols=30, d_key=1, H=3, K=12)
    dsc = oracle.desc(s)
    sr = rng.standard_normal((100, 3, 20))
    sc = rng.standard_normal((100, 3, 30))
    idx, sel, g, _ = oracle.select(dsc, sr, sc, oracle.CARTESIAN)
    np.testing.assert_allclose(g.sum(-1), 1.0, rtol=1e-14)
    assert np.all(np.diff(g, axis=-1) <= 0)
    assert np.all(np.diff(sel, axis=-1) <= 0)
    # every row's ids are distinct
    assert all(len(set(r)) == 12 for r in idx.reshape(-1, 12).tolist())
    # K = 1: one expert with gate 1
    _, _, g1, _ = oracle.select(oracle.desc(s, K=1), sr, sc, oracle.CARTESIAN)
    assert np.all(g1 == 1.0)


def test_zero_input_selects_first_ids():
    # x = 0: every cell scores 0, so the lowest K ids win with equal gates 1/K.
    w = synth.WORKLOADS["tiny_f32"]
    dsc = oracle.desc(w, T=3)
    kr, kc = synth.make_keys(w)
    sr, sc = oracle.half_scores(dsc, np.zeros((3, w.d), np.float32), kr, kc)
    idx, _, g, _ = oracle.select(dsc, sr, sc, oracle.CARTESIAN)
    assert np.array_equal(idx, np.broadcast_to(np.arange(w.K), idx.shape))
    np.testing.assert_allclose(g, 1.0 / w.K, rtol=1e-15)


# ---------------------------------------------------------------- schedule (Eq. 12, 13)

@pytest.mark.parametrize("B", [1, 2, 7])
def test_schedule_is_stable_sort_by_group(B):
    # Catches an unstable placement, a wrong group rank and off-by-one offsets.
    rng = np.random.default_rng(7)
    s = Shape(T=300, d=2, n_rows=8, n_cols=9, d_key=1, H=2, K=5, group_size=B)
    dsc = oracle.desc(s)
    N = 72
    idx = np.stack([rng.permutation(N)[:5] for _ in range(600)]).astype(np.int32)
    idx[idx == 13] = 14  # leave an id unused
    idx = np.stack([np.unique(r)[:5] if len(np.unique(r)) >= 5 else r for r in idx]).astype(
        np.int32)
    perm, active, off, dense = oracle.schedule(dsc, idx)
    flat = idx.ravel()
    assert np.array_equal(active, np.unique(flat))
    rank = np.searchsorted(active, flat)
    want = np.argsort(rank // B, kind="stable")
    assert np.array_equal(perm, want)
    counts = np.bincount(flat, minlength=N)
    assert np.array_equal(off, np.concatenate([[0], np.cumsum(counts[active])]))
    assert np.array_equal(dense, np.concatenate([[0], np.cumsum(counts)]))
    assert off[-1] == flat.size == dense[-1]


def test_schedule_invariants_on_router_output():
    w = synth.WORKLOADS["tiny_f32"]
    inp = synth.make_inputs(w)
    dsc = oracle.desc(w)
    sr, sc = oracle.half_scores(dsc, inp["x"], inp["keys_row"], inp["keys_col"])
    idx, _, _, _ = oracle.select(dsc, sr, sc, oracle.CARTESIAN)
    perm, active, off, dense = oracle.schedule(dsc, idx)
    flat = idx.ravel()
    assert np.array_equal(np.sort(perm), np.arange(flat.size))
    for a, e in enumerate(active):
        seg = perm[off[a]:off[a + 1]]
        assert np.all(flat[seg] == e)
        assert np.all(np.diff(seg) > 0)
    assert off[-1] == w.M


# ---------------------------------------------------------------- expert compute (Eq. 4, 7, 14)

def test_forward_hand_example(golden_dir):
    # Catches a wrong gate, a wrong activation, a wrong expert row and a wrong output column.
    case = _load(golden_dir, "forward_onehot.json")
    phi = {float(k): v for k, v in _load(golden_dir, "activation_values.json")["phi"].items()}
    s = Shape(T=1, d=4, n_rows=2, n_cols=2, d_key=2, H=1, K=4)
    dsc = oracle.desc(s)
    eye = np.eye(4, dtype=np.float32)
    y, idx, g = oracle.layer_forward(dsc, np.array(case["x"], np.float32),
                                     np.array(case["keys_row"], np.float32),
                                     np.array(case["keys_col"], np.float32), eye, eye)
    assert idx.ravel().tolist() == case["idx"]
    e = math.e
    Z = e ** 3 + e ** 2 + e + 1
    want = [(e / Z) * phi[1.0], (e ** 3 / Z) * -(1 - phi[1.0]), (1 / Z) * 0.5 * phi[0.5],
            (e ** 2 / Z) * 2 * phi[2.0]]
    np.testing.assert_allclose(y[0], want, rtol=1e-14)


def _random_layer(seed, T=40, d=16, nr=6, nc=5, dk=8, H=3, K=4):
    rng = np.random.default_rng(seed)
    s = Shape(T=T, d=d, n_rows=nr, n_cols=nc, d_key=dk, H=H, K=K)
    N = nr * nc
    x = rng.standard_normal((T, d)).astype(np.float32)
    kr = rng.standard_normal((H, nr, dk)).astype(np.float32)
    kc = rng.standard_normal((H, nc, dk)).astype(np.float32)
    u = (rng.standard_normal((N, d)) / 4).astype(np.float32)
    v = (rng.standard_normal((N, d)) / 4).astype(np.float32)
    return s, x, kr, kc, u, v


@pytest.mark.parametrize("act", ["gelu", "silu"])
def test_forward_scheduled_equals_token_order_bitwise(act):
    s, x, kr, kc, u, v = _random_layer(8)
    s.act = act
    dsc = oracle.desc(s)
    sr, sc = oracle.half_scores(dsc, x, kr, kc)
    idx, _, g, _ = oracle.select(dsc, sr, sc)
    y0 = oracle.expert_forward(dsc, x, u, v, idx, g, scheduled=False)
    y1 = oracle.expert_forward(dsc, x, u, v, idx, g, scheduled=True)
    assert np.array_equal(y0, y1)


def test_forward_linearity_and_head_additivity():
    s, x, kr, kc, u, v = _random_layer(9)
    dsc = oracle.desc(s)
    sr, sc = oracle.half_scores(dsc, x, kr, kc)
    idx, _, g, _ = oracle.select(dsc, sr, sc)
    y = oracle.expert_forward(dsc, x, u, v, idx, g)
    # linear in V (a power of two keeps it exact)
    y2 = oracle.expert_forward(dsc, x, u, 2 * v, idx, g)
    assert np.array_equal(y2, 2 * y)
    # y is the sum over heads of each head's own contribution
    parts = 0
    for h in range(s.H):
        d1 = oracle.desc(s, H=1)
        parts = parts + oracle.expert_forward(d1, x, u, v, idx[:, h:h + 1], g[:, h:h + 1])
    np.testing.assert_allclose(y, parts, rtol=1e-12, atol=1e-14)


def test_forward_constant_tables_closed_form():
    # All u rows equal c and all v rows equal w: y_t = H * act(x_t . c) * w (gates sum to 1).
    s, x, kr, kc, u, v = _random_layer(10)
    dsc = oracle.desc(s)
    N = s.n_rows * s.n_cols
    c = np.linspace(-0.5, 0.5, s.d).astype(np.float32)
    wv = np.linspace(1, 2, s.d).astype(np.float32)
    y, _, _ = oracle.layer_forward(dsc, x, kr, kc, np.tile(c, (N, 1)), np.tile(wv, (N, 1)))
    z = x.astype(np.float64) @ c.astype(np.float64)
    want = s.H * np.array([oracle.act(GELU, zz) for zz in z])[:, None] * wv[None, :]
    np.testing.assert_allclose(y, want, rtol=1e-12)


def test_forward_zero_input_is_zero():
    s, x, kr, kc, u, v = _random_layer(11)
    y, idx, g = oracle.layer_forward(oracle.desc(s), np.zeros_like(x), kr, kc, u, v)
    assert np.all(y == 0.0)


def test_forward_single_expert_per_head():
    # K = 1: gate 1 and y = sum_h act(x . u_e) v_e.
    s, x, kr, kc, u, v = _random_layer(12, K=1)
    dsc = oracle.desc(s)
    y, idx, g = oracle.layer_forward(dsc, x, kr, kc, u, v)
    assert np.all(g == 1.0)
    want = np.zeros((s.T, s.d))
    for t in range(s.T):
        for h in range(s.H):
            e = idx[t, h, 0]
            z = float(x[t].astype(np.float64) @ u[e].astype(np.float64))
            want[t] += oracle.act(GELU, z) * v[e].astype(np.float64)
    np.testing.assert_allclose(y, want, rtol=1e-12, atol=1e-15)


def test_rejects_bad_shapes():
    s = Shape(T=4, d=8, n_rows=2, n_cols=2, d_key=5, H=1, K=2)  # 2 * d_key > d in split mode
    with pytest.raises(ValueError):
        oracle.half_scores(oracle.desc(s), np.zeros((4, 8)), np.zeros((1, 2, 5)),
                           np.zeros((1, 2, 5)))
    s = Shape(T=4, d=8, n_rows=2, n_cols=2, d_key=4, H=1, K=5)  # K > N
    with pytest.raises(ValueError):
        oracle.select(oracle.desc(s), np.zeros((4, 1, 2)), np.zeros((4, 1, 2)))


# ------------------------------------------------------------------ dense router (ablation)

def _product_key_gates(kr, kc, d, query_mode):
    """Gate table [H, N, d] whose dense logits equal the Cartesian scores: row n = i * n_cols + j
    holds keys_row[h, i] on the row query's columns and keys_col[h, j] on the column query's."""
    H, nr, dk = kr.shape
    nc = kc.shape[1]
    c0 = dk if query_mode == "split" else 0
    wg = np.zeros((H, nr * nc, d), np.float32)
    for i in range(nr):
        for j in range(nc):
            wg[:, i * nc + j, 0:dk] += kr[:, i]
            wg[:, i * nc + j, c0:c0 + dk] += kc[:, j]
    return wg


@pytest.mark.parametrize("mode", ["split", "shared"])
def test_dense_router_on_product_keys_equals_cartesian(mode):
    # With small-integer inputs every dot product is exact, so scoring all N cells densely
    # with w_gate[n] = (keys_row[i], keys_col[j]) must select exactly what the Cartesian router
    # selects, ties and order included.
    rng = np.random.default_rng(11)
    for (nr, nc, K) in [(6, 5, 4), (7, 9, 13), (4, 4, 16), (1, 8, 3), (10, 3, 1)]:
        dk = 3
        d = 2 * dk if mode == "split" else dk
        s = Shape(T=9, d=d, n_rows=nr, n_cols=nc, d_key=dk, H=2, K=K, query_mode=mode)
        dsc = oracle.desc(s)
        x = rng.integers(-2, 3, size=(s.T, d)).astype(np.float32)
        kr = rng.integers(-2, 3, size=(2, nr, dk)).astype(np.float32)
        kc = rng.integers(-2, 3, size=(2, nc, dk)).astype(np.float32)
        sr, sc = oracle.half_scores(dsc, x, kr, kc)
        i_c, _, g_c, _ = oracle.select(dsc, sr, sc, oracle.CARTESIAN, n_threads=1)
        i_d, g_d, L = oracle.route_dense(dsc, x, _product_key_gates(kr, kc, d, mode),
                                         with_logits=True, n_threads=1)
        assert np.array_equal(i_d, i_c), (nr, nc, K)
        np.testing.assert_array_equal(g_d, g_c)
        assert np.array_equal(L, (sr[..., :, None] + sc[..., None, :]).reshape(L.shape))


def test_dense_router_matches_numpy_definition():
    rng = np.random.default_rng(12)
    s = Shape(T=30, d=24, n_rows=9, n_cols=11, d_key=4, H=3, K=7)
    dsc = oracle.desc(s)
    x = rng.standard_normal((s.T, s.d)).astype(np.float32)
    wg = rng.standard_normal((s.H, 99, s.d)).astype(np.float32)
    idx, g, L = oracle.route_dense(dsc, x, wg, with_logits=True)
    want_L = np.einsum("td,hnd->thn", x.astype(np.float64), wg.astype(np.float64))
    np.testing.assert_allclose(L, want_L, rtol=1e-12, atol=1e-12)
    for t in range(s.T):
        for h in range(s.H):
            top = _brute_topk_lexsort(want_L[t, h], s.K)
            assert np.array_equal(idx[t, h], top)
            e = np.exp(want_L[t, h, top] - want_L[t, h, top[0]])
            np.testing.assert_allclose(g[t, h], e / e.sum(), rtol=1e-12)


def test_dense_select_ties_and_full_k():
    # Integer logits with heavy ties: ids ascending among equals; K = N returns every expert.
    rng = np.random.default_rng(13)
    s = Shape(T=20, d=2, n_rows=5, n_cols=6, d_key=1, H=2, K=30)
    L = rng.integers(-3, 4, size=(s.T, s.H, 30)).astype(np.float32)
    for K in (1, 4, 30):
        idx, g = oracle.select_dense_f32(oracle.desc(s, K=K), L)
        for t in range(s.T):
            for h in range(s.H):
                assert np.array_equal(idx[t, h], _brute_topk_lexsort(L[t, h].astype(np.float64), K))
        np.testing.assert_allclose(g.sum(axis=2), 1.0, rtol=1e-14)


# ------------------------------------------------------------------ shared dense MLP (Eq. 7)

def test_shared_mlp_hand_example(golden_dir):
    # d = 2, d_ff = 2: gate rows e0, e1; up rows 2 e0 and (e0 + e1); w_down swaps the features.
    # For x = (1, -2): g = (1, -2), u = (2, -1), a = (silu(1) * 2, silu(-2) * -1) with
    # silu(z) = z * logistic(z) from the table; y = (a_1, a_0) added to y0.
    lg = _load(golden_dir, "activation_values.json")["logistic"]
    s = Shape(T=1, d=2, n_rows=1, n_cols=1, d_key=1, H=1, K=1)
    x = np.array([[1.0, -2.0]], np.float32)
    w_gu = np.array([[1, 0], [0, 1], [2, 0], [1, 1]], np.float32)
    w_down = np.array([[0, 1], [1, 0]], np.float32)
    a0 = 1.0 * lg["1"] * 2.0
    a1 = -2.0 * lg["-2"] * -1.0
    y = oracle.shared_mlp(oracle.desc(s), x, w_gu, w_down, y=np.array([[0.5, -0.25]]))
    np.testing.assert_allclose(y, [[0.5 + a1, -0.25 + a0]], rtol=1e-15)


def test_shared_mlp_matches_numpy_and_is_linear_in_w_down():
    rng = np.random.default_rng(21)
    s = Shape(T=17, d=12, n_rows=2, n_cols=2, d_key=2, H=1, K=1)
    dsc = oracle.desc(s)
    x = rng.standard_normal((s.T, s.d)).astype(np.float32)
    w_gu = rng.standard_normal((2 * 9, s.d)).astype(np.float32)
    w_down = rng.standard_normal((s.d, 9)).astype(np.float32)
    y = oracle.shared_mlp(dsc, x, w_gu, w_down)
    h = x.astype(np.float64) @ w_gu.astype(np.float64).T
    g, u = h[:, :9], h[:, 9:]
    want = (g / (1.0 + np.exp(-g)) * u) @ w_down.astype(np.float64).T
    np.testing.assert_allclose(y, want, rtol=1e-12, atol=1e-12)
    # scaling w_down by a power of two scales every product and sum exactly
    y2 = oracle.shared_mlp(dsc, x, w_gu, 2.0 * w_down)
    np.testing.assert_array_equal(y2, 2.0 * y)
    assert np.all(oracle.shared_mlp(dsc, np.zeros_like(x), w_gu, w_down) == 0.0)


# ------------------------------------------------------------------ expert backward

@pytest.mark.parametrize("act", ["gelu", "silu"])
def test_activation_derivative_matches_central_differences(act):
    kind = {"gelu": 0, "silu": 1}[act]
    for z in (-3.0, -1.3, -0.2, 0.0, 0.4, 1.0, 2.7):
        h = 1e-5
        fd = (oracle.act(kind, z + h) - oracle.act(kind, z - h)) / (2 * h)
        assert abs(oracle.act_grad(kind, z) - fd) < 1e-9
    # closed forms at 0: GELU' = Phi(0) = 1/2, SiLU' = s(0) = 1/2
    assert oracle.act_grad(kind, 0.0) == 0.5


def _backward_case(seed, act):
    rng = np.random.default_rng(seed)
    s = Shape(T=5, d=6, n_rows=3, n_cols=4, d_key=2, H=2, K=3, act=act)
    N = s.n_rows * s.n_cols
    # dyadic values, so a perturbation of 2^-12 is exact in float32
    x = (rng.integers(-8, 9, size=(s.T, s.d)) / 8).astype(np.float32)
    u = (rng.integers(-8, 9, size=(N, s.d)) / 16).astype(np.float32)
    v = (rng.integers(-8, 9, size=(N, s.d)) / 16).astype(np.float32)
    idx = np.stack([rng.choice(N, s.K, replace=False) for _ in range(s.T * s.H)]).reshape(
        s.T, s.H, s.K).astype(np.int32)
    idx[0, 1] = idx[0, 0]   # one expert picked by both heads of a token
    scores = np.sort(rng.standard_normal((s.T, s.H, s.K)), axis=-1)[..., ::-1].copy()
    dy = rng.standard_normal((s.T, s.d))
    return s, x, u, v, idx, scores, dy


def _softmax(scores):
    e = np.exp(scores - scores[..., :1])
    return e / e.sum(axis=-1, keepdims=True)


@pytest.mark.parametrize("act", ["gelu", "silu"])
def test_expert_backward_matches_finite_differences(act):
    s, x, u, v, idx, scores, dy = _backward_case(31, act)
    dsc = oracle.desc(s)
    gates = _softmax(scores)

    def loss(x=x, u=u, v=v, gates=gates):
        y = oracle.expert_forward(dsc, x, u, v, idx, gates, scheduled=False, n_threads=1)
        return float(np.sum(dy * y))

    g = oracle.expert_backward(dsc, x, u, v, idx, gates, dy, n_threads=1)
    h = 2.0 ** -12
    for (t, m) in [(0, 0), (1, 3), (4, 5), (2, 2)]:
        xp, xm = x.copy(), x.copy()
        xp[t, m] += h
        xm[t, m] -= h
        fd = (loss(x=xp) - loss(x=xm)) / (2 * h)
        assert abs(g["dx"][t, m] - fd) <= 1e-6 * max(1.0, abs(fd))
    rows = {int(e): r for r, e in enumerate(g["active"])}
    assert sorted(rows) == sorted(set(idx.ravel().tolist()))
    for e in sorted(rows)[:4]:
        for m in (0, 5):
            for name, tab in (("du_rows", u), ("dv_rows", v)):
                tp, tm = tab.copy(), tab.copy()
                tp[e, m] += h
                tm[e, m] -= h
                kw = {"u": tp} if name == "du_rows" else {"v": tp}
                kw2 = {"u": tm} if name == "du_rows" else {"v": tm}
                fd = (loss(**kw) - loss(**kw2)) / (2 * h)
                assert abs(g[name][rows[e], m] - fd) <= 1e-6 * max(1.0, abs(fd)), (name, e, m)
    hg = 1e-6
    for p in [(0, 0, 0), (0, 1, 2), (3, 1, 1)]:
        gp, gm = gates.copy(), gates.copy()
        gp[p] += hg
        gm[p] -= hg
        fd = (loss(gates=gp) - loss(gates=gm)) / (2 * hg)
        assert abs(g["dgates"][p] - fd) <= 1e-7 * max(1.0, abs(fd))
    for p in [(0, 0, 0), (2, 1, 2), (4, 0, 1)]:
        sp, sm = scores.copy(), scores.copy()
        sp[p] += hg
        sm[p] -= hg
        fd = (loss(gates=_softmax(sp)) - loss(gates=_softmax(sm))) / (2 * hg)
        assert abs(g["dscores"][p] - fd) <= 1e-7 * max(1.0, abs(fd))
    # the softmax gradient sums to zero over each (token, head) row
    np.testing.assert_allclose(g["dscores"].sum(axis=-1), 0.0, atol=1e-12)


def test_expert_backward_linearity_in_dy():
    s, x, u, v, idx, scores, dy = _backward_case(32, "gelu")
    dsc = oracle.desc(s)
    gates = _softmax(scores)
    g1 = oracle.expert_backward(dsc, x, u, v, idx, gates, dy)
    g2 = oracle.expert_backward(dsc, x, u, v, idx, gates, 2.0 * dy)
    for k in ("dx", "du_rows", "dv_rows", "dgates", "dscores"):
        np.testing.assert_array_equal(g2[k], 2.0 * g1[k])


@pytest.mark.parametrize("mode", ["split", "shared"])
def test_route_backward_matches_finite_differences(mode):
    # With the selections held fixed, L = sum_p dscores_p S_p is linear in x and the sub-keys,
    # so central differences of the oracle's own half-scores give the gradient up to rounding.
    rng = np.random.default_rng(41)
    dk = 3
    d = 2 * dk if mode == "split" else dk + 2
    s = Shape(T=5, d=d, n_rows=4, n_cols=3, d_key=dk, H=2, K=3, query_mode=mode)
    dsc = oracle.desc(s)
    x = (rng.integers(-8, 9, size=(s.T, d)) / 8).astype(np.float32)
    kr = (rng.integers(-8, 9, size=(s.H, s.n_rows, dk)) / 8).astype(np.float32)
    kc = (rng.integers(-8, 9, size=(s.H, s.n_cols, dk)) / 8).astype(np.float32)
    N = s.n_rows * s.n_cols
    idx = np.stack([rng.choice(N, s.K, replace=False) for _ in range(s.T * s.H)]).reshape(
        s.T, s.H, s.K).astype(np.int32)
    ds = rng.standard_normal((s.T, s.H, s.K))

    def loss(x=x, kr=kr, kc=kc):
        sr, sc = oracle.half_scores(dsc, x, kr, kc, n_threads=1)
        i, j = idx // s.n_cols, idx % s.n_cols
        S = np.take_along_axis(sr, i, axis=2) + np.take_along_axis(sc, j, axis=2)
        return float(np.sum(ds * S))

    dx, dkr, dkc = oracle.route_backward(dsc, x, kr, kc, idx, ds, n_threads=1)
    h = 2.0 ** -10
    for arr, grad, key in ((x, dx, "x"), (kr, dkr, "kr"), (kc, dkc, "kc")):
        for pos in [tuple(rng.integers(0, n) for n in arr.shape) for _ in range(6)]:
            ap, am = arr.copy(), arr.copy()
            ap[pos] += h
            am[pos] -= h
            fd = (loss(**{key: ap}) - loss(**{key: am})) / (2 * h)
            assert abs(grad[pos] - fd) <= 1e-9 * max(1.0, abs(fd)), (key, pos)
    # rows no task selected have zero gradient
    used_r = {(h_, int(i)) for h_ in range(s.H) for i in (idx[:, h_] // s.n_cols).ravel()}
    for h_ in range(s.H):
        for i in range(s.n_rows):
            if (h_, i) not in used_r:
                assert np.all(dkr[h_, i] == 0.0)
