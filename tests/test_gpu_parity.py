"""GPU parity: the HIP library, called through its C ABI, against the oracle on the same seeded inputs.

Tiers: half-scores within Higham's fp32 dot bound; selection bit-exact on identical fp32 logits;
schedule bit-exact; expert compute and whole layer within the stated relative tolerance
(1e-5 fp32, 2e-2 bf16), with routing bit-exact on every (token, head) row whose top-(K+1)
score gaps are certified larger than the logit error.
"""
import gc
import sys

import numpy as np
import pytest

import oracle
import synth
from gpu_support import (GATE_TOL, backward_error_bounds, compare_routing, gate_bound_check,
                         grouped_gap_bound,
                         higham_bound, row_rel_err, to_dev, tol, upload)

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
import paper_2602_05711_amd as P  # noqa: E402
from paper_2602_05711_amd import binding as B  # noqa: E402


def say(*a):
    print(*a, file=sys.stderr, flush=True)


W = synth.WORKLOADS
RAGGED = synth.Workload("ragged_bf16", T=300, d=208, n_rows=40, n_cols=72, d_key=96, H=3, K=13)
SHAPES = {
    "tiny_f32": W["tiny_f32"],
    "small_bf16": W["small_bf16"],
    "ragged_bf16": RAGGED,
    "ragged_f32": RAGGED.with_(name="ragged_f32", dtype="f32"),
    "shared_bf16": W["small_bf16"].with_(name="shared_bf16", T=500, d_key=512,
                                         query_mode="shared"),
    "silu_k1_bf16": RAGGED.with_(name="silu_k1_bf16", act="silu", K=1),
    "k64_bf16": synth.Workload("k64_bf16", T=200, d=256, n_rows=64, n_cols=64, d_key=64, H=2,
                               K=64),
    "one_row_f32": synth.Workload("one_row_f32", T=100, d=64, n_rows=1, n_cols=96, d_key=32,
                                  H=2, K=9, dtype="f32"),
    "all_experts_bf16": synth.Workload("all_experts_bf16", T=64, d=128, n_rows=4, n_cols=4,
                                       d_key=64, H=2, K=16),
    "wide_bf16": synth.Workload("wide_bf16", T=70, d=8192, n_rows=16, n_cols=32, d_key=64, H=2,
                                K=8),
    "wide_f32": synth.Workload("wide_f32", T=70, d=4096, n_rows=32, n_cols=16, d_key=2048, H=1,
                               K=5, dtype="f32"),
    # T <= 64 with d_key % 256 == 0: the decode-shaped logit kernel, ragged key tiles
    "skinny_bf16": synth.Workload("skinny_bf16", T=40, d=1024, n_rows=48, n_cols=80, d_key=256,
                                  H=3, K=7),
    "skinny1_bf16": synth.Workload("skinny1_bf16", T=1, d=1024, n_rows=48, n_cols=80, d_key=512,
                                   H=2, K=12),
    # T <= 4: the coalesced few-token logit kernel (d_key 256 and 128; key rows past a head's
    # end and a key count that is not a multiple of the sixteen per workgroup)
    "few3_bf16": synth.Workload("few3_bf16", T=3, d=512, n_rows=40, n_cols=23, d_key=256, H=2,
                                K=7),
    "few2_bf16": synth.Workload("few2_bf16", T=2, d=256, n_rows=9, n_cols=31, d_key=128, H=3,
                                K=5),
    # decode-sized layers (slot-order dot) with 96, 100 and 128 slots per token: the routed sum
    # in sixteen partial rows per token, some of them empty; fp32
    "slots96_bf16": synth.Workload("slots96_bf16", T=40, d=512, n_rows=64, n_cols=48,
                                   d_key=128, H=4, K=24),
    "slots100_bf16": synth.Workload("slots100_bf16", T=9, d=1024, n_rows=30, n_cols=50,
                                    d_key=256, H=4, K=25),
    "slots128_f32": synth.Workload("slots128_f32", T=5, d=256, n_rows=32, n_cols=32, d_key=64,
                                   H=2, K=64, dtype="f32"),
    "decode8_bf16": synth.Workload("decode8_bf16", T=8, d=2048, n_rows=100, n_cols=36,
                                   d_key=1024, H=2, K=9),
    # the selection kernel forming the slot-order dot (256 or more (token, head) rows, a square
    # grid of 256 or 512): one pick per row; three (a partial group of four); 64 (the wave's
    # width) with d = 1024
    "fused_k1_bf16": synth.Workload("fused_k1_bf16", T=64, d=512, n_rows=256, n_cols=256,
                                    d_key=256, H=4, K=1),
    "fused_k3_bf16": synth.Workload("fused_k3_bf16", T=100, d=512, n_rows=256, n_cols=256,
                                    d_key=128, H=3, K=3, act="silu"),
    "fused_k64_bf16": synth.Workload("fused_k64_bf16", T=32, d=1024, n_rows=512, n_cols=512,
                                     d_key=512, H=8, K=64),
    "decode_dk768_bf16": synth.Workload("decode_dk768_bf16", T=20, d=1536, n_rows=70, n_cols=64,
                                        d_key=768, H=2, K=5),
    # K > 64 (workgroup-per-row selection), incl. the paper's benchmark grid 320 x 320, K = 512
    "k256_bf16": synth.Workload("k256_bf16", T=100, d=256, n_rows=64, n_cols=64, d_key=64, H=2,
                                K=256),
    "paper_k512_bf16": synth.Workload("paper_k512_bf16", T=256, d=1024, n_rows=320, n_cols=320,
                                      d_key=512, H=1, K=512),
    # one head with K >= N / 64: the routed sum as one dense GEMM over all experts (Eq. 14 with
    # a single group); split over the expert dimension, N not a multiple of the split width
    "dense_bf16": synth.Workload("dense_bf16", T=300, d=256, n_rows=32, n_cols=32, d_key=64, H=1,
                                 K=64),
    "dense_k100_bf16": synth.Workload("dense_k100_bf16", T=77, d=192, n_rows=40, n_cols=50,
                                      d_key=64, H=1, K=100),
    # several row and column tiles of the dense first product (42 tiles over 8 XCDs), N and d
    # not multiples of 256, the expert dimension padded to the split width (3584 > 3360)
    "dense_wide_bf16": synth.Workload("dense_wide_bf16", T=700, d=320, n_rows=56, n_cols=60,
                                      d_key=64, H=1, K=64),
    # every expert selected by every token (K = N): the epilogue's queues hold all 2048 cells of
    # each quarter; SiLU in the masked-activation epilogue, shared query
    "dense_all_bf16": synth.Workload("dense_all_bf16", T=300, d=128, n_rows=8, n_cols=8, d_key=64,
                                     H=1, K=64),
    "dense_silu_bf16": synth.Workload("dense_silu_bf16", T=260, d=192, n_rows=24, n_cols=40,
                                      d_key=64, H=1, K=40, act="silu", query_mode="shared"),
    # groups of 64 experts with about twelve slot tiles each: the grouped GEMM's tiles are
    # shared out to the XCDs by token range
    "bucket_bf16": synth.Workload("bucket_bf16", T=3000, d=128, n_rows=64, n_cols=64, d_key=64,
                                  H=2, K=128),
    # at most 8192 tasks (the layer's slot-order dot, no schedule), every expert picked by every
    # token: 400 and 2730 tasks per expert, and the largest such batch (8190 tasks, ragged)
    "slots_crowded_bf16": synth.Workload("slots_crowded_bf16", T=200, d=256, n_rows=2, n_cols=4,
                                         d_key=64, H=2, K=8),
    "slots_crowded_f32": synth.Workload("slots_crowded_f32", T=1365, d=128, n_rows=1, n_cols=3,
                                        d_key=32, H=2, K=3, dtype="f32"),
}


def host_inputs(w):
    inp = synth.make_inputs(w)
    f32 = {k: synth.as_f32(v) for k, v in inp.items()}
    return inp, f32


def gpu_layer(w, dev):
    d = B.make_desc(w)
    y = torch.empty((w.T, w.d), dtype=torch.float32, device="cuda")
    idx = torch.empty((w.T, w.H, w.K), dtype=torch.int32, device="cuda")
    g = torch.empty((w.T, w.H, w.K), dtype=torch.float32, device="cuda")
    P.omnimoe_layer_forward(d, dev["x"], dev["keys_row"], dev["keys_col"], dev["u"], dev["v"], y,
                            idx, g)
    torch.cuda.synchronize()
    return y.cpu().numpy(), idx.cpu().numpy(), g.cpu().numpy()


def gpu_half_scores(w, dev):
    d = B.make_desc(w)
    hs = torch.empty((w.T, w.H, w.n_rows + w.n_cols), dtype=torch.float32, device="cuda")
    idx = torch.empty((w.T, w.H, w.K), dtype=torch.int32, device="cuda")
    g = torch.empty((w.T, w.H, w.K), dtype=torch.float32, device="cuda")
    P.omnimoe_route(d, dev["x"], dev["keys_row"], dev["keys_col"], idx, g, half_scores=hs)
    torch.cuda.synchronize()
    return hs.cpu().numpy(), idx.cpu().numpy(), g.cpu().numpy()


# ------------------------------------------------------------------ logits and routing

@pytest.mark.parametrize("name", list(SHAPES))
def test_route_half_scores_and_selection(name):
    w = SHAPES[name]
    say(f"[route] {name} T={w.T} d={w.d} grid={w.n_rows}x{w.n_cols} dk={w.d_key} H={w.H} K={w.K}")
    inp, f = host_inputs(w)
    dev = upload(inp)
    hs, idx, g = gpu_half_scores(w, dev)
    dsc = oracle.desc(w)
    sr, sc = oracle.half_scores(dsc, f["x"], f["keys_row"], f["keys_col"])
    c0 = w.d_key if w.query_mode == "split" else 0
    bound_r = higham_bound(f["x"][:, :w.d_key], f["keys_row"])
    bound_c = higham_bound(f["x"][:, c0:c0 + w.d_key], f["keys_col"])
    err_r = np.abs(hs[..., :w.n_rows] - sr)
    err_c = np.abs(hs[..., w.n_rows:] - sc)
    assert np.all(err_r <= bound_r + 1e-30) and np.all(err_c <= bound_c + 1e-30)
    # selection on the GPU's own logits is exact
    ri, _, rg, inexact = oracle.select_f32(dsc, hs, oracle.CARTESIAN)
    assert inexact == 0
    assert np.array_equal(idx, ri)
    np.testing.assert_allclose(g, rg, rtol=GATE_TOL, atol=1e-7)
    # against the fp64 router, exact outside certified near-ties
    delta = max(float(err_r.max()), float(err_c.max()), 1e-300)
    unc, unc_rows, npos = compare_routing(w, idx, sr, sc, delta)
    say(f"  max logit err {delta:.3e}, uncertified positions {unc} of {npos} "
        f"(rows {unc_rows} of {w.T * w.H})")


SELECT_CASES = [
    # (n_rows, n_cols, K, H, T, tie_heavy)
    (64, 64, 8, 1, 256, False), (256, 256, 16, 4, 300, False), (1024, 1024, 16, 8, 40, False),
    (40, 72, 13, 3, 100, False), (64, 64, 64, 2, 50, False), (1, 50, 7, 2, 40, False),
    (50, 1, 7, 2, 40, False), (8, 8, 64, 1, 30, False), (4096, 4096, 16, 1, 6, False),
    (3000, 17, 20, 2, 9, False), (64, 64, 8, 1, 64, True), (256, 256, 16, 2, 64, True),
    (1024, 1024, 64, 1, 16, True), (16, 16, 33, 3, 20, True),
    # K > 64: one workgroup per row (full half sorts, Cartesian radix select)
    (320, 320, 512, 1, 12, False), (320, 320, 4096, 1, 6, False), (64, 64, 65, 2, 20, False),
    (1024, 1024, 128, 8, 8, False), (4096, 4096, 4096, 1, 3, False), (50, 7, 300, 2, 10, False),
    (16, 16, 256, 1, 8, False), (256, 256, 1000, 1, 10, True), (64, 64, 200, 2, 12, True),
]


@pytest.mark.parametrize("case", SELECT_CASES, ids=[str(c) for c in SELECT_CASES])
def test_select_bitexact(case):
    nr, nc, K, H, T, ties = case
    say(f"[select] grid={nr}x{nc} K={K} H={H} T={T} ties={ties}")
    rng = np.random.default_rng(nr * 7919 + nc * 31 + K)
    if ties:
        hs = rng.integers(-3, 4, size=(T, H, nr + nc)).astype(np.float32)
        hs[hs == 0] = -0.0 if rng.random() < 0.5 else 0.0
    else:
        hs = rng.standard_normal((T, H, nr + nc)).astype(np.float32)
    w = synth.Workload("sel", T=T, d=16, n_rows=nr, n_cols=nc, d_key=8, H=H, K=K, dtype="f32")
    d = B.make_desc(w)
    idx = torch.empty((T, H, K), dtype=torch.int32, device="cuda")
    g = torch.empty((T, H, K), dtype=torch.float32, device="cuda")
    P.omnimoe_select(d, to_dev(hs), idx, g)
    torch.cuda.synchronize()
    ri, _, rg, inexact = oracle.select_f32(oracle.desc(w), hs, oracle.CARTESIAN)
    bi, _, _, _ = oracle.select_f32(oracle.desc(w), hs, oracle.BRUTE)
    assert inexact == 0 and np.array_equal(ri, bi)
    assert np.array_equal(idx.cpu().numpy(), ri)
    np.testing.assert_allclose(g.cpu().numpy(), rg, rtol=GATE_TOL, atol=1e-7)


# ------------------------------------------------------------------ schedule

def _zipf_ids(rng, M, N, s=1.1):
    ranks = np.arange(1, N + 1, dtype=np.float64)
    p = ranks ** -s
    p /= p.sum()
    ids = rng.choice(N, size=M, p=p)
    return rng.permutation(N)[ids].astype(np.int32)


SCHEDULE_CASES = [
    # (T, H, K, n_rows, n_cols, kind)
    (256, 1, 8, 64, 64, "uniform"), (4096, 4, 16, 256, 256, "uniform"), (3, 1, 1, 1, 7, "uniform"),
    (999, 3, 1, 1, 1, "uniform"), (1000, 2, 7, 200, 250, "uniform"),
    (16384, 8, 16, 1024, 1024, "uniform"), (16384, 8, 16, 1024, 1024, "zipf"),
    (64, 8, 16, 1024, 1024, "uniform"), (1, 8, 16, 1024, 1024, "zipf"),
    (5000, 2, 3, 4096, 4096, "uniform"),
    # 4097 .. 8192 tasks: expert ranges over several workgroups, and the fallback when one
    # range holds too many tasks (few experts, skew)
    (64, 8, 16, 1024, 1024, "zipf"), (256, 8, 4, 2, 2, "zipf"), (40, 8, 16, 64, 64, "uniform"),
    (256, 8, 3, 1, 3, "uniform"), (33, 8, 16, 1024, 1024, "uniform"),
    # radix passes with a ragged last tile and a tiny digit range (2 bits; one expert)
    (3000, 4, 1, 1, 3, "uniform"), (2500, 4, 1, 1, 1, "uniform"), (4099, 3, 1, 2, 3, "zipf"),
]


@pytest.mark.parametrize("case", SCHEDULE_CASES, ids=[str(c) for c in SCHEDULE_CASES])
def test_schedule_bitexact(case):
    T, H, K, nr, nc, kind = case
    N = nr * nc
    say(f"[schedule] T={T} H={H} K={K} N={N} {kind}")
    rng = np.random.default_rng(T + 17 * K + N % 1009)
    M = T * H * K
    ids = (_zipf_ids(rng, M, N) if kind == "zipf" else rng.integers(0, N, size=M)).astype(
        np.int32)
    w = synth.Workload("sch", T=T, d=16, n_rows=nr, n_cols=nc, d_key=8, H=H, K=K, dtype="f32")
    d = B.make_desc(w)
    A = min(M, N)
    perm = torch.empty(M, dtype=torch.int32, device="cuda")
    active = torch.full((A,), -7, dtype=torch.int32, device="cuda")
    off = torch.full((A + 1,), -7, dtype=torch.int32, device="cuda")
    na = torch.zeros(1, dtype=torch.int32, device="cuda")
    dense = torch.empty(N + 1, dtype=torch.int32, device="cuda")
    P.omnimoe_schedule(d, to_dev(ids), perm, active, off, na, dense)
    torch.cuda.synchronize()
    rperm, ract, roff, rdense = oracle.schedule(oracle.desc(w), ids)
    n = int(na.item())
    assert n == len(ract)
    assert np.array_equal(perm.cpu().numpy(), rperm)
    assert np.array_equal(active.cpu().numpy()[:n], ract)
    assert np.array_equal(off.cpu().numpy()[:n + 1], roff)
    assert np.array_equal(dense.cpu().numpy(), rdense)


GROUP_CASES = [
    # (T, H, K, n_rows, n_cols, kind, B)
    (256, 1, 8, 64, 64, "uniform", 2), (4096, 4, 16, 256, 256, "uniform", 7),
    (16384, 8, 16, 1024, 1024, "zipf", 64), (64, 8, 16, 1024, 1024, "uniform", 3),
    (3, 1, 1, 1, 7, "uniform", 5), (5000, 2, 3, 4096, 4096, "uniform", 1000),
    (4096, 1, 512, 320, 320, "uniform", 16),
]


@pytest.mark.parametrize("case", GROUP_CASES, ids=[str(c) for c in GROUP_CASES])
def test_schedule_groups_bitexact(case):
    # Groups of B active experts (Eq. 13): tasks ordered by (group, task id).
    T, H, K, nr, nc, kind, Bg = case
    N = nr * nc
    say(f"[schedule B={Bg}] T={T} H={H} K={K} N={N} {kind}")
    rng = np.random.default_rng(T + 17 * K + N % 1009 + Bg)
    M = T * H * K
    if K > 16:
        ids = np.stack([rng.choice(N, K, replace=False) for _ in range(T * H)]).astype(np.int32)
    else:
        ids = (_zipf_ids(rng, M, N) if kind == "zipf" else rng.integers(0, N, size=M)).astype(
            np.int32)
    w = synth.Workload("sch", T=T, d=16, n_rows=nr, n_cols=nc, d_key=8, H=H, K=K, dtype="f32")
    d = B.make_desc(w)
    d.group_size = Bg
    A = min(M, N)
    perm = torch.empty(M, dtype=torch.int32, device="cuda")
    active = torch.full((A,), -7, dtype=torch.int32, device="cuda")
    off = torch.full((A + 1,), -7, dtype=torch.int32, device="cuda")
    na = torch.zeros(1, dtype=torch.int32, device="cuda")
    dense = torch.empty(N + 1, dtype=torch.int32, device="cuda")
    P.omnimoe_schedule(d, to_dev(ids.ravel()), perm, active, off, na, dense)
    torch.cuda.synchronize()
    rperm, ract, roff, rdense = oracle.schedule(oracle.desc(w, group_size=Bg), ids.ravel())
    n = int(na.item())
    assert n == len(ract)
    assert np.array_equal(perm.cpu().numpy(), rperm)
    assert np.array_equal(active.cpu().numpy()[:n], ract)
    assert np.array_equal(off.cpu().numpy()[:n + 1], roff)
    assert np.array_equal(dense.cpu().numpy(), rdense)


def grouped_path(w):
    """Whether the layer runs the grouped expert GEMM for group sizes above 1."""
    return w.bf16 and w.d % 64 == 0


@pytest.mark.parametrize("name", ["small_bf16", "skinny_bf16", "k256_bf16", "ragged_bf16"])
def test_layer_group_size(name):
    # Routing does not depend on B. With B > 1 the expert activations come from the grouped GEMM
    # (bf16, d % 64 == 0): equal to the B = 1 result up to the order of the fp32 dot sums, within
    # the element-wise bound of that reordering; otherwise bit for bit.
    w = SHAPES[name]
    inp, f = host_inputs(w)
    dev = upload(inp)
    y1, i1, g1 = gpu_layer(w, dev)
    for Bg in (4, 33):
        say(f"[layer B={Bg}] {name}")
        yb, ib, gb = gpu_layer(w.with_(group_size=Bg), dev)
        assert np.array_equal(ib, i1) and np.array_equal(gb.view(np.uint8), g1.view(np.uint8))
        if grouped_path(w):
            bound = grouped_gap_bound(f, i1, g1, w.d, oracle.desc(w).act)
            gap = np.abs(yb.astype(np.float64) - y1)
            say(f"  max gap / bound {(gap / bound).max():.3e}")
            assert np.all(gap <= bound)
        else:
            assert np.array_equal(yb.view(np.uint8), y1.view(np.uint8))


GROUPED_CASES = [
    # (shape, B): partial expert tiles, groups of 64 and of more than 64 experts, a single group
    # holding every active expert, B = 1, wide d, few tokens, K > 64 and the paper's grid
    ("small_bf16", 2), ("small_bf16", 64), ("small_bf16", 100), ("k64_bf16", 33),
    ("all_experts_bf16", 5), ("all_experts_bf16", 1 << 20), ("k64_bf16", 1),
    ("wide_bf16", 3), ("skinny_bf16", 16), ("skinny1_bf16", 7), ("k256_bf16", 64),
    ("shared_bf16", 48), ("paper_k512_bf16", 320), ("bucket_bf16", 64), ("bucket_bf16", 100),
]


@pytest.mark.parametrize("case", GROUPED_CASES, ids=[f"{n}-B{b}" for n, b in GROUPED_CASES])
def test_expert_forward_grouped(case):
    name, Bg = case
    w1 = SHAPES[name]
    w = w1.with_(group_size=Bg)
    say(f"[grouped] {name} B={Bg}")
    inp, f = host_inputs(w)
    dev = upload(inp)
    dsc = oracle.desc(w)
    sr, sc = oracle.half_scores(dsc, f["x"], f["keys_row"], f["keys_col"])
    idx, _, g64, _ = oracle.select(dsc, sr, sc, oracle.CARTESIAN)
    g32 = g64.astype(np.float32)
    perm, active, _, _ = oracle.schedule(dsc, idx)
    perm1, _, _, _ = oracle.schedule(oracle.desc(w1), idx)
    cap = min(w.M, w.N)
    act_pad = np.zeros(cap, dtype=np.int32)
    act_pad[:len(active)] = active
    gi, gg = to_dev(idx), to_dev(g32)
    y = torch.full((w.T, w.d), float("nan"), dtype=torch.float32, device="cuda")
    y1 = torch.empty((w.T, w.d), dtype=torch.float32, device="cuda")
    na = torch.tensor([len(active)], dtype=torch.int32, device="cuda")
    P.omnimoe_expert_forward_grouped(B.make_desc(w), dev["x"], dev["u"], dev["v"], gi, gg,
                                     to_dev(perm), to_dev(act_pad), na, y)
    P.omnimoe_expert_forward(B.make_desc(w1), dev["x"], dev["u"], dev["v"], gi, gg,
                             to_dev(perm1), y1)
    y_again = torch.empty_like(y)
    P.omnimoe_expert_forward_grouped(B.make_desc(w), dev["x"], dev["u"], dev["v"], gi, gg,
                                     to_dev(perm), to_dev(act_pad), na, y_again)
    torch.cuda.synchronize()
    y, y1, y_again = y.cpu().numpy(), y1.cpu().numpy(), y_again.cpu().numpy()
    assert np.array_equal(y.view(np.uint8), y_again.view(np.uint8))
    y_ref = oracle.expert_forward(dsc, f["x"], f["u"], f["v"], idx, g32.astype(np.float64))
    err = row_rel_err(y, y_ref)
    bound = grouped_gap_bound(f, idx, g32, w.d, dsc.act)
    gap = np.abs(y.astype(np.float64) - y1)
    say(f"  max row rel err {err.max():.3e}; max gap / bound {(gap / bound).max():.3e}")
    assert err.max() <= tol(w)
    assert np.all(gap <= bound)


# ------------------------------------------------------------------ expert compute

EXPERT_SHAPES = ["tiny_f32", "small_bf16", "ragged_bf16", "ragged_f32", "silu_k1_bf16",
                 "k64_bf16", "all_experts_bf16", "wide_bf16", "wide_f32"]


def _expert_case(name):
    """Oracle routing and schedule of one shape, the oracle's y, and the inputs on the GPU."""
    w = SHAPES[name]
    inp, f = host_inputs(w)
    dsc = oracle.desc(w)
    sr, sc = oracle.half_scores(dsc, f["x"], f["keys_row"], f["keys_col"])
    idx, _, g64, _ = oracle.select(dsc, sr, sc, oracle.CARTESIAN)
    g32 = g64.astype(np.float32)
    perm, _, _, _ = oracle.schedule(dsc, idx)
    y_ref = oracle.expert_forward(dsc, f["x"], f["u"], f["v"], idx, g32.astype(np.float64))
    return w, upload(inp), idx, g32, perm, y_ref


@pytest.mark.parametrize("name", EXPERT_SHAPES)
def test_expert_forward(name):
    say(f"[expert] {name}")
    w, dev, idx, g32, perm, y_ref = _expert_case(name)
    y = torch.empty((w.T, w.d), dtype=torch.float32, device="cuda")
    P.omnimoe_expert_forward(B.make_desc(w), dev["x"], dev["u"], dev["v"], to_dev(idx),
                             to_dev(g32), to_dev(perm), y)
    torch.cuda.synchronize()
    err = row_rel_err(y.cpu().numpy(), y_ref)
    say(f"  max row rel err {err.max():.3e}")
    assert err.max() <= tol(w)


@pytest.mark.parametrize("name", EXPERT_SHAPES)
def test_token_centric_ablation(name):
    # Without the schedule: within tolerance of the oracle, and equal to the scheduled path (same
    # dot, activation and slot-order sum). Below 1024 tokens the scheduled path adds each
    # token's slots in several partial sums, so there the two agree to rounding only.
    say(f"[token-centric] {name}")
    w, dev, idx, g32, perm, y_ref = _expert_case(name)
    d = B.make_desc(w)
    y = torch.empty((w.T, w.d), dtype=torch.float32, device="cuda")
    y_tc = torch.full((w.T, w.d), float("nan"), dtype=torch.float32, device="cuda")
    gi, gg = to_dev(idx), to_dev(g32)
    P.omnimoe_expert_forward(d, dev["x"], dev["u"], dev["v"], gi, gg, to_dev(perm), y)
    P.omnimoe_expert_forward_token_centric(d, dev["x"], dev["u"], dev["v"], gi, gg, y_tc)
    torch.cuda.synchronize()
    y_tc = y_tc.cpu().numpy()
    err = row_rel_err(y_tc, y_ref)
    say(f"  max row rel err {err.max():.3e}")
    assert err.max() <= tol(w)
    y = y.cpu().numpy()
    if w.T >= 1024:
        assert np.array_equal(y_tc, y)
    else:
        assert row_rel_err(y_tc, y.astype(np.float64)).max() <= 1e-6


@pytest.mark.parametrize("name", EXPERT_SHAPES)
def test_expert_forward_scatter(name):
    # Contribution rows a_p v_e written expert by expert, then summed per token in slot order:
    # within tolerance of the oracle, the same bits on a second call (into a workspace full of
    # the first call's rows), and within fp32 rounding of the slot-order sum (which fuses each
    # product into the sum; here each product is rounded first).
    say(f"[scatter] {name}")
    w, dev, idx, g32, perm, y_ref = _expert_case(name)
    d = B.make_desc(w)
    gi, gg, gp = to_dev(idx), to_dev(g32), to_dev(perm)
    ws = B.workspace(d, B.STAGE_EXPERT_SCATTER)
    y = torch.empty((w.T, w.d), dtype=torch.float32, device="cuda")
    y_sc = torch.full((w.T, w.d), float("nan"), dtype=torch.float32, device="cuda")
    y_sc2 = torch.full_like(y_sc, float("nan"))
    P.omnimoe_expert_forward(d, dev["x"], dev["u"], dev["v"], gi, gg, gp, y)
    P.omnimoe_expert_forward_scatter(d, dev["x"], dev["u"], dev["v"], gi, gg, gp, y_sc, ws=ws)
    P.omnimoe_expert_forward_scatter(d, dev["x"], dev["u"], dev["v"], gi, gg, gp, y_sc2, ws=ws)
    torch.cuda.synchronize()
    y_sc, y_sc2 = y_sc.cpu().numpy(), y_sc2.cpu().numpy()
    assert np.array_equal(y_sc.view(np.uint8), y_sc2.view(np.uint8))
    err = row_rel_err(y_sc, y_ref)
    say(f"  max row rel err {err.max():.3e}")
    assert err.max() <= tol(w)
    if w.dtype == "f32" or not (w.H == 1 and w.K * 64 >= w.N):  # not the dense routed sum
        assert row_rel_err(y_sc, y.cpu().numpy().astype(np.float64)).max() <= 1e-5


@pytest.mark.parametrize("name", ["dense_bf16", "dense_k100_bf16"])
def test_dense_routed_sum(name):
    # y = A V with A[t, e] = a_p rounded to bf16: within tolerance of the oracle, the same on a
    # second run, and within the bf16 rounding of a (plus fp32 sums) of the slot-order sum of
    # the token-centric kernel, which keeps a in fp32.
    say(f"[dense routed sum] {name}")
    w, dev, idx, g32, perm, y_ref = _expert_case(name)
    d = B.make_desc(w)
    gi, gg = to_dev(idx), to_dev(g32)
    y = torch.empty((w.T, w.d), dtype=torch.float32, device="cuda")
    y2 = torch.empty_like(y)
    y_tc = torch.empty_like(y)
    P.omnimoe_expert_forward(d, dev["x"], dev["u"], dev["v"], gi, gg, to_dev(perm), y)
    P.omnimoe_expert_forward(d, dev["x"], dev["u"], dev["v"], gi, gg, to_dev(perm), y2)
    P.omnimoe_expert_forward_token_centric(d, dev["x"], dev["u"], dev["v"], gi, gg, y_tc)
    torch.cuda.synchronize()
    y, y2, y_tc = y.cpu().numpy(), y2.cpu().numpy(), y_tc.cpu().numpy()
    assert np.array_equal(y.view(np.uint8), y2.view(np.uint8))
    err = row_rel_err(y, y_ref)
    say(f"  max row rel err {err.max():.3e}")
    assert err.max() <= tol(w)
    # |a_p| = g_p |act(x_t . u_e)| <= g_p ||x_t|| ||u_e|| (|GELU(z)|, |SiLU(z)| <= |z|)
    _, f = host_inputs(w)
    xn = np.linalg.norm(f["x"].astype(np.float64), axis=1)
    un = np.linalg.norm(f["u"].astype(np.float64), axis=1)
    va = np.abs(f["v"].astype(np.float64))
    flat = idx.reshape(w.T, -1)
    a = g32.reshape(w.T, -1).astype(np.float64) * xn[:, None] * un[flat]
    mass = np.zeros((w.T, w.d))
    for j in range(flat.shape[1]):
        mass += a[:, j:j + 1] * va[flat[:, j]]
    bound = mass * (2.0 ** -8 + 2 * (flat.shape[1] + 4) * 2.0 ** -24) + 1e-30
    gap = np.abs(y.astype(np.float64) - y_tc)
    say(f"  max gap / bound {(gap / bound).max():.3e}")
    assert np.all(gap <= bound)


GROUP_ROWS_CASES = [
    # (shape, B): the second product of Eq. 14 per group (partial rows per (group, token)
    # slot): small and large groups, one group holding every expert, B = 1, wide d (several
    # 512-column chunks), K > 64 and the paper's grid, many slot tiles per group
    ("small_bf16", 2), ("small_bf16", 64), ("k64_bf16", 33), ("all_experts_bf16", 1 << 20),
    ("k64_bf16", 1), ("wide_bf16", 3), ("shared_bf16", 48), ("k256_bf16", 64),
    ("paper_k512_bf16", 320), ("bucket_bf16", 100), ("dense_bf16", 8),
]


@pytest.mark.parametrize("case", GROUP_ROWS_CASES, ids=[f"{n}-B{b}" for n, b in GROUP_ROWS_CASES])
def test_expert_forward_group_rows(case):
    # Within tolerance of the oracle, the same bits on a second run, and element-wise within the
    # reordering bound of the slot-order sum: both paths form the same a[p] (the grouped dot)
    # and add the same H K terms a_p v_e per token in fp32, in two orders (each within
    # gamma_{HK} sum |a v| of the exact sum).
    name, Bg = case
    w = SHAPES[name].with_(group_size=Bg)
    say(f"[group rows] {name} B={Bg}")
    inp, f = host_inputs(w)
    dev = upload(inp)
    dsc = oracle.desc(w)
    sr, sc = oracle.half_scores(dsc, f["x"], f["keys_row"], f["keys_col"])
    idx, _, g64, _ = oracle.select(dsc, sr, sc, oracle.CARTESIAN)
    g32 = g64.astype(np.float32)
    perm, active, _, _ = oracle.schedule(dsc, idx)
    act_pad = np.zeros(min(w.M, w.N), dtype=np.int32)
    act_pad[:len(active)] = active
    gi, gg, gp, ga = to_dev(idx), to_dev(g32), to_dev(perm), to_dev(act_pad)
    na = torch.tensor([len(active)], dtype=torch.int32, device="cuda")
    d = B.make_desc(w)
    ys = []
    for _ in range(2):
        y = torch.full((w.T, w.d), float("nan"), dtype=torch.float32, device="cuda")
        P.omnimoe_expert_forward_group_rows(d, dev["x"], dev["u"], dev["v"], gi, gg, gp, ga, na, y)
        ys.append(y)
    y_ref_path = torch.empty((w.T, w.d), dtype=torch.float32, device="cuda")
    P.omnimoe_expert_forward_grouped(d, dev["x"], dev["u"], dev["v"], gi, gg, gp, ga, na,
                                     y_ref_path)
    torch.cuda.synchronize()
    y0, y1, yg = (t.cpu().numpy() for t in (ys[0], ys[1], y_ref_path))
    assert np.array_equal(y0.view(np.uint8), y1.view(np.uint8))
    y_ref = oracle.expert_forward(dsc, f["x"], f["u"], f["v"], idx, g32.astype(np.float64))
    err = row_rel_err(y0, y_ref)
    n = w.H * w.K
    gam = 2.02 * (n + 1) * 2.0 ** -24 / (1 - (n + 1) * 2.0 ** -24)
    # |a_p| <= g_p |x_t . u_e| (|act(z)| <= |z|), computed in fp64 from the inputs
    flat = idx.reshape(w.T, -1)
    xu = np.abs(np.einsum("td,tnd->tn", f["x"].astype(np.float64),
                          f["u"][flat].astype(np.float64)))
    amag = g32.reshape(w.T, -1).astype(np.float64) * xu * 1.01
    mass = np.einsum("tn,tnd->td", amag, np.abs(f["v"][flat].astype(np.float64)))
    gap = np.abs(y0.astype(np.float64) - yg)
    say(f"  max row rel err {err.max():.3e}; max gap / bound {(gap / (gam * mass + 1e-30)).max():.3e}")
    assert err.max() <= tol(w)
    if not (w.H == 1 and w.K * 64 >= w.N):  # the grouped path's own sum is the slot-order one
        assert np.all(gap <= gam * mass + 1e-30)


def test_expert_forward_group_rows_rejects_fp32():
    w = SHAPES["ragged_f32"].with_(group_size=4)
    inp, _ = host_inputs(w)
    dev = upload(inp)
    z = torch.zeros(w.M, dtype=torch.int32, device="cuda")
    y = torch.empty((w.T, w.d), dtype=torch.float32, device="cuda")
    with pytest.raises(B.OmnimoeError) as ei:
        P.omnimoe_expert_forward_group_rows(B.make_desc(w), dev["x"], dev["u"], dev["v"], z,
                                            z.float(), z, z, z[:1], y,
                                            ws=torch.empty(1 << 20, dtype=torch.uint8,
                                                           device="cuda"))
    assert "unsupported" in str(ei.value)


@pytest.mark.parametrize("name", ["dense_bf16", "dense_k100_bf16", "dense_wide_bf16",
                                  "dense_all_bf16", "dense_silu_bf16"])
def test_dense_expert_dot_layer(name):
    # One head with K >= N / 64 and groups of one expert: the layer forms the a_p inside one dense
    # product x U^T over all experts (gate and activation kept at the selected cells only) and
    # sums y = A V densely, with no schedule. The same bits on a second run, and on the layer's
    # own routing within an element-wise bound of the token-centric stage (a in fp32, slot-order
    # sums): A holds each a_p rounded to bf16 once (2^-9 |a|); the x . u sums run in another
    # order (at most 2 d 2^-24 ||x|| ||u|| apart, times |act'| <= 1.13); the two y sums (H K
    # terms, plus the split partials) each within gamma_n of the exact one.
    w = SHAPES[name]
    d = B.make_desc(w)
    assert P.omnimoe_layer_path(d) == B.PATH_DENSE_SUM | B.PATH_DENSE_DOT
    assert not P.omnimoe_layer_path(B.make_desc(w.with_(group_size=4))) & B.PATH_DENSE_DOT
    say(f"[dense expert dot, layer] {name}")
    inp, f = host_inputs(w)
    dev = upload(inp)
    y, idx, g = gpu_layer(w, dev)
    y2, idx2, g2 = gpu_layer(w, dev)
    assert np.array_equal(y.view(np.uint8), y2.view(np.uint8)) and np.array_equal(idx, idx2)
    y_tc = torch.empty((w.T, w.d), dtype=torch.float32, device="cuda")
    P.omnimoe_expert_forward_token_centric(d, dev["x"], dev["u"], dev["v"], to_dev(idx),
                                           to_dev(g), y_tc)
    torch.cuda.synchronize()
    y_tc = y_tc.cpu().numpy().astype(np.float64)
    xn = np.linalg.norm(f["x"].astype(np.float64), axis=1)
    un = np.linalg.norm(f["u"].astype(np.float64), axis=1)
    va = np.abs(f["v"].astype(np.float64))
    flat = idx.reshape(w.T, -1)
    a = g.reshape(w.T, -1).astype(np.float64) * xn[:, None] * un[flat]
    mass = np.zeros((w.T, w.d))
    for j in range(flat.shape[1]):
        mass += a[:, j:j + 1] * va[flat[:, j]]
    n = flat.shape[1] + 520
    bound = mass * (2.0 ** -8 + (2.3 * w.d + 2 * n) * 2.0 ** -24) + 1e-30
    gap = np.abs(y.astype(np.float64) - y_tc)
    say(f"  max gap / bound {(gap / bound).max():.3e}; max row rel err "
        f"{row_rel_err(y, y_tc).max():.3e}")
    assert np.all(gap <= bound)


@pytest.mark.parametrize("grouped", [False, True])
def test_dense_routed_sum_repeated_ids(grouped):
    # Caller-supplied idx may name one expert in several slots of a token (the router never
    # does): the dense routed sum must add every such slot, as the oracle does, the same way on
    # every run. Token 0 repeats one expert twice, token 5 three times, token 9 in every slot.
    name = "dense_bf16"
    w = SHAPES[name].with_(group_size=8 if grouped else 1)
    say(f"[dense routed sum, repeated ids] {name} grouped={grouped}")
    inp, f = host_inputs(w)
    dev = upload(inp)
    dsc = oracle.desc(w)
    sr, sc = oracle.half_scores(dsc, f["x"], f["keys_row"], f["keys_col"])
    idx, _, g64, _ = oracle.select(dsc, sr, sc, oracle.CARTESIAN)
    idx = idx.copy()
    idx[0, 0, 1] = idx[0, 0, 0]
    idx[5, 0, [3, 7, 40]] = idx[5, 0, 2]
    idx[9, 0, :] = idx[9, 0, 0]
    g32 = g64.astype(np.float32)
    perm, active, _, _ = oracle.schedule(dsc, idx)
    gi, gg = to_dev(idx), to_dev(g32)
    ys = []
    for _ in range(2):
        y = torch.full((w.T, w.d), float("nan"), dtype=torch.float32, device="cuda")
        if grouped:
            act_pad = np.zeros(min(w.M, w.N), dtype=np.int32)
            act_pad[:len(active)] = active
            na = torch.tensor([len(active)], dtype=torch.int32, device="cuda")
            P.omnimoe_expert_forward_grouped(B.make_desc(w), dev["x"], dev["u"], dev["v"], gi,
                                             gg, to_dev(perm), to_dev(act_pad), na, y)
        else:
            P.omnimoe_expert_forward(B.make_desc(w), dev["x"], dev["u"], dev["v"], gi, gg,
                                     to_dev(perm), y)
        torch.cuda.synchronize()
        ys.append(y.cpu().numpy())
    assert np.array_equal(ys[0].view(np.uint8), ys[1].view(np.uint8))
    y_ref = oracle.expert_forward(dsc, f["x"], f["u"], f["v"], idx, g32.astype(np.float64))
    err = row_rel_err(ys[0], y_ref)
    say(f"  max row rel err {err.max():.3e} (tokens 0, 5, 9: {err[[0, 5, 9]].max():.3e})")
    assert err.max() <= tol(w)


# ------------------------------------------------------------------ whole layer

def layer_parity(w, y, idx, g, hs, route_idx, route_g, x_f32, kr, kc, rows_of, tokens=None):
    """The GPU layer's outputs (y, idx, g over all T tokens) against the oracle.

    * the layer and omnimoe_route (which also returns the fp32 logits hs) route identically;
    * P1, every token: the oracle's selection on the GPU's own fp32 logits equals idx bit for
      bit, gates within GATE_TOL;
    * on `tokens` (all by default), with the oracle's fp64 logits: logit error delta, routing
      by compare_routing (certified positions exact; containment, band and order elsewhere),
      gates against the fp64 softmax of the exact scores of the GPU's picks, and y against
      the oracle's expert forward on the GPU's own idx and gates (no token is left out).
    rows_of(name, ids) returns rows `ids` of table "u" or "v" as float32."""
    assert np.array_equal(idx, route_idx), "layer and route select differently"
    assert np.array_equal(g.view(np.uint32), route_g.view(np.uint32))
    ri, _, rg, inexact = oracle.select_f32(oracle.desc(w), hs, oracle.CARTESIAN)
    assert inexact == 0
    p1 = np.all(idx == ri, axis=-1)
    assert p1.all(), f"P1: selection of the GPU logits differs on {int((~p1).sum())} rows"
    np.testing.assert_allclose(g, rg, rtol=GATE_TOL, atol=1e-7)
    if tokens is None:
        tokens = np.arange(w.T)
    ws = w.with_(T=len(tokens))
    dsc = oracle.desc(ws)
    xs = x_f32[tokens]
    sr, sc = oracle.half_scores(dsc, xs, kr, kc)
    hs_t = hs[tokens]
    delta = max(float(np.abs(hs_t[..., :w.n_rows] - sr).max()),
                float(np.abs(hs_t[..., w.n_rows:] - sc).max()), 1e-300)
    del hs_t
    it, ig = idx[tokens], g[tokens]
    unc, unc_rows, npos = compare_routing(ws, it, sr, sc, delta)
    gerr = gate_bound_check(ig, sr, sc, it, w.n_cols, delta, GATE_TOL)
    del sr, sc
    ids = np.unique(it)
    remap = np.searchsorted(ids, it).astype(np.int32)
    u, v = rows_of("u", ids), rows_of("v", ids)
    y_ref = oracle.expert_forward(dsc, xs, u, v, remap, ig.astype(np.float64))
    del u, v
    err = row_rel_err(y[tokens], y_ref)
    say(f"  {w.name}: P1 rows {idx.shape[0] * idx.shape[1]} exact; logit err {delta:.2e}; "
        f"uncertified positions {unc} of {npos} (rows {unc_rows}); max gate rel err {gerr:.2e}; "
        f"tokens compared {len(tokens)}/{w.T}; max row rel err {err.max():.3e}")
    assert err.max() <= tol(w)
    return {"uncertified": unc, "positions": npos, "delta": delta, "err": float(err.max())}


@pytest.mark.parametrize("name", list(SHAPES))
def test_layer_forward(name):
    w = SHAPES[name]
    say(f"[layer] {name}")
    inp, f = host_inputs(w)
    dev = upload(inp)
    y, idx, g = gpu_layer(w, dev)
    hs, ri, rg = gpu_half_scores(w, dev)
    layer_parity(w, y, idx, g, hs, ri, rg, f["x"], f["keys_row"], f["keys_col"],
                 lambda name, ids: f[name][ids])
    # the oracle's own whole layer (its fp64 routing) on the tokens routed identically
    y_orc, idx_orc, _ = oracle.layer_forward(oracle.desc(w), f["x"], f["keys_row"],
                                              f["keys_col"], f["u"], f["v"])
    same = np.all(idx == idx_orc, axis=(1, 2))
    assert same.mean() > 0.5
    assert row_rel_err(y, y_orc)[same].max() <= tol(w)


@pytest.mark.parametrize("name", ["fused_k1_bf16", "fused_k3_bf16", "fused_k64_bf16",
                                  "small_bf16"])
def test_fused_selection_dot_matches_expert_stage(name):
    # Where the selection kernel forms the slot-order a_p (omnimoe_layer_path), the layer's y must
    # equal, bit for bit, the expert stage launched on its own (omnimoe_expert_forward, the
    # expert-major dot) on the layer's own routing: both form every a_p the same way.
    w = SHAPES[name]
    d = B.make_desc(w)
    assert P.omnimoe_layer_path(d) & B.PATH_SELECT_DOT
    say(f"[fused selection + dot] {name}")
    inp, _ = host_inputs(w)
    dev = upload(inp)
    y, idx, g = gpu_layer(w, dev)
    perm, _, _, _ = oracle.schedule(oracle.desc(w), idx)
    y2 = torch.empty((w.T, w.d), dtype=torch.float32, device="cuda")
    P.omnimoe_expert_forward(d, dev["x"], dev["u"], dev["v"], to_dev(idx), to_dev(g),
                             to_dev(perm), y2)
    torch.cuda.synchronize()
    assert np.array_equal(y.view(np.uint8), y2.cpu().numpy().view(np.uint8))


def test_layer_is_deterministic():
    w = W["small_bf16"]
    inp, _ = host_inputs(w)
    dev = upload(inp)
    a = gpu_layer(w, dev)
    b = gpu_layer(w, dev)
    for x, z in zip(a, b):
        assert np.array_equal(x.view(np.uint8), z.view(np.uint8))


@pytest.mark.parametrize("name", ["small_bf16", "decode64_like_bf16", "grouped_b64_bf16",
                                  "grouped_k256_b100_bf16", "dense_wide_bf16"])
def test_layer_graph_replays_match_eager(name):
    # The layer call allocates nothing and clears with kernels only, so it can be captured in a
    # HIP graph; every replay (with other eager work and synchronisations in between) must
    # reproduce the eager result bit for bit, idx and gates included.
    w = {"small_bf16": W["small_bf16"],
         "decode64_like_bf16": SHAPES["skinny_bf16"].with_(T=64),
         # groups of B > 1: the grouped GEMM, its plan and the group sort inside the graph
         "grouped_b64_bf16": W["small_bf16"].with_(group_size=64),
         "grouped_k256_b100_bf16": SHAPES["k256_bf16"].with_(group_size=100),
         # both products dense over all experts (selection mask, masked-activation GEMM)
         "dense_wide_bf16": SHAPES["dense_wide_bf16"]}[name]
    inp, _ = host_inputs(w)
    dev = upload(inp)
    y_ref, idx_ref, g_ref = gpu_layer(w, dev)
    d = B.make_desc(w)
    ws = B.workspace(d, B.STAGE_LAYER)
    y = torch.empty((w.T, w.d), dtype=torch.float32, device="cuda")
    idx = torch.empty((w.T, w.H, w.K), dtype=torch.int32, device="cuda")
    g = torch.empty((w.T, w.H, w.K), dtype=torch.float32, device="cuda")
    graph = torch.cuda.CUDAGraph()
    cap = torch.cuda.Stream()
    cap.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(cap):
        with torch.cuda.graph(graph, stream=cap):
            P.omnimoe_layer_forward(d, dev["x"], dev["keys_row"], dev["keys_col"], dev["u"],
                                    dev["v"], y, idx, g, ws=ws, stream=cap)
    torch.cuda.current_stream().wait_stream(cap)
    torch.cuda.synchronize()
    for rep in range(3):
        y.fill_(float("nan"))
        idx.fill_(-1)
        ws.fill_(0xAB)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert np.array_equal(y.cpu().numpy().view(np.uint8), y_ref.view(np.uint8)), rep
        assert np.array_equal(idx.cpu().numpy(), idx_ref), rep
        assert np.array_equal(g.cpu().numpy().view(np.uint8), g_ref.view(np.uint8)), rep
        _ = gpu_layer(w, dev)  # eager work between replays


def test_zero_input_closed_form():
    w = SHAPES["ragged_bf16"]
    inp, _ = host_inputs(w)
    inp["x"] = np.zeros_like(inp["x"])
    y, idx, g = gpu_layer(w, upload(inp))
    assert np.array_equal(idx, np.broadcast_to(np.arange(w.K, dtype=np.int32), idx.shape))
    np.testing.assert_allclose(g, 1.0 / w.K, rtol=1e-6)
    assert np.all(y == 0.0)


def test_timed_layer_matches_and_reports():
    w = W["small_bf16"]
    inp, _ = host_inputs(w)
    dev = upload(inp)
    y0, _, _ = gpu_layer(w, dev)
    d = B.make_desc(w)
    ws = B.workspace(d, B.STAGE_LAYER)
    y = torch.empty((w.T, w.d), dtype=torch.float32, device="cuda")
    t = B.Timer(4)
    for _ in range(3):
        t.layer_forward(d, dev["x"], dev["keys_row"], dev["keys_col"], dev["u"], dev["v"], y, ws)
    ms, n = t.read()
    t.close()
    assert n == 3 and all(v > 0 for v in ms.values())
    assert np.array_equal(y.cpu().numpy(), y0)


# ------------------------------------------------------------------ full-size shapes

@pytest.fixture(scope="module")
def train_tables():
    """Sub-keys and expert tables of the 1024^2-expert, d=2048 layer, on the GPU (8 GiB)."""
    w = W["train_bf16"]
    kr, kc = synth.make_keys(w)
    dev = {"keys_row": to_dev(kr), "keys_col": to_dev(kc)}
    for name in ("u", "v"):
        dev[name] = to_dev(synth.make_expert_rows(w, name))
        gc.collect()
    yield dev, synth.as_f32(kr), synth.as_f32(kc)
    dev.clear()
    torch.cuda.empty_cache()


def _full_parity(w, dev, kr, kc, tokens=None):
    """Full-size GPU layer against the oracle on every token (or on `tokens`); the expert rows
    the compared tokens reach are drawn by id."""
    x = synth.make_x(w)
    d = dict(dev, x=to_dev(x))
    y, idx, g = gpu_layer(w, d)
    hs, ri, rg = gpu_half_scores(w, d)
    del d
    torch.cuda.empty_cache()

    def rows_of(name, ids):
        return synth.as_f32(synth.make_expert_rows(w, name, rows=ids))

    st = layer_parity(w, y, idx, g, hs, ri, rg, synth.as_f32(x), kr, kc, rows_of, tokens)
    del hs
    gc.collect()
    return y, idx, st


def test_train_shape_full(train_tables):
    # Every one of the 16384 tokens: P1 on the GPU's logits, routing against the fp64 oracle,
    # gates, and y against the oracle on the GPU's routing.
    dev, kr, kc = train_tables
    w = W["train_bf16"]
    say("[full] train_bf16 T=16384, all tokens")
    y, idx, st = _full_parity(w, dev, kr, kc)
    assert np.isfinite(y).all()
    assert st["uncertified"] < 0.01 * st["positions"]


def test_skewed_shape_full(train_tables):
    # Same expert tables as the training shape (same seed and streams), skewed sub-keys.
    dev, _, _ = train_tables
    w = W["skew_bf16"]
    say("[full] skew_bf16 T=16384, all tokens")
    kr, kc = synth.make_keys(w)
    dev = dict(dev, keys_row=to_dev(kr), keys_col=to_dev(kc))
    y, idx, st = _full_parity(w, dev, synth.as_f32(kr), synth.as_f32(kc))
    counts = np.bincount(idx.ravel(), minlength=w.N)
    share = np.sort(counts)[::-1][: w.N // 10].sum() / idx.size
    say(f"  top-10% share {share:.4f}, active {int((counts > 0).sum())}, max {counts.max()}")
    assert abs(share - 0.50) < 0.02


def test_dp_share_shape_full(train_tables):
    # 2048 tokens against the full tables: one GPU's share of a data-parallel split.
    dev, kr, kc = train_tables
    w = W["dp8share_bf16"]
    say("[full] dp8share_bf16 T=2048, all tokens")
    y, idx, _ = _full_parity(w, dev, kr, kc)
    assert np.isfinite(y).all()


PAPER_CASES = [("paper_k512_bf16", 1), ("paper_k512_bf16", 64), ("paper_k512_bf16", 320),
               ("paper_k4096_bf16", 1), ("paper_k4096_bf16", 64), ("paper_k4096_bf16", 320),
               # the benchmark table's sweeps: K = 1024 .. 4096 at 1k tokens, 1k .. 16k tokens
               # at K = 512
               ("paper_t1k_k1024_bf16", 64), ("paper_t1k_k2048_bf16", 1),
               ("paper_t1k_k2048_bf16", 64), ("paper_t1k_k4096_bf16", 1),
               ("paper_t1k_k4096_bf16", 64),
               ("paper_t1k_k512_bf16", 64), ("paper_t2k_k512_bf16", 64),
               ("paper_t8k_k512_bf16", 64), ("paper_t16k_k512_bf16", 64),
               ("paper_t16k_k512_bf16", 1)]


@pytest.mark.parametrize("case", PAPER_CASES, ids=[f"{n}-B{b}" for n, b in PAPER_CASES])
def test_paper_benchmark_shapes_full(case):
    # The paper's speed-benchmark shape: 4096 tokens, 320 x 320 experts of d = 1024, one head,
    # K = 512 and 4096 (about 16.8 M tasks at K = 4096), every token checked; with groups of
    # B > 1 experts the expert stage is the grouped GEMM (B = 64: slot tiles split by token
    # range over the XCDs; B = 320: one grid row of experts per group).
    name, Bg = case
    w = W[name].with_(group_size=Bg)
    say(f"[full] {name} T={w.T} K={w.K} B={Bg}, all tokens")
    kr, kc = synth.make_keys(w)
    dev = {"keys_row": to_dev(kr), "keys_col": to_dev(kc),
           "u": to_dev(synth.make_expert_rows(w, "u")), "v": to_dev(synth.make_expert_rows(w, "v"))}
    y, idx, _ = _full_parity(w, dev, synth.as_f32(kr), synth.as_f32(kc))
    assert np.isfinite(y).all()


@pytest.mark.parametrize("name", ["decode64_bf16", "decode1_bf16"])
def test_decode_shapes(train_tables, name):
    dev, kr, kc = train_tables
    w = W[name]
    say(f"[full] {name}")
    _full_parity(w, dev, kr, kc)


# ------------------------------------------------------------------ dense router (ablation)

DENSE_SHAPES = {
    "tiny_f32": W["tiny_f32"],
    "ragged_bf16": RAGGED,
    "odd_n_bf16": synth.Workload("odd_n_bf16", T=100, d=128, n_rows=7, n_cols=9, d_key=64, H=2,
                                 K=5),
    "k64_bf16": SHAPES["k64_bf16"],
    "wide_rows_bf16": synth.Workload("wide_rows_bf16", T=512, d=128, n_rows=128, n_cols=128,
                                     d_key=64, H=1, K=16),
    # 64 tokens: the skinny logit kernel, 65536-wide rows
    "small64_bf16": W["small_bf16"].with_(name="small64_bf16", T=64),
    # one token: the few-token logit kernel on a single (N-wide) half, the other half empty
    "one_token_bf16": W["small_bf16"].with_(name="one_token_bf16", T=1),
}


@pytest.mark.parametrize("name", list(DENSE_SHAPES))
def test_route_dense(name):
    w = DENSE_SHAPES[name]
    say(f"[dense route] {name} T={w.T} d={w.d} N={w.N} H={w.H} K={w.K}")
    x = synth.make_x(w)
    wg = synth.make_gate_table(w)
    xf, wgf = synth.as_f32(x), synth.as_f32(wg)
    d = B.make_desc(w)
    L = torch.empty((w.T, w.H, w.N), dtype=torch.float32, device="cuda")
    idx = torch.empty((w.T, w.H, w.K), dtype=torch.int32, device="cuda")
    g = torch.empty((w.T, w.H, w.K), dtype=torch.float32, device="cuda")
    P.omnimoe_route_dense(d, to_dev(x), to_dev(wg), idx, g, logits=L)
    # the same call through the workspace (no logits buffer) gives the same selection
    idx2 = torch.empty_like(idx)
    g2 = torch.empty_like(g)
    P.omnimoe_route_dense(d, to_dev(x), to_dev(wg), idx2, g2)
    torch.cuda.synchronize()
    L, idx, g = L.cpu().numpy(), idx.cpu().numpy(), g.cpu().numpy()
    assert np.array_equal(idx, idx2.cpu().numpy())
    assert np.array_equal(g, g2.cpu().numpy())
    dsc = oracle.desc(w)
    ref_idx, ref_g, ref_L = oracle.route_dense(dsc, xf, wgf, with_logits=True)
    bound = higham_bound(xf, wgf)
    err = np.abs(L - ref_L)
    assert np.all(err <= bound + 1e-30)
    # selection on the GPU's own logits is exact
    si, sg = oracle.select_dense_f32(dsc, L)
    assert np.array_equal(idx, si)
    np.testing.assert_allclose(g, sg, rtol=GATE_TOL, atol=1e-7)
    # against the fp64 router: exact wherever the top-(K+1) gaps exceed twice the logit error
    delta = max(float(err.max()), 1e-300)
    srt = -np.sort(-ref_L, axis=-1)[..., : w.K + 1]
    cert = (-np.diff(srt, axis=-1)).min(axis=-1) > 2 * delta if w.K < w.N else \
        np.ones(srt.shape[:-1], bool)
    assert np.array_equal(idx[cert], ref_idx[cert])
    say(f"  max logit err {delta:.3e}, uncertified rows {int((~cert).sum())} of {w.T * w.H}")


@pytest.mark.parametrize("n,K,tie", [(4096, 16, False), (65536, 64, False), (63, 5, False),
                                     (4096, 64, True), (65536, 16, True), (1000, 1000 // 16, True)])
def test_select_dense_bitexact(n, K, tie):
    rng = np.random.default_rng(n + K)
    T, H = 24, 2
    if tie:
        L = rng.integers(-3, 4, size=(T, H, n)).astype(np.float32)
        L[0, 0, :] = 0.0
        L[1, 0, ::2] = -0.0
    else:
        L = rng.standard_normal((T, H, n)).astype(np.float32)
    nr = 1
    while n % (nr * 2) == 0 and nr * 2 <= 4096 and n // (nr * 2) >= 1 and nr < 64:
        nr *= 2
    w = synth.Workload("sel", T=T, d=16, n_rows=nr, n_cols=n // nr, d_key=8, H=H, K=K)
    say(f"[dense select] n={n} K={K} tie={tie}")
    idx = torch.empty((T, H, K), dtype=torch.int32, device="cuda")
    g = torch.empty((T, H, K), dtype=torch.float32, device="cuda")
    P.omnimoe_select_dense(B.make_desc(w), to_dev(L), idx, g)
    torch.cuda.synchronize()
    ri, rg = oracle.select_dense_f32(oracle.desc(w), L)
    assert np.array_equal(idx.cpu().numpy(), ri)
    np.testing.assert_allclose(g.cpu().numpy(), rg, rtol=GATE_TOL, atol=1e-7)


# ------------------------------------------------------------------ shared dense MLP (Eq. 7)

MLP_CASES = {
    "tiny_f32": (W["tiny_f32"], 64),
    "ragged_bf16": (RAGGED, 104),
    "small_bf16": (W["small_bf16"], 512),
    "skinny_bf16": (SHAPES["skinny_bf16"], 512),
    "few_token_bf16": (SHAPES["skinny1_bf16"], 512),
    # a decode step's width: both projections on the few-token kernel with 2048-wide rows and
    # an empty second half
    "decode1_bf16": (W["decode1_bf16"], 2048),
    "few3_bf16": (SHAPES["few3_bf16"], 384),
    "wide_f32": (SHAPES["wide_f32"], 1024),
}


def _mlp_parity(w, d_ff, tokens=None):
    x = synth.make_x(w)
    w_gu, w_down = synth.make_mlp_weights(w, d_ff)
    rng = np.random.default_rng(w.T + d_ff)
    y0 = rng.standard_normal((w.T, w.d)).astype(np.float32)
    y = to_dev(y0.copy())
    P.omnimoe_shared_mlp(B.make_desc(w), d_ff, to_dev(x), to_dev(w_gu), to_dev(w_down), y)
    torch.cuda.synchronize()
    y = y.cpu().numpy()
    tok = np.arange(w.T) if tokens is None else tokens
    dsc = oracle.desc(w, T=len(tok))
    ref = oracle.shared_mlp(dsc, synth.as_f32(x[tok]), synth.as_f32(w_gu),
                            synth.as_f32(w_down), y=y0[tok])
    # error relative to the MLP term itself (y0 only shifts both sides)
    err = row_rel_err(y[tok] - y0[tok], ref - y0[tok])
    say(f"  max row rel err {err.max():.3e}")
    assert err.max() <= tol(w)


@pytest.mark.parametrize("name", list(MLP_CASES))
def test_shared_mlp(name):
    w, d_ff = MLP_CASES[name]
    say(f"[mlp] {name} T={w.T} d={w.d} d_ff={d_ff}")
    _mlp_parity(w, d_ff)


def test_shared_mlp_train_shape_sampled():
    w = W["train_bf16"]
    say("[mlp] train_bf16 T=16384 d=2048 d_ff=2048, sampled tokens")
    rng = np.random.default_rng(5)
    tokens = np.unique(np.concatenate([[0, w.T - 1], rng.choice(w.T, 30, replace=False)]))
    _mlp_parity(w, 2048, tokens)


# ------------------------------------------------------------------ plain-C caller of the ABI

@pytest.mark.parametrize("name", ["tiny_f32", "small_bf16"])
def test_c_abi_caller(name, tmp_path):
    # tests/abi_c/layer_main calls omnimoe_workspace_size and omnimoe_layer_forward from C with
    # hipMalloc'd buffers (no Python in the loop); its output must equal the binding's bit for
    # bit and the oracle's within tolerance.
    import os
    import subprocess
    w = W[name]
    exe = os.path.join(os.path.dirname(os.path.abspath(__file__)), "abi_c", "layer_main")
    assert os.path.exists(exe), "build() compiles tests/abi_c/layer_main"
    inp, f = host_inputs(w)
    d = B.make_desc(w)
    src, dst = tmp_path / "in.bin", tmp_path / "out.bin"
    with open(src, "wb") as fh:
        fh.write(bytes(d))
        for k in ("x", "keys_row", "keys_col", "u", "v"):
            fh.write(np.ascontiguousarray(inp[k]).tobytes())
    say(f"[c abi] {name}")
    r = subprocess.run([exe, str(src), str(dst)], capture_output=True, text=True, timeout=120)
    say(r.stdout.strip(), r.stderr.strip())
    assert r.returncode == 0
    raw = np.fromfile(dst, dtype=np.uint8)
    ny, nm = w.T * w.d * 4, w.M * 4
    assert raw.size == ny + 2 * nm
    y = raw[:ny].view(np.float32).reshape(w.T, w.d)
    idx = raw[ny:ny + nm].view(np.int32).reshape(w.T, w.H, w.K)
    g = raw[ny + nm:].view(np.float32).reshape(w.T, w.H, w.K)
    y_b, idx_b, g_b = gpu_layer(w, upload(inp))
    assert np.array_equal(y.view(np.uint8), y_b.view(np.uint8))
    assert np.array_equal(idx, idx_b) and np.array_equal(g.view(np.uint8), g_b.view(np.uint8))
    dsc = oracle.desc(w)
    sr, sc = oracle.half_scores(dsc, f["x"], f["keys_row"], f["keys_col"])
    ref_idx, _, ref_g, _ = oracle.select(dsc, sr, sc, oracle.CARTESIAN)
    same = np.all(idx == ref_idx, axis=(1, 2))
    y_ref = oracle.expert_forward(dsc, f["x"], f["u"], f["v"], ref_idx, ref_g)
    assert row_rel_err(y, y_ref)[same].max() <= tol(w)


# ------------------------------------------------------------------ expert backward

@pytest.mark.parametrize("name", ["tiny_f32", "small_bf16", "ragged_bf16", "ragged_f32",
                                  "silu_k1_bf16", "k64_bf16", "all_experts_bf16", "k256_bf16"])
def test_expert_backward(name):
    w, dev, idx, g32, perm, _ = _expert_case(name)
    say(f"[backward] {name}")
    dsc = oracle.desc(w)
    _, act_ref, off_ref, _ = oracle.schedule(dsc, idx)
    rng = np.random.default_rng(len(name))
    dy = rng.standard_normal((w.T, w.d)).astype(np.float32)
    A = min(w.M, w.N)
    out = {k: torch.full(shape, float("nan"), dtype=torch.float32, device="cuda") for k, shape in
           [("dx", (w.T, w.d)), ("du", (A, w.d)), ("dv", (A, w.d)), ("dg", (w.T, w.H, w.K)),
            ("ds", (w.T, w.H, w.K))]}
    off = torch.full((A + 1,), -1, dtype=torch.int32, device="cuda")
    off[: len(off_ref)] = to_dev(off_ref)
    na = torch.tensor([len(act_ref)], dtype=torch.int32, device="cuda")
    d = B.make_desc(w)
    args = (d, dev["x"], dev["u"], dev["v"], to_dev(idx), to_dev(g32), to_dev(perm), off, na,
            to_dev(dy), out["dx"], out["du"], out["dv"], out["dg"], out["ds"])
    P.omnimoe_expert_backward(*args)
    torch.cuda.synchronize()
    got = {k: v.cpu().numpy() for k, v in out.items()}
    ref = oracle.expert_backward(dsc, synth.as_f32(synth.make_x(w)),
                                 synth.as_f32(synth.make_expert_rows(w, "u")),
                                 synth.as_f32(synth.make_expert_rows(w, "v")), idx,
                                 g32.astype(np.float64), dy.astype(np.float64))
    n = len(ref["active"])
    assert np.array_equal(ref["active"], act_ref)
    # Element-wise bounds: a token whose h = x . u nearly cancels has an fp32 dot error that is
    # large relative to h itself, so a relative tolerance per row would not hold; the bound
    # follows the dot products' error (Higham) through the backward formulas.
    kind = 1 if w.act == "silu" else 0
    bnd = backward_error_bounds(
        synth.as_f32(synth.make_x(w)), synth.as_f32(synth.make_expert_rows(w, "u")),
        synth.as_f32(synth.make_expert_rows(w, "v")), idx, g32, dy,
        np.vectorize(lambda z: oracle.act(kind, z)), np.vectorize(lambda z: oracle.act_grad(kind, z)))
    pairs = {"dx": (got["dx"], ref["dx"], bnd["dx"]),
             "du": (got["du"][:n], ref["du_rows"], bnd["du"]),
             "dv": (got["dv"][:n], ref["dv_rows"], bnd["dv"]),
             "dgates": (got["dg"], ref["dgates"], bnd["dgates"]),
             "dscores": (got["ds"], ref["dscores"], bnd["dscores"])}
    for k, (gv, rv, bv) in pairs.items():
        err = np.abs(gv.astype(np.float64) - rv)
        ratio = (err / (2 * bv + 1e-30)).max()
        say(f"  {k}: max row rel err {row_rel_err(gv.reshape(rv.shape[0], -1), rv.reshape(rv.shape[0], -1)).max():.2e}, "
            f"max err / bound {ratio:.2f}")
        assert np.all(err <= 2 * bv + 1e-30), k
    # same bits on a second run
    P.omnimoe_expert_backward(*args)
    torch.cuda.synchronize()
    for k, v in out.items():
        rows = n if k in ("du", "dv") else None
        assert np.array_equal(v.cpu().numpy()[:rows].view(np.uint8), got[k][:rows].view(np.uint8))


@pytest.mark.parametrize("name", ["tiny_f32", "small_bf16", "ragged_bf16", "ragged_f32",
                                  "shared_bf16", "k256_bf16", "skinny_bf16"])
def test_route_backward(name):
    w = SHAPES[name]
    say(f"[route backward] {name}")
    inp, f = host_inputs(w)
    dsc = oracle.desc(w)
    sr, sc = oracle.half_scores(dsc, f["x"], f["keys_row"], f["keys_col"])
    idx, _, _, _ = oracle.select(dsc, sr, sc, oracle.CARTESIAN)
    rng = np.random.default_rng(7 + len(name))
    ds = rng.standard_normal((w.T, w.H, w.K)).astype(np.float32)
    dx0 = rng.standard_normal((w.T, w.d)).astype(np.float32)
    dev = upload(inp)
    dx = to_dev(dx0.copy())
    dkr = torch.full((w.H, w.n_rows, w.d_key), float("nan"), dtype=torch.float32, device="cuda")
    dkc = torch.full((w.H, w.n_cols, w.d_key), float("nan"), dtype=torch.float32, device="cuda")
    P.omnimoe_route_backward(B.make_desc(w), dev["x"], dev["keys_row"], dev["keys_col"],
                             to_dev(idx), to_dev(ds), dx, dkr, dkc)
    torch.cuda.synchronize()
    got = (dx.cpu().numpy(), dkr.cpu().numpy(), dkc.cpu().numpy())
    ref = oracle.route_backward(dsc, f["x"], f["keys_row"], f["keys_col"], idx, ds, dx=dx0)
    # the same sums over absolute values bound the fp32 summation error (Higham): gamma_n times
    # the sum of |terms|, n the number of terms of the element
    absb = oracle.route_backward(dsc, np.abs(f["x"]), np.abs(f["keys_row"]),
                                 np.abs(f["keys_col"]), idx, np.abs(ds), dx=np.abs(dx0))
    u = 2.0 ** -23
    hk = w.H * w.K
    i_r = (np.arange(w.H)[None, :, None] * w.n_rows + idx // w.n_cols).ravel()
    i_c = (np.arange(w.H)[None, :, None] * w.n_cols + idx % w.n_cols).ravel()
    n_r = np.bincount(i_r, minlength=w.H * w.n_rows).reshape(w.H, w.n_rows, 1) + 1
    n_c = np.bincount(i_c, minlength=w.H * w.n_cols).reshape(w.H, w.n_cols, 1) + 1
    for k, gv, rv, ab, n in (("dx", got[0], ref[0], absb[0], 2 * hk + 2),
                             ("dkeys_row", got[1], ref[1], absb[1], n_r),
                             ("dkeys_col", got[2], ref[2], absb[2], n_c)):
        bound = 2 * (n * u / (1 - n * u)) * ab + 1e-30
        err = np.abs(gv.astype(np.float64) - rv)
        say(f"  {k}: max err / bound {(err / bound).max():.3f}")
        assert np.all(err <= bound), k
