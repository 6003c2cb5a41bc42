"""The C ABI library loads, exports what include/omnimoe.h declares, and rejects bad arguments
before touching the GPU (these calls return from the host-side checks, so they run without one)."""
import ctypes
import os
import re

import pytest

import paper_2602_05711_amd as P
from paper_2602_05711_amd import binding as B
import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
OK, INVALID, UNSUPPORTED, ALIGN, WORKSPACE = 0, 1, 2, 3, 4


def _declared_functions():
    with open(os.path.join(ROOT, "include", "omnimoe.h")) as f:
        text = f.read()
    return sorted(set(re.findall(r"^(?:omnimoe_status|const char\*)\s+(omnimoe_\w+)\(", text,
                                 flags=re.M)))


def test_header_matches_exports():
    lib = P.load_library()
    names = _declared_functions()
    assert len(names) == 23
    assert sorted(P.EXPORTED) == names
    for n in names:
        assert hasattr(lib, n), n


def test_descriptor_layout_matches_header():
    # int64 T followed by ten int32 fields: 8 + 40 bytes.
    assert ctypes.sizeof(B.OmnimoeLayerDesc) == 48
    assert B.OmnimoeLayerDesc.d.offset == 8


def _ws(desc, stage=B.STAGE_LAYER):
    n = ctypes.c_size_t(0)
    st = P.load_library().omnimoe_workspace_size(ctypes.byref(desc), stage, ctypes.byref(n))
    return st, n.value


@pytest.mark.parametrize("field,value,status", [
    ("K", 4097, UNSUPPORTED), ("K", 0, INVALID), ("d", 100, INVALID), ("d", 0, INVALID),
    ("d_key", 300, INVALID), ("d_key", 12, INVALID), ("n_rows", 0, INVALID),
    ("n_rows", 4097, INVALID), ("H", 0, INVALID), ("dtype", 7, INVALID), ("act", 3, INVALID),
    ("query_mode", 2, INVALID), ("group_size", 0, INVALID),
    ("T", -1, INVALID),
])
def test_workspace_size_rejects(field, value, status):
    d = B.make_desc(synth.WORKLOADS["small_bf16"])
    setattr(d, field, value)
    assert _ws(d)[0] == status


def test_group_sizes_are_accepted():
    d = B.make_desc(synth.WORKLOADS["small_bf16"])
    for b in (2, 7, 1 << 20):
        d.group_size = b
        assert _ws(d)[0] == OK


def test_wide_fp32_is_unsupported():
    d = B.make_desc(synth.WORKLOADS["tiny_f32"])
    d.d = 8192
    assert _ws(d)[0] == UNSUPPORTED
    d.dtype = B.OMNIMOE_BF16
    assert _ws(d)[0] == OK


def test_k_above_grid_is_invalid():
    d = B.make_desc(synth.WORKLOADS["tiny_f32"])
    d.n_rows, d.n_cols, d.K = 2, 3, 7
    assert _ws(d)[0] == INVALID


def test_shared_query_allows_full_width_keys():
    d = B.make_desc(synth.WORKLOADS["small_bf16"])
    d.d_key = 512
    assert _ws(d)[0] == INVALID
    d.query_mode = B.OMNIMOE_QUERY_SHARED
    assert _ws(d)[0] == OK


def test_workspace_sizes_cover_buffers():
    w = synth.WORKLOADS["train_bf16"]
    d = B.make_desc(w)
    st, route = _ws(d, B.STAGE_ROUTE)
    assert st == OK and route >= w.T * w.H * (w.n_rows + w.n_cols) * 4
    st, layer = _ws(d, B.STAGE_LAYER)
    assert st == OK and layer >= route + 3 * w.M * 4
    assert _ws(d, 11)[0] == INVALID
    # groups of B: partial rows for min(M, ceil(min(M, N) / B) T) slots of d floats
    pg = synth.WORKLOADS["paper_t1k_k1024_bf16"].with_(group_size=320)
    st, rows = _ws(B.make_desc(pg), B.STAGE_EXPERT_GROUP_ROWS)
    bound = min(pg.M, -(-min(pg.M, pg.N) // 320) * pg.T)
    assert st == OK and rows >= pg.M * 4 + bound * pg.d * 4 and bound == 320 * 1024
    st, scatter = _ws(d, B.STAGE_EXPERT_SCATTER)
    assert st == OK and scatter >= w.M * 4 + w.M * w.d * 4  # a[] and the contribution rows
    st, grouped = _ws(d, B.STAGE_EXPERT_GROUPED)
    assert st == OK and grouped >= w.M * 4 + w.N * 4 + 2 * w.M * 4
    st, dense = _ws(d, B.STAGE_ROUTE_DENSE)
    assert st == OK and dense >= w.T * w.H * w.N * 4
    # one head with K >= N / 64: the routed sum is one dense product, whose bf16 A [T, N] and
    # V transposed [d, N] live in the expert and layer workspaces
    p = synth.WORKLOADS["paper_k4096_bf16"]
    dp = B.make_desc(p)
    st, ex = _ws(dp, B.STAGE_EXPERT)
    assert st == OK and ex >= p.M * 4 + p.T * p.N * 2 + p.d * p.N * 2
    st, lay = _ws(dp, B.STAGE_LAYER)
    # the layer's dense first product adds each token's selection mask and prefix counts
    # ([T, N / 32] each) and its gates in expert-id order
    assert st == OK and lay >= ex + 2 * p.T * (p.N // 32) * 4 + p.M * 4
    dp.K = 1024  # below N / 64: the slot-order sum, no dense buffers
    st, ex2 = _ws(dp, B.STAGE_EXPERT)
    assert st == OK and ex2 < p.T * p.N * 2


def test_entry_points_check_pointers_before_launch():
    lib = P.load_library()
    d = B.make_desc(synth.WORKLOADS["tiny_f32"])
    a = ctypes.c_void_p(0x10000)   # aligned, never dereferenced: the checks fail first
    bad = ctypes.c_void_p(0x10004)
    n = ctypes.c_size_t
    D = ctypes.byref(d)
    assert lib.omnimoe_route(D, None, a, a, a, a, None, a, n(1 << 30), None) == INVALID
    assert lib.omnimoe_route(D, bad, a, a, a, a, None, a, n(1 << 30), None) == ALIGN
    assert lib.omnimoe_route(D, a, a, a, a, a, None, a, n(16), None) == WORKSPACE
    assert lib.omnimoe_select(D, a, a, None, None, n(0), None) == INVALID
    assert lib.omnimoe_schedule(D, a, a, a, a, a, bad, a, n(1 << 30), None) == ALIGN
    assert lib.omnimoe_schedule(D, a, a, a, a, a, None, a, n(8), None) == WORKSPACE
    assert lib.omnimoe_expert_forward(D, a, a, a, a, a, None, a, a, n(1 << 30), None) == INVALID
    assert lib.omnimoe_expert_forward_token_centric(D, a, a, None, a, a, a, None) == INVALID
    assert lib.omnimoe_expert_forward_scatter(D, a, a, a, a, a, None, a, a, n(1 << 40),
                                              None) == INVALID
    assert lib.omnimoe_expert_forward_scatter(D, a, a, a, a, a, a, a, bad, n(1 << 40),
                                              None) == ALIGN
    assert lib.omnimoe_expert_forward_scatter(D, a, a, a, a, a, a, a, a, n(16),
                                              None) == WORKSPACE
    assert lib.omnimoe_expert_forward_grouped(D, a, a, a, a, a, a, None, a, a, a, n(1 << 40),
                                              None) == INVALID
    assert lib.omnimoe_expert_forward_grouped(D, a, a, a, a, a, a, a, bad, a, a, n(1 << 40),
                                              None) == ALIGN
    # fp32 tables: the grouped path runs on bf16 matrix cores only
    assert lib.omnimoe_expert_forward_grouped(D, a, a, a, a, a, a, a, a, a, a, n(1 << 40),
                                              None) == UNSUPPORTED
    db = B.make_desc(synth.WORKLOADS["small_bf16"])
    assert lib.omnimoe_expert_forward_grouped(ctypes.byref(db), a, a, a, a, a, a, a, a, a, a,
                                              n(16), None) == WORKSPACE
    db.d = 520  # d % 64 != 0
    assert lib.omnimoe_expert_forward_grouped(ctypes.byref(db), a, a, a, a, a, a, a, a, a, a,
                                              n(1 << 40), None) == UNSUPPORTED
    assert lib.omnimoe_route_dense(D, a, None, a, a, None, a, n(1 << 40), None) == INVALID
    assert lib.omnimoe_route_dense(D, a, a, a, a, None, a, n(16), None) == WORKSPACE
    assert lib.omnimoe_route_dense(D, a, a, a, a, bad, a, n(16), None) == ALIGN
    assert lib.omnimoe_select_dense(D, a, bad, a, None) == ALIGN
    assert lib.omnimoe_expert_backward(D, a, a, a, a, a, a, a, a, a, a, a, a, a, None, a,
                                       n(1 << 40), None) == INVALID
    assert lib.omnimoe_expert_backward(D, a, a, a, a, a, a, a, a, a, a, a, a, a, a, a, n(4),
                                       None) == WORKSPACE
    assert lib.omnimoe_route_backward(D, a, a, a, a, a, a, a, a, a, n(4), None) == WORKSPACE
    assert lib.omnimoe_route_backward(D, a, a, a, a, None, a, a, a, a, n(1 << 40),
                                      None) == INVALID
    assert lib.omnimoe_shared_mlp(D, 12, a, a, a, a, a, n(1 << 40), None) == INVALID
    assert lib.omnimoe_shared_mlp(D, 64, a, a, a, a, a, n(16), None) == WORKSPACE
    assert lib.omnimoe_shared_mlp(D, 64, a, a, bad, a, a, n(1 << 40), None) == ALIGN
    sz = ctypes.c_size_t(0)
    assert lib.omnimoe_shared_mlp_workspace_size(D, 64, ctypes.byref(sz)) == OK
    assert sz.value >= 256 * 64 * 4 * 3
    assert lib.omnimoe_expert_forward_token_centric(D, a, a, a, a, a, bad, None) == ALIGN
    assert lib.omnimoe_layer_forward(D, a, a, a, a, a, a, None, None, a, n(8), None) == WORKSPACE
    assert lib.omnimoe_layer_forward(D, a, a, a, a, a, a, bad, None, a, n(1 << 40), None) == ALIGN
    assert lib.omnimoe_layer_forward_timed(D, a, a, a, a, a, a, None, None, a, n(1 << 40), None,
                                           None) == INVALID
    assert lib.omnimoe_layer_forward_noalloc(D, a, a, a, a, a, bad, None, None, None) == ALIGN
    assert lib.omnimoe_layer_forward_noalloc(D, a, a, a, a, a, a, None, bad, None) == ALIGN
    assert lib.omnimoe_layer_forward_noalloc(D, a, a, a, None, a, a, None, None, None) == INVALID


def test_noalloc_rejects_shapes_beyond_its_scratch():
    # The layer workspace of the shape must fit the library's static scratch; larger shapes
    # are refused before any device call (this runs without a GPU).
    with open(os.path.join(ROOT, "include", "omnimoe.h")) as f:
        m = re.search(r"#define OMNIMOE_NOALLOC_SCRATCH_BYTES \(([\d\s*]+)\)", f.read())
    assert m and eval(m.group(1)) == B.NOALLOC_SCRATCH_BYTES
    lib = P.load_library()
    a = ctypes.c_void_p(1 << 20)
    w = synth.WORKLOADS["train_bf16"]
    for T, fits in ((16384, False), (900, True), (1000, False)):
        d = B.make_desc(w, T=T)
        need = ctypes.c_size_t(0)
        assert lib.omnimoe_workspace_size(ctypes.byref(d), B.STAGE_LAYER, ctypes.byref(need)) == OK
        assert (need.value <= B.NOALLOC_SCRATCH_BYTES) == fits, (T, need.value)
        if not fits:
            assert lib.omnimoe_layer_forward_noalloc(ctypes.byref(d), a, a, a, a, a, a, None,
                                                     None, None) == WORKSPACE


def test_zero_tokens_is_a_noop():
    lib = P.load_library()
    d = B.make_desc(synth.WORKLOADS["small_bf16"], T=0)
    D = ctypes.byref(d)
    n = ctypes.c_size_t
    assert lib.omnimoe_route(D, None, None, None, None, None, None, None, n(0), None) == OK
    assert lib.omnimoe_expert_forward(D, None, None, None, None, None, None, None, None, n(0),
                                      None) == OK
    assert lib.omnimoe_expert_forward_token_centric(D, None, None, None, None, None, None,
                                                    None) == OK
    assert lib.omnimoe_expert_forward_scatter(D, None, None, None, None, None, None, None, None,
                                              n(0), None) == OK
    assert lib.omnimoe_layer_forward(D, None, None, None, None, None, None, None, None, None,
                                     n(0), None) == OK
    assert lib.omnimoe_layer_forward_noalloc(D, None, None, None, None, None, None, None, None,
                                             None) == OK


def test_status_strings():
    lib = P.load_library()
    assert lib.omnimoe_status_string(0) == b"ok"
    assert lib.omnimoe_status_string(4) == b"workspace too small"
    assert lib.omnimoe_status_string(99) == b"unknown status"


def test_binding_raises_on_error():
    d = B.make_desc(synth.WORKLOADS["small_bf16"])
    d.K = 5000
    with pytest.raises(B.OmnimoeError):
        B.omnimoe_workspace_size(d, B.STAGE_LAYER)


def test_layer_path_flags():
    # Host-side only: which kernels the layer runs for a descriptor.
    f = {w: P.omnimoe_layer_path(B.make_desc(synth.WORKLOADS[w]))
         for w in ("train_bf16", "skew_bf16", "decode1_bf16", "decode64_bf16", "dp8share_bf16",
                   "small_bf16", "tiny_f32", "paper_k512_bf16", "paper_k4096_bf16")}
    assert f["train_bf16"] == B.PATH_SCHEDULE and f["skew_bf16"] == B.PATH_SCHEDULE
    # a decode step forms no schedule; with 512 (token, head) rows the selection forms the dot,
    # with 8 a separate kernel does
    assert f["decode1_bf16"] == 0
    assert f["decode64_bf16"] == B.PATH_SELECT_DOT
    assert f["dp8share_bf16"] == B.PATH_SELECT_DOT and f["small_bf16"] == B.PATH_SELECT_DOT
    assert f["tiny_f32"] == 0  # fp32: no fused selection
    assert f["paper_k512_bf16"] == B.PATH_SCHEDULE
    # one head with K >= N / 64 and groups of one expert: both products dense over all experts
    assert f["paper_k4096_bf16"] == B.PATH_DENSE_SUM | B.PATH_DENSE_DOT
    grouped = B.make_desc(synth.WORKLOADS["paper_k4096_bf16"].with_(group_size=64))
    assert P.omnimoe_layer_path(grouped) == B.PATH_SCHEDULE | B.PATH_GROUPED | B.PATH_DENSE_SUM
    bad = B.make_desc(synth.WORKLOADS["small_bf16"])
    bad.K = 0
    with pytest.raises(P.OmnimoeError):
        P.omnimoe_layer_path(bad)
    assert P.load_library().omnimoe_layer_path(ctypes.byref(bad), None) == INVALID
