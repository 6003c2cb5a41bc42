"""omnimoe_layer_forward_noalloc (workspace in the library's static scratch) against
omnimoe_layer_forward (caller workspace): the same kernels on the same inputs, so y, idx and
gates must be identical bit for bit, on two calls in a row, the second with fewer tokens (the
scratch keeps the first call's contents)."""
import sys

import numpy as np
import pytest

import synth
from gpu_support import to_dev

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
import paper_2602_05711_amd as P  # noqa: E402
from paper_2602_05711_amd import binding as B  # noqa: E402


def say(*a):
    print(*a, file=sys.stderr, flush=True)


CASES = [
    # (shape, group size, tokens of the first call, tokens of the second)
    ("small_bf16", 1, 4096, 1000),      # per-task dot, token-major accumulate
    ("small_bf16", 16, 2048, 333),      # grouped expert GEMM (Eq. 14, B > 1)
    ("dense_bf16", 1, 300, 77),         # one head, K >= N / 64: the dense routed sum
    ("tiny_f32", 1, 256, 100),          # fp32 layer
]
DENSE = synth.Workload("dense_bf16", T=300, d=256, n_rows=32, n_cols=32, d_key=64, H=1, K=64)


def _outputs(w, T):
    y = torch.full((T, w.d), float("nan"), dtype=torch.float32, device="cuda")
    idx = torch.full((T, w.H, w.K), -1, dtype=torch.int32, device="cuda")
    g = torch.full((T, w.H, w.K), float("nan"), dtype=torch.float32, device="cuda")
    return y, idx, g


@pytest.mark.parametrize("case", CASES, ids=[f"{c[0]}-B{c[1]}" for c in CASES])
def test_noalloc_matches_layer_forward(case):
    name, Bg, T1, T2 = case
    base = DENSE if name == "dense_bf16" else synth.WORKLOADS[name]
    w = base.with_(group_size=Bg, T=T1)
    say(f"[noalloc] {name} B={Bg} T={T1} then T={T2}")
    inp = synth.make_inputs(w)
    dev = {k: to_dev(v) for k, v in inp.items()}
    x1 = dev["x"]
    x2 = to_dev(np.ascontiguousarray(inp["x"][::-1][:T2]))  # other tokens, fewer of them
    for x in (x1, x2):
        T = x.shape[0]
        d = B.make_desc(w, T=T)
        ref = _outputs(w, T)
        P.omnimoe_layer_forward(d, x, dev["keys_row"], dev["keys_col"], dev["u"], dev["v"], *ref)
        got = _outputs(w, T)
        P.omnimoe_layer_forward_noalloc(d, x, dev["keys_row"], dev["keys_col"], dev["u"],
                                        dev["v"], *got)
        torch.cuda.synchronize()
        for r, o in zip(ref, got):
            r, o = r.cpu().numpy(), o.cpu().numpy()
            assert np.array_equal(r.view(np.uint8), o.view(np.uint8)), f"T={T}"
        assert np.isfinite(got[0].cpu().numpy()).all()
        say(f"  T={T}: identical to omnimoe_layer_forward")
