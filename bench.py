#!/usr/bin/env python3
"""Throughput of the atomic-expert layer forward on one MI355X.

One step = one omnimoe_layer_forward call (router GEMM, selection, schedule, expert compute)
over the whole batch of seeded synthetic tokens, inputs resident in HBM. Prints one JSON line:
tokens/s, the roofline fraction of the dominant kernel (timed with HIP events on the call's
stream) and the oracle's throughput on a bounded token sample on the host cores.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "atomic-expert layer fwd tokens/sec on 1 MI355X; achieved HBM GB/s & MFMA util"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0      # dense bf16 MFMA
FP32_PEAK_TFLOPS = 157.3       # fp32 vector


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def kernel_sources_hash(files):
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, "paper_2602_05711_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


# Source files each kernel group is built from (a counter file stays valid while they match).
KERNEL_FILES = {
    "score": ["score_gemm.hip", "device_common.hpp"],
    "select": ["select.hip", "device_common.hpp"],
    "schedule": ["schedule.hip", "device_common.hpp"],
    "expert_dot": ["expert.hip", "device_common.hpp"],
    "accumulate": ["expert.hip", "device_common.hpp"],
}


def algorithmic_work(w, n_active):
    """Per-launch algorithmic bytes (or FLOP) of each kernel group, from the layer's own sizes."""
    s_in = 2 if w.bf16 else 4
    M, T, d = w.M, w.T, w.d
    return {
        # 2 T H (n_rows + n_cols) d_key FLOP (App. A, Eq. ii per head)
        "score": ("mfma" if w.bf16 else "alu",
                  2.0 * T * w.H * (w.n_rows + w.n_cols) * w.d_key),
        # read the fp32 logits once, write idx and gates
        "select": ("hbm", 4.0 * T * w.H * (w.n_rows + w.n_cols) + 8.0 * M),
        # read idx, write perm, active list and offsets
        "schedule": ("hbm", 4.0 * M + 4.0 * M + 8.0 * n_active),
        # each active u row once, each token row once, perm/idx/gate in and a out per task
        "expert_dot": ("hbm", float(n_active) * d * s_in + T * d * s_in + 16.0 * M),
        # each active v row once, y written once, a and idx read per task
        "accumulate": ("hbm", float(n_active) * d * s_in + T * d * 4.0 + 8.0 * M),
    }


def load_traffic(kernel, workload):
    """HBM bytes per launch from the committed rocprofv3 counter summary, or None when the
    kernel's sources changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    if t.get("sources_sha256_16") != kernel_sources_hash(KERNEL_FILES[kernel]):
        return None
    return t.get("bytes_per_launch")


def load_mfma_busy(kernel, workload):
    """MFMA-busy fraction of a matrix-core kernel from the committed rocprofv3 counter summary
    (SQ_VALU_MFMA_BUSY_CYCLES over the SIMDs' cycles in the kernel), or None when absent or the
    kernel's sources changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_mfma.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    if t.get("sources_sha256_16") != kernel_sources_hash(KERNEL_FILES[kernel]):
        return None
    return {k: t[k] for k in ("mfma_busy", "simd_cycles", "mfma_busy_cycles", "normalisation")
            if k in t}


def routing_stats(idx, N):
    """Expert usage of one batch: active experts, usage, KL(z || uniform), top-10% share."""
    import numpy as np
    counts = np.bincount(idx.ravel(), minlength=N)
    z = counts[counts > 0] / idx.size
    top = np.sort(counts)[::-1]
    return {"n_active": int((counts > 0).sum()), "usage": float((counts > 0).mean()),
            "kl_to_uniform": float(np.sum(z * np.log(z * N))),
            "top10pct_share": float(top[: max(1, N // 10)].sum() / idx.size),
            "max_segment": int(top[0])}


def cpu_bruteforce(w, inp, sample_tokens, threads):
    """Oracle selection by the plain definition (all n_rows x n_cols cells per token and head)
    on the first `sample_tokens` tokens; the logits are computed outside the timed region."""
    import oracle
    import synth

    T = min(sample_tokens, w.T)
    dsc = oracle.desc(w, T=T)
    sr, sc = oracle.half_scores(dsc, synth.as_f32(inp["x"][:T]), synth.as_f32(inp["keys_row"]),
                                synth.as_f32(inp["keys_col"]), n_threads=threads)
    t0 = time.perf_counter()
    oracle.select(dsc, sr, sc, oracle.BRUTE, n_threads=threads)
    dt = time.perf_counter() - t0
    return {"value": T / dt, "unit": "tokens/s", "cores": threads,
            "sample": f"brute-force top-{w.K} over all {w.N} cells, first {T} tokens, {dt:.1f} s"}


def cpu_baseline(w, inp, sample_tokens, threads):
    """Oracle (route + schedule + scheduled forward) on the first `sample_tokens` tokens."""
    import numpy as np
    import oracle
    import synth

    T = min(sample_tokens, w.T)
    x = synth.as_f32(inp["x"][:T])
    kr = synth.as_f32(inp["keys_row"])
    kc = synth.as_f32(inp["keys_col"])
    dsc = oracle.desc(w, T=T)
    # Expert rows the sample reaches, drawn by id and stored compactly (float32 copies of the
    # full tables would not fit twice in host memory); the monotone id remap keeps the order.
    sr, sc = oracle.half_scores(dsc, x, kr, kc, n_threads=threads)
    idx, _, _, _ = oracle.select(dsc, sr, sc, oracle.CARTESIAN, n_threads=threads)
    ids = np.unique(idx)
    u = synth.as_f32(synth.make_expert_rows(w, "u", rows=ids))
    v = synth.as_f32(synth.make_expert_rows(w, "v", rows=ids))
    # Timed: logits, Cartesian selection and gates, then the scheduled (expert-major) forward.
    t0 = time.perf_counter()
    sr, sc = oracle.half_scores(dsc, x, kr, kc, n_threads=threads)
    idx, _, g, _ = oracle.select(dsc, sr, sc, oracle.CARTESIAN, n_threads=threads)
    remap = np.searchsorted(ids, idx).astype(np.int32)
    oracle.expert_forward(dsc, x, u, v, remap, g, scheduled=True, n_threads=threads)
    dt = time.perf_counter() - t0
    return {"value": T / dt, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": f"first {T} of {w.T} tokens of {w.name} (full router over all "
                      f"{w.n_rows}x{w.n_cols} sub-keys, Cartesian selection, schedule, "
                      f"expert-major forward), fp64, {dt:.1f} s on {threads} threads of "
                      f"{cpu_model()}"}


def host_threads():
    """Threads for the oracle leg: every core this process may run on, unless the job's CPU
    share is set smaller (OMP_NUM_THREADS, as on a one-GPU job that is allotted 16 cores)."""
    affinity = len(os.sched_getaffinity(0))
    share = os.environ.get("OMP_NUM_THREADS", "")
    threads = min(affinity, int(share)) if share.isdigit() and int(share) > 0 else affinity
    return max(1, threads), {"nproc": os.cpu_count(), "affinity": affinity,
                             "omp_num_threads": share or None, "cpu_model": cpu_model()}


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown CPU"


def extras(args, w, desc, d_in, dev, idx, g, y, stream, per, ms_step, ev0, ev1, sched):
    """The shared SwiGLU branch and the two ablations of Table 3, timed like the layer."""
    import torch
    import paper_2602_05711_amd as P
    import synth as _synth

    # Ablation of the schedule (Table 3, "w/o Expert-Centric Scheduling"): the same expert
    # compute token by token, each task gathering its own u and v rows.
    y_tc = torch.empty_like(y)
    tc = lambda: P.omnimoe_expert_forward_token_centric(  # noqa: E731
        desc, d_in["x"], d_in["u"], d_in["v"], idx, g, y_tc, stream=stream)
    for _ in range(2):
        tc()
    ev0.record(stream)
    for _ in range(args.steps):
        tc()
    ev1.record(stream)
    torch.cuda.synchronize()
    tc_ms = ev0.elapsed_time(ev1) / args.steps
    # The layer's dot: its own kernel group, or, where the selection kernel forms it, the
    # selection group less the plain selection on the same logits.
    dot_ms = per["expert_dot"]
    if P.omnimoe_layer_path(desc) & P.binding.PATH_SELECT_DOT:
        hs = torch.empty((w.T, w.H, w.n_rows + w.n_cols), dtype=torch.float32, device="cuda")
        i2, g2 = torch.empty_like(idx), torch.empty_like(g)
        P.omnimoe_route(desc, d_in["x"], d_in["keys_row"], d_in["keys_col"], i2, g2,
                        half_scores=hs, stream=stream)
        sel = lambda: P.omnimoe_select(desc, hs, i2, g2, stream=stream)  # noqa: E731
        for _ in range(2):
            sel()
        ev0.record(stream)
        for _ in range(args.steps):
            sel()
        ev1.record(stream)
        torch.cuda.synchronize()
        dot_ms = max(per["select"] - ev0.elapsed_time(ev1) / args.steps, 0.0)
        del hs, i2, g2
    ec_ms = per["schedule"] + dot_ms + per["accumulate"]
    ablation = {"token_centric_expert_ms": tc_ms, "expert_centric_expert_ms": ec_ms,
                "token_over_expert_centric": tc_ms / ec_ms,
                "same_y": bool(torch.equal(y_tc, y))}
    log(f"expert stage: expert-centric (schedule + dot + accumulate) {ec_ms:.3f} ms, "
        f"token-centric {tc_ms:.3f} ms")
    del y_tc

    # The accumulate in expert-major order (v read once per expert run): contribution rows
    # a_p v_e [M, d] fp32, then a token-major sum in slot order. Same dot kernel in front.
    contrib = None
    perm = sched[0]
    sc_bytes = P.omnimoe_workspace_size(desc, P.binding.STAGE_EXPERT_SCATTER)
    if sc_bytes <= (64 << 30):
        ws_sc = torch.empty(sc_bytes, dtype=torch.uint8, device="cuda")
        y_sc = torch.empty_like(y)
        sc = lambda: P.omnimoe_expert_forward_scatter(  # noqa: E731
            desc, d_in["x"], d_in["u"], d_in["v"], idx, g, perm, y_sc, ws=ws_sc, stream=stream)
        for _ in range(2):
            sc()
        ev0.record(stream)
        for _ in range(args.steps):
            sc()
        ev1.record(stream)
        torch.cuda.synchronize()
        sc_ms = ev0.elapsed_time(ev1) / args.steps
        slot_ms = dot_ms + per["accumulate"]
        den = y.abs().amax(dim=1).clamp_min(1e-30)
        rel = float(((y_sc - y).abs().amax(dim=1) / den).max())
        contrib = {"dot_scatter_reduce_ms": sc_ms, "dot_accumulate_ms": slot_ms,
                   "ratio": sc_ms / slot_ms, "buffer_bytes": sc_bytes,
                   "max_row_rel_diff": rel}
        log(f"contribution rows: dot + scatter + reduce {sc_ms:.3f} ms against dot + "
            f"slot-order accumulate {slot_ms:.3f} ms")
        del ws_sc, y_sc

    # The full OmniMoE FFN adds the shared dense SwiGLU branch (Eq. 7) to the routed output;
    # its width here is d_ff = d, the ratio of the paper's benchmark configuration.
    d_ff = w.d
    gu, dn = _synth.make_mlp_weights(w, d_ff)
    gu, dn = dev(gu), dev(dn)
    ws_mlp = torch.empty(P.omnimoe_shared_mlp_workspace_size(desc, d_ff), dtype=torch.uint8,
                         device="cuda")
    mlp = lambda: P.omnimoe_shared_mlp(  # noqa: E731
        desc, d_ff, d_in["x"], gu, dn, y, ws=ws_mlp, stream=stream)
    for _ in range(2):
        mlp()
    ev0.record(stream)
    for _ in range(args.steps):
        mlp()
    ev1.record(stream)
    torch.cuda.synchronize()
    mlp_ms = ev0.elapsed_time(ev1) / args.steps
    mlp_flop = 2.0 * w.T * w.d * 3 * d_ff
    shared_mlp = {"d_ff": d_ff, "ms": mlp_ms, "TFLOPs": mlp_flop / (mlp_ms * 1e-3) / 1e12,
                  "ffn_ms": ms_step + mlp_ms, "routed_share": ms_step / (ms_step + mlp_ms)}
    log(f"shared SwiGLU branch (d_ff={d_ff}): {mlp_ms:.3f} ms; routed layer + branch "
        f"{ms_step + mlp_ms:.3f} ms")
    del gu, dn, ws_mlp

    # Ablation of the router (Table 3, "w/o Cartesian Product Router"): a dense router with a
    # gating vector per expert, all N logits per (token, head) materialised.
    dense_bytes = w.T * w.H * w.N * 4
    if w.K > 64:
        no_cpr = {"skipped": "the dense router's selection takes K <= 64"}
    elif dense_bytes <= (8 << 30):
        wg = dev(_synth.make_gate_table(w))
        wsd = P.workspace(desc, 5)
        idx_d, g_d = torch.empty_like(idx), torch.empty_like(g)
        rd = lambda: P.omnimoe_route_dense(  # noqa: E731
            desc, d_in["x"], wg, idx_d, g_d, ws=wsd, stream=stream)
        for _ in range(2):
            rd()
        ev0.record(stream)
        for _ in range(args.steps):
            rd()
        ev1.record(stream)
        torch.cuda.synchronize()
        dr_ms = ev0.elapsed_time(ev1) / args.steps
        cr_ms = per["score"] + per["select"]
        no_cpr = {"dense_route_ms": dr_ms, "cartesian_route_ms": cr_ms,
                  "route_ratio": dr_ms / cr_ms, "logit_bytes": dense_bytes,
                  "layer_ratio": (dr_ms + ec_ms) / (cr_ms + ec_ms)}
        log(f"router: Cartesian {cr_ms:.3f} ms, dense over all {w.N} experts {dr_ms:.3f} ms")
        del wg, wsd
    else:
        no_cpr = {"skipped": f"the dense logits would take {dense_bytes / 2**30:.0f} GiB"}

    # The grouped expert GEMM (Eq. 14): the same layer with groups of B active experts, per kernel
    # group (the schedule then adds the group sort, the expert stage the group plan).
    grouped = None
    gb = args.grouped_b
    if gb > 1 and w.group_size == 1 and w.bf16 and w.d % 64 == 0:
        wg = w.with_(group_size=gb)
        dg = P.make_desc(wg)
        wsg = P.workspace(dg, 4)
        yg = torch.empty_like(y)
        for _ in range(2):
            P.omnimoe_layer_forward(dg, d_in["x"], d_in["keys_row"], d_in["keys_col"], d_in["u"],
                                    d_in["v"], yg, ws=wsg, stream=stream)
        tg = P.Timer(args.steps)
        for _ in range(args.steps):
            tg.layer_forward(dg, d_in["x"], d_in["keys_row"], d_in["keys_col"], d_in["u"],
                             d_in["v"], yg, wsg, stream=stream)
        msg, ng = tg.read()
        tg.close()
        perg = {k: v / ng for k, v in msg.items()}
        y1 = torch.empty_like(y)  # the per-task layer again (y itself now holds the MLP too)
        P.omnimoe_layer_forward(desc, d_in["x"], d_in["keys_row"], d_in["keys_col"], d_in["u"],
                                d_in["v"], y1, stream=stream)
        torch.cuda.synchronize()
        rel = float(((yg - y1).abs().amax(dim=1) / y1.abs().amax(dim=1).clamp_min(1e-30)).max())
        grouped = {"group_size": gb, "per_kernel_ms": perg, "layer_ms": sum(perg.values()),
                   "expert_stage_ms": perg["expert_dot"] + perg["accumulate"],
                   "per_task_expert_stage_ms": dot_ms + per["accumulate"],
                   "max_row_rel_diff_vs_per_task": rel}
        del y1
        log(f"grouped GEMM, B={gb}: layer {grouped['layer_ms']:.3f} ms (dot "
            f"{perg['expert_dot']:.3f} ms vs per-task {dot_ms:.3f} ms)")
        del wsg, yg

    # The second product of Eq. 14 per group (partial rows per (group, token) slot, then a
    # token-major sum over groups) against the grouped path's slot-order sum, for each B.
    group_rows = None
    if w.bf16 and w.d % 64 == 0 and args.group_rows_b:
        group_rows = []
        for gb in [int(b) for b in args.group_rows_b.split(",")]:
            wg = w.with_(group_size=gb)
            dg = P.make_desc(wg)
            need = P.omnimoe_workspace_size(dg, 10)
            if need > (8 << 30):
                group_rows.append({"group_size": gb, "skipped": f"workspace {need / 2**30:.1f} GiB"})
                continue
            permg = torch.empty(w.M, dtype=torch.int32, device="cuda")
            cap = min(w.M, w.N)
            actg = torch.empty(cap, dtype=torch.int32, device="cuda")
            offg = torch.empty(cap + 1, dtype=torch.int32, device="cuda")
            nag = torch.empty(1, dtype=torch.int32, device="cuda")
            P.omnimoe_schedule(dg, idx, permg, actg, offg, nag)
            wsr = P.workspace(dg, 10)
            wsq = P.workspace(dg, 8)
            yr = torch.empty_like(y)
            yq = torch.empty_like(y)
            runs = {
                "group_rows": lambda: P.omnimoe_expert_forward_group_rows(
                    dg, d_in["x"], d_in["u"], d_in["v"], idx, g, permg, actg, nag, yr, ws=wsr,
                    stream=stream),
                "grouped_slot_order_sum": lambda: P.omnimoe_expert_forward_grouped(
                    dg, d_in["x"], d_in["u"], d_in["v"], idx, g, permg, actg, nag, yq, ws=wsq,
                    stream=stream),
            }
            rec = {"group_size": gb}
            for name, fn in runs.items():
                for _ in range(2):
                    fn()
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                e0.record(stream)
                for _ in range(args.steps):
                    fn()
                e1.record(stream)
                torch.cuda.synchronize()
                rec[name + "_ms"] = e0.elapsed_time(e1) / args.steps
            rec["max_row_rel_diff"] = float(((yr - yq).abs().amax(dim=1) /
                                             yq.abs().amax(dim=1).clamp_min(1e-30)).max())
            rec["per_task_expert_stage_ms"] = dot_ms + per["accumulate"]
            group_rows.append(rec)
            log(f"group rows, B={gb}: {rec['group_rows_ms']:.3f} ms (grouped dot + slot-order sum "
                f"{rec['grouped_slot_order_sum_ms']:.3f} ms; per-task stage "
                f"{rec['per_task_expert_stage_ms']:.3f} ms)")
            del wsr, wsq, yr, yq, permg, actg, offg, nag

    # Backward of the expert compute (training): token pass, per-expert pass over the
    # schedule's segments, softmax pass; dy is a seeded standard normal.
    perm, off, na, n_active = sched
    backward = None
    if w.d <= (4096 if w.bf16 else 2048):
        gen = torch.Generator(device="cuda")
        gen.manual_seed(0)
        dy = torch.randn((w.T, w.d), generator=gen, device="cuda", dtype=torch.float32)
        dx = torch.empty_like(dy)
        du = torch.empty((max(1, n_active), w.d), dtype=torch.float32, device="cuda")
        dv = torch.empty_like(du)
        dgt = torch.empty_like(g)
        dsc = torch.empty_like(g)
        wsb = P.workspace(desc, 6)
        bw = lambda: P.omnimoe_expert_backward(  # noqa: E731
            desc, d_in["x"], d_in["u"], d_in["v"], idx, g, perm, off, na, dy, dx, du, dv, dgt,
            dsc, ws=wsb, stream=stream)
        bw()
        ev0.record(stream)
        for _ in range(args.steps):
            bw()
        ev1.record(stream)
        torch.cuda.synchronize()
        bw_ms = ev0.elapsed_time(ev1) / args.steps
        # router backward from the score gradients just computed (selections fixed)
        dkr = torch.empty((w.H, w.n_rows, w.d_key), dtype=torch.float32, device="cuda")
        dkc = torch.empty((w.H, w.n_cols, w.d_key), dtype=torch.float32, device="cuda")
        wsr = P.workspace(desc, 7)
        rb = lambda: P.omnimoe_route_backward(  # noqa: E731
            desc, d_in["x"], d_in["keys_row"], d_in["keys_col"], idx, dsc, dx, dkr, dkc,
            ws=wsr, stream=stream)
        rb()
        ev0.record(stream)
        for _ in range(args.steps):
            rb()
        ev1.record(stream)
        torch.cuda.synchronize()
        rb_ms = ev0.elapsed_time(ev1) / args.steps
        backward = {"expert_backward_ms": bw_ms, "route_backward_ms": rb_ms,
                    "active_rows": n_active,
                    "tokens_per_s": w.T / ((bw_ms + rb_ms) * 1e-3)}
        log(f"expert backward: {bw_ms:.3f} ms, router backward: {rb_ms:.3f} ms")
        del dy, dx, du, dv, wsb, dkr, dkc, wsr
    return ablation, shared_mlp, no_cpr, backward, grouped, contrib, group_rows


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="train_bf16")
    ap.add_argument("--cpu-sample", type=int, default=16384,
                    help="tokens for the oracle leg (16384: about 10 s on 16 host threads)")
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle leg")
    ap.add_argument("--single-thread-sample", type=int, default=256,
                    help="tokens for the oracle leg on one host thread (0: skip)")
    ap.add_argument("--brute-sample", type=int, default=256,
                    help="tokens for the oracle's brute-force selection timing (0: skip)")
    ap.add_argument("--out", default=None, help="also write the JSON line here")
    ap.add_argument("--graph", action="store_true",
                    help="time replays of one layer call captured in a HIP graph")
    ap.add_argument("--no-cold", action="store_true",
                    help="skip the second timing with the caches flushed before each step")
    ap.add_argument("--layer-only", action="store_true",
                    help="time the layer alone: no cold timing, shared branch or ablations (for "
                         "kernel traces and counters that should hold the layer's kernels only)")
    ap.add_argument("--group-size", type=int, default=0,
                    help="execution-group size B of the schedule (0: the workload's own); with "
                         "B > 1 the layer runs the grouped expert GEMM")
    ap.add_argument("--grouped-b", type=int, default=64,
                    help="group size of the grouped-GEMM comparison timed beside the layer "
                         "(0: skip)")
    ap.add_argument("--group-rows-b", default="",
                    help="comma-separated group sizes at which the second product of Eq. 14 per "
                         "group (partial rows) is timed against the slot-order sum")
    ap.add_argument("--copy-bytes", type=int, default=0,
                    help="after timing, run a plain device copy of this many bytes twice "
                         "(a known-size reference for rocprofv3 FETCH_SIZE / WRITE_SIZE)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: this layer runs on a single MI355X and has no "
              f"multi-GPU path (asked for --gpus {args.gpus}).", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import synth
    import paper_2602_05711_amd as P
    from paper_2602_05711_amd import binding as B

    w = synth.WORKLOADS[args.workload]
    if args.group_size > 0:
        w = w.with_(group_size=args.group_size)
    log(f"workload {w.name}: T={w.T} d={w.d} grid={w.n_rows}x{w.n_cols} d_key={w.d_key} "
        f"H={w.H} K={w.K} B={w.group_size} {w.dtype}")
    t0 = time.time()
    inp = synth.make_inputs(w)
    log(f"generated inputs in {time.time() - t0:.1f} s")

    def dev(a):
        if a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16)).cuda().view(torch.bfloat16)
        return torch.from_numpy(a).cuda()

    d_in = {k: dev(v) for k, v in inp.items()}
    torch.cuda.synchronize()
    log("inputs resident on the GPU")
    desc = P.make_desc(w)
    ws = P.workspace(desc, 4)
    y = torch.empty((w.T, w.d), dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()

    def step():
        P.omnimoe_layer_forward(desc, d_in["x"], d_in["keys_row"], d_in["keys_col"], d_in["u"],
                                d_in["v"], y, ws=ws, stream=stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log(f"warmup {args.warmup} done")
    if args.graph:
        # One layer call captured once (the library allocates nothing and never synchronises
        # inside a call), then replayed as the timed step.
        graph = torch.cuda.CUDAGraph()
        cap = torch.cuda.Stream()
        cap.wait_stream(stream)
        with torch.cuda.stream(cap):
            with torch.cuda.graph(graph, stream=cap):
                P.omnimoe_layer_forward(desc, d_in["x"], d_in["keys_row"], d_in["keys_col"],
                                        d_in["u"], d_in["v"], y, ws=ws, stream=cap)
        stream.wait_stream(cap)
        torch.cuda.synchronize()
        step = graph.replay  # noqa: F811
        for _ in range(args.warmup):
            step()
        torch.cuda.synchronize()
        log("captured the layer call in a graph")
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(args.steps):
        step()
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms_step = ev0.elapsed_time(ev1) / args.steps
    log(f"timed {args.steps} steps: {ms_step:.3f} ms/step (wall {1e3 * wall / args.steps:.3f})")

    # Cold steps: before each one a 512 MiB fill evicts the L2 and the MALL, so the step reads
    # its inputs (x, sub-keys, expert rows) from HBM; only the layer call sits between events.
    cold = None
    if not (args.no_cold or args.layer_only):
        flush = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(args.steps)]
        for e0, e1 in evs:
            flush.fill_(1)
            e0.record(stream)
            step()
            e1.record(stream)
        torch.cuda.synchronize()
        cold_ms = sorted(e0.elapsed_time(e1) for e0, e1 in evs)
        med = cold_ms[len(cold_ms) // 2]
        cold = {"ms_per_step_median": med, "tokens_per_s": w.T / (med * 1e-3),
                "flush_bytes": 512 << 20}
        del flush
        log(f"cold steps (512 MiB flush before each): median {med:.3f} ms")

    # Per-kernel durations: the same calls with HIP events around each kernel group.
    timer = P.Timer(args.steps)
    for _ in range(args.steps):
        timer.layer_forward(desc, d_in["x"], d_in["keys_row"], d_in["keys_col"], d_in["u"],
                            d_in["v"], y, ws, stream=stream)
    ms, n = timer.read()
    timer.close()
    per = {k: v / n for k, v in ms.items()}

    # Active experts of this batch, for the algorithmic byte counts.
    idx = torch.empty((w.T, w.H, w.K), dtype=torch.int32, device="cuda")
    g = torch.empty((w.T, w.H, w.K), dtype=torch.float32, device="cuda")
    P.omnimoe_route(desc, d_in["x"], d_in["keys_row"], d_in["keys_col"], idx, g)
    A = min(w.M, w.N)
    perm = torch.empty(w.M, dtype=torch.int32, device="cuda")
    act = torch.empty(A, dtype=torch.int32, device="cuda")
    off = torch.empty(A + 1, dtype=torch.int32, device="cuda")
    na = torch.zeros(1, dtype=torch.int32, device="cuda")
    # expert-major schedule (group size 1): the backward walks its per-expert segments
    P.omnimoe_schedule(P.make_desc(w.with_(group_size=1)), idx, perm, act, off, na)
    torch.cuda.synchronize()
    n_active = int(na.item())
    routing = routing_stats(idx.cpu().numpy(), w.N)
    assert routing["n_active"] == n_active

    ablation = shared_mlp = no_cpr = backward = grouped = contrib = group_rows = None
    if not args.layer_only:
        ablation, shared_mlp, no_cpr, backward, grouped, contrib, group_rows = extras(
            args, w, desc, d_in, dev, idx, g, y, stream, per, ms_step, ev0, ev1,
            (perm, off, na, n_active))

    work = algorithmic_work(w, n_active)
    path = P.omnimoe_layer_path(desc)
    # Kernel groups the layer does not launch for this shape: no schedule (slot-order dot), or
    # a dot formed by the selection kernel, whose time and bytes then count under "select".
    absent = {}
    if not path & (B.PATH_SCHEDULE | B.PATH_DENSE_DOT):
        absent["schedule"] = "not formed (slot-order dot)"
    if path & B.PATH_SELECT_DOT:
        absent["expert_dot"] = "formed by the selection kernel"
        work["select"] = ("hbm", work["select"][1] + work["expert_dot"][1])
    # Products dense over all experts (Eq. 14 with a single group) are MFMA GEMMs: priced by the
    # FLOP they perform, 2 T N d each (the expert dimension padded to the split width).
    dense_flop = 2.0 * w.T * w.N * w.d
    if path & B.PATH_DENSE_SUM:
        work["accumulate"] = ("mfma", dense_flop)
    if path & B.PATH_DENSE_DOT:
        work["expert_dot"] = ("mfma", dense_flop)
        # the selection-mask pass: idx and gates in; mask, prefix counts and sorted gates out
        work["schedule"] = ("hbm", 8.0 * w.M + 8.0 * w.T * ((w.N + 31) // 32) + 4.0 * w.M)
    kernels = {}
    for k, (bound, amount) in work.items():
        if k in absent:
            kernels[k] = {"absent": absent[k], "ms": per[k]}
            continue
        t_s = per[k] * 1e-3
        if bound == "hbm":
            ach = amount / t_s / 1e9
            kernels[k] = {"bound": "hbm", "ms": per[k], "achieved": ach, "unit": "GB/s",
                          "frac": ach / HBM_PEAK_GBS, "algorithmic_bytes": amount}
        else:
            peak = BF16_PEAK_TFLOPS if bound == "mfma" else FP32_PEAK_TFLOPS
            ach = amount / t_s / 1e12
            kernels[k] = {"bound": bound, "ms": per[k], "achieved": ach, "unit": "TFLOP/s",
                          "frac": ach / peak, "flop": amount}
    for k, kd in kernels.items():
        if "absent" in kd:
            continue
        tb = load_traffic(k, w.name)
        if tb is not None:
            # rocprofv3 bytes (L2 misses, MALL hits included) over the event-timed duration
            kd["counter_bytes"] = tb
            kd["counter_GBps"] = tb / (per[k] * 1e-3) / 1e9
        if kd["bound"] == "mfma":
            mb = load_mfma_busy(k, w.name)
            if mb is not None:
                kd["mfma_busy"] = mb
    dom = max((k for k in per if k not in absent), key=per.get)
    kd = kernels[dom]
    traffic = load_traffic(dom, w.name)
    roofline = {"kernel": dom, "bound": kd["bound"], "achieved": kd["achieved"],
                "peak": HBM_PEAK_GBS if kd["bound"] == "hbm" else (
                    BF16_PEAK_TFLOPS if kd["bound"] == "mfma" else FP32_PEAK_TFLOPS),
                "unit": kd["unit"], "frac": kd["frac"], "traffic": traffic,
                "ms_per_launch": per[dom]}
    log("per kernel: " + ", ".join(f"{k} {v:.3f} ms" for k, v in per.items()))

    if args.copy_bytes > 0:
        n = args.copy_bytes // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(2):
            dst.copy_(src)
        torch.cuda.synchronize()
        log(f"copied {n * 4} bytes twice")
        del src, dst

    cpu = None
    if not args.no_cpu:
        threads, hostinfo = host_threads()
        log(f"oracle leg: {args.cpu_sample} tokens on {threads} host threads ({hostinfo})")
        cpu = cpu_baseline(w, inp, args.cpu_sample, threads)
        cpu.update(hostinfo)
        log(f"oracle {cpu['value']:.1f} tokens/s")
        if args.single_thread_sample > 0:
            cpu["single_thread"] = cpu_baseline(w, inp, args.single_thread_sample, 1)
            log(f"oracle on one thread {cpu['single_thread']['value']:.1f} tokens/s")
        if args.brute_sample > 0:
            cpu["bruteforce_select"] = cpu_bruteforce(w, inp, args.brute_sample, threads)
            log(f"oracle brute-force selection {cpu['bruteforce_select']['value']:.1f} tokens/s")

    line = {
        "metric": METRIC, "value": w.T / (ms_step * 1e-3), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": w.dtype, "data": "synthetic",
        "config": {"workload": w.name, "T": w.T, "d": w.d, "n_rows": w.n_rows,
                   "n_cols": w.n_cols, "N": w.N, "d_key": w.d_key, "H": w.H, "K": w.K,
                   "act": w.act, "query": w.query_mode, "group_size": w.group_size,
                   "graph": bool(args.graph)},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "cold": cold,
        "shared_mlp": shared_mlp,
        "expert_backward": backward,
        "ablation_no_schedule": ablation,
        "ablation_no_cartesian_router": no_cpr,
        "grouped_expert_gemm": grouped,
        "group_rows_second_product": group_rows,
        "accumulate_contribution_rows": contrib,
        "n_active": n_active, "eta": w.M / max(1, n_active), "routing": routing,
        "schedule_share": per["schedule"] / sum(per.values()) if path & B.PATH_SCHEDULE else 0.0,
        "layer_path": {"schedule": bool(path & B.PATH_SCHEDULE),
                       "grouped": bool(path & B.PATH_GROUPED),
                       "select_forms_dot": bool(path & B.PATH_SELECT_DOT),
                       "dense_routed_sum": bool(path & B.PATH_DENSE_SUM),
                       "dense_expert_dot": bool(path & B.PATH_DENSE_DOT)},
        "kernels": kernels,
    }
    s = json.dumps(line)
    print(s, flush=True)
    if args.out:
        with open(args.out, "w") as f:
            f.write(s + "\n")


if __name__ == "__main__":
    main()
