#!/usr/bin/env python3
"""Calibrates the sub-key skew of the skewed-routing workload with the oracle router.

The workload has the training shape (16384 tokens, d=2048, 1024 x 1024 experts, H=8, K=16) and
should route about half of all (token, expert) pairs to the 10% most used experts. Sub-key row
i of each half is scaled by c_i = ((pi(i) + 1) / n)^(-alpha) (normalised to mean c^2 = 1; see
synth.skew_row_scale), and alpha is found by bisection on the top-10% share measured by routing
the full batch through the oracle (fp64 logits, Cartesian top-K). Writes skew_calibration.json
next to this file; synth.WORKLOADS["skew_bf16"] carries the resulting alpha.

Run: python tests/golden/calibrate_skew.py   (about ten oracle routings of the full batch)
"""
import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import oracle  # noqa: E402
import synth  # noqa: E402

TARGET, TOL = 0.50, 0.02


def route_stats(w, x):
    kr, kc = synth.make_keys(w)
    dsc = oracle.desc(w)
    sr, sc = oracle.half_scores(dsc, x, synth.as_f32(kr), synth.as_f32(kc))
    idx, _, _, _ = oracle.select(dsc, sr, sc, oracle.CARTESIAN)
    counts = np.bincount(idx.ravel(), minlength=w.N)
    top = np.sort(counts)[::-1]
    share = float(top[: w.N // 10].sum() / idx.size)
    return {"alpha": w.skew_alpha, "top10_share": share, "n_active": int((counts > 0).sum()),
            "max_segment": int(top[0]), "usage": float((counts > 0).mean())}


def main():
    base = synth.WORKLOADS["train_bf16"]
    x = synth.as_f32(synth.make_x(base))
    history = []
    lo, hi = 0.0, 2.0
    best = None
    for it in range(14):
        a = 0.5 * (lo + hi)
        t0 = time.time()
        st = route_stats(base.with_(name="skew_bf16", skew_alpha=a), x)
        st["seconds"] = round(time.time() - t0, 1)
        history.append(st)
        print(json.dumps(st), flush=True)
        if best is None or abs(st["top10_share"] - TARGET) < abs(best["top10_share"] - TARGET):
            best = st
        if abs(st["top10_share"] - TARGET) <= TOL / 4:
            break
        if st["top10_share"] < TARGET:
            lo = a
        else:
            hi = a
    uniform = route_stats(base, x)
    out = {"target_top10_share": TARGET, "tolerance": TOL, "chosen": best,
           "uniform_reference": uniform, "bisection": history}
    with open(os.path.join(HERE, "skew_calibration.json"), "w") as f:
        json.dump(out, f, indent=1)
    print("chosen alpha", best["alpha"], "share", best["top10_share"])


if __name__ == "__main__":
    main()
