"""Write noise_floor.json: how far the bf16 rounding contract lets two exact
implementations of the pipeline drift apart, measured with the CPU oracle
only.

For each workload, every sampled image runs through the oracle twice in
bf16emu mode: once with float32 (BLAS) accumulation of the matrix products
and once accumulating in float64 (rounded once to float32).  The second run
follows the first one's discrete decisions (any disagreement is adopted), so
both share one trajectory; the only difference is summation order.  The
maximum |logit difference|, |exit confidence difference| and (learned
prune scorer) |token score difference| over the sample
are the floors any other bf16 implementation (the GPU path included) must
be allowed; the parity tests use a multiple of them where it exceeds the
literal bounds (2e-2 for logits, 1e-3 for exit margins).

Usage:  python tests/golden/make_noise_floor.py [workload ...]
        (with names: recompute only those rows of the plan, keep the rest)
"""
from __future__ import annotations

import json
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import numpy as np  # noqa: E402

from oracle import fusion_oracle as fo  # noqa: E402
from synth import configs, images, weights  # noqa: E402

PLAN = [("deit_ti", 1.0, 64), ("deit_s", 1.0, 32), ("deit_b", 1.0, 12),
        ("deit_s_384", 0.5, 6), ("deit_s_384", 1.0, 6), ("deit_s_384", 1.5, 6),
        ("deit_s_paper", 1.0, 32)]


def floor(name, rho, n):
    cfg = configs.get(name)
    W = fo.prepare_weights(weights.make_weights(cfg), "bf16emu")
    imgs = images.make_images(cfg, batch=n)
    delta = [1.0] * len(cfg["exits"])
    dl, dc, ds = [], [], []
    for i in range(n):
        a = fo.run_sample(imgs[i], W, cfg, "bf16emu", delta=delta, rho=rho)
        f = {b: dict(r=tb.get("r", 0), merge=tb.get("merge", {}), exit=False,
                     ids=tb["ids"]) for b, tb in a["trace"].items()}
        with fo.accumulate("fp64"):
            b_ = fo.run_sample(imgs[i], W, cfg, "bf16emu", delta=delta, rho=rho,
                               follow=f, tol=1.0)
        dl.append(float(np.abs(a["logits"] - b_["logits"]).max()))
        dc.append(max(abs(a["trace"][e]["c"] - b_["trace"][e]["c"])
                      for e in cfg["exits"]))
        for p in cfg["prunes"]:
            if "scores" in a["trace"].get(p, {}):
                ds.append(float(np.abs(a["trace"][p]["scores"]
                                       - b_["trace"][p]["scores"]).max()))
    out = dict(workload=name, rho=rho, samples=n, max_dlogit=max(dl),
               median_dlogit=float(np.median(dl)), max_dc=max(dc),
               median_dc=float(np.median(dc)))
    if ds:
        out["max_dscore"] = max(ds)
    return out


def main():
    only = set(sys.argv[1:])
    path = os.path.join(HERE, "noise_floor.json")
    old = {}
    if only and os.path.exists(path):
        with open(path) as f:
            old = {(w["workload"], w["rho"]): w for w in json.load(f)["workloads"]}
    out = {"method": __doc__.split("Usage")[0].strip(), "workloads": []}
    for name, rho, n in PLAN:
        if only and name not in only and (name, rho) in old:
            out["workloads"].append(old[(name, rho)])
            continue
        t0 = time.time()
        r = floor(name, rho, n)
        out["workloads"].append(r)
        print(r, f"{time.time() - t0:.0f}s", flush=True)
    with open(path, "w") as f:
        json.dump(out, f, indent=1)


if __name__ == "__main__":
    main()
