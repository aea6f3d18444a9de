"""Write noise_floor.json: how far the bf16 rounding contract lets two exact
implementations of the pipeline drift apart, measured with the CPU oracle
only.

For each workload, every sampled image runs through the oracle twice in
bf16emu mode: once with float32 (BLAS) accumulation of the matrix products
and the exact-erf GELU, and once accumulating in float64 (rounded once to
float32) with GELU evaluated by the rational approximation 7.1.28 of
Abramowitz & Stegun (|erfc error| <= 3e-7, the form the GPU path uses).
The second run follows the first one's discrete decisions (any
disagreement is adopted), so both share one trajectory; the only
differences are summation order and the GELU approximation.  The maximum
|logit difference|, |exit confidence difference|, |router count-expression
difference| (2 rho m r_b, or rho m N / 2, in count units) and |token score
difference| before a prune (in the prune margin's units: N x probability
for CLS-attention scores, score units for the learned scorer) over the
sample are the floors any
other bf16 implementation (the GPU path included) must be allowed; the
parity tests use a multiple of them where it exceeds the literal bounds
(2e-2 for logits, 1e-3 for exit, router and prune margins).

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

# every sample of every batch the GPU parity tests compare
PLAN = [("deit_ti", 1.0, 64), ("deit_ti", 1.5, 64), ("deit_s", 1.0, 256),
        ("deit_b", 1.0, 256), ("deit_s_384", 0.5, 64), ("deit_s_384", 1.0, 64),
        ("deit_s_384", 1.5, 64), ("deit_s_paper", 1.0, 256),
        ("deit_s_paper", 5.0 / 3.0, 256)]


def gelu_as7128(x):
    """GELU(v) = max(v, 0) - |v| Q(|v|), Q(a) = erfc(a / sqrt 2) / 2 with
    erfc(z) = (1 + a1 z + ... + a6 z^6)^-16 (Abramowitz & Stegun 7.1.28),
    evaluated in float64 and rounded to float32."""
    a = np.abs(np.asarray(x, dtype=np.float64))
    z = a / np.sqrt(2.0)
    c = (0.0705230784, 0.0422820123, 0.0092705272, 0.0001520143, 0.0002765672,
         0.0000430638)
    p = 1.0 + z * (c[0] + z * (c[1] + z * (c[2] + z * (c[3] + z * (c[4] + z * c[5])))))
    q = 0.5 * p ** -16.0
    return (np.maximum(np.asarray(x, np.float64), 0.0) - a * q).astype(np.float32)


class gelu_approx:
    """Context manager: the oracle's GELU replaced by gelu_as7128."""

    def __enter__(self):
        self.prev, fo.gelu = fo.gelu, gelu_as7128

    def __exit__(self, *exc):
        fo.gelu = self.prev


def count_expression_drift(cfg, rho, ta, tb):
    """|change of the merge-count expression| between two runs' router
    outputs m, in count units (slope 2 rho r_b, or rho N / 2)."""
    out = []
    for b in cfg["merges"]:
        if b in ta and b in tb and "m" in ta[b]:
            dm = abs(ta[b]["m"] - tb[b]["m"])
            if cfg.get("merge_rule", "budget") == "fraction":
                slope = 0.5 * rho * (ta[b]["T"] - 1)
            else:
                slope = 2.0 * rho * cfg["r_b"][b - 1]
            out.append(slope * dm)
    return out


_CTX = {}


def _one(args):
    """Both runs of sample i; returns its drifts (worker process)."""
    name, rho, n, i = args
    key = (name, n)
    if key not in _CTX:
        cfg = configs.get(name)
        W = fo.prepare_weights(weights.make_weights(cfg), "bf16emu")
        _CTX[key] = (cfg, W, images.make_images(cfg, batch=n))
    cfg, W, imgs = _CTX[key]
    delta = [1.0] * len(cfg["exits"])
    a = fo.run_sample(imgs[i], W, cfg, "bf16emu", delta=delta, rho=rho)
    f = {b: dict(r=tb.get("r", 0), merge=tb.get("merge", {}), exit=False,
                 ids=tb["ids"]) for b, tb in a["trace"].items()}
    with fo.accumulate("fp64"), gelu_approx():
        b_ = fo.run_sample(imgs[i], W, cfg, "bf16emu", delta=delta, rho=rho,
                           follow=f, tol=1.0)
    # token-score drift in the prune margin's units: score units for the
    # learned scorer, N x probability for CLS-attention scores
    ds = [float(a["trace"][p]["score_unit"]
                * np.abs(a["trace"][p]["scores"] - b_["trace"][p]["scores"]).max())
          for p in cfg["prunes"] if "scores" in a["trace"].get(p, {})]
    return (float(np.abs(a["logits"] - b_["logits"]).max()),
            max(abs(a["trace"][e]["c"] - b_["trace"][e]["c"]) for e in cfg["exits"]),
            ds, count_expression_drift(cfg, rho, a["trace"], b_["trace"]))


def floor(name, rho, n, pool):
    rows = pool.map(_one, [(name, rho, n, i) for i in range(n)], chunksize=4)
    dl = [r[0] for r in rows]
    dc = [r[1] for r in rows]
    ds = [v for r in rows for v in r[2]]
    dt = [v for r in rows for v in r[3]]
    out = dict(workload=name, rho=rho, samples=n, max_dlogit=max(dl),
               median_dlogit=float(np.median(dl)), max_dc=max(dc),
               median_dc=float(np.median(dc)))
    if ds:
        out["max_dscore"] = max(ds)
    if dt:
        out["max_dcount"] = max(dt)
        out["median_dcount"] = float(np.median(dt))
    return out


def main():
    only = set(sys.argv[1:])
    path = os.path.join(HERE, "noise_floor.json")
    old = {}
    if only and os.path.exists(path):
        with open(path) as f:
            old = {(w["workload"], w["rho"]): w for w in json.load(f)["workloads"]}
    out = {"method": __doc__.split("Usage")[0].strip(), "workloads": []}
    import multiprocessing as mp
    with mp.get_context("fork").Pool(max(1, (os.cpu_count() or 2) - 1)) as pool:
        for name, rho, n in PLAN:
            if only and name not in only and (name, rho) in old:
                out["workloads"].append(old[(name, rho)])
                continue
            t0 = time.time()
            r = floor(name, rho, n, pool)
            out["workloads"].append(r)
            print(r, f"{time.time() - t0:.0f}s", flush=True)
    with open(path, "w") as f:
        json.dump(out, f, indent=1)


if __name__ == "__main__":
    main()
