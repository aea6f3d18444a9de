"""Write exit_thresholds.json: shared exit thresholds that make a target
fraction of a workload's batch exit early, computed with the CPU oracle only.

Reading (the workload asks for thresholds at confidence percentiles chosen
so that 0 %, 50 % and 90 % of samples exit early): run the oracle with both
exit heads disabled, take c_hat_i = max over exit heads of the sample's exit
confidence (with a shared threshold delta, sample i exits early iff
c_hat_i >= delta, because its trajectory up to the exit is the same), sort
c_hat descending, and for target fraction e put delta midway between the
n-th and (n+1)-th values, n = round(e B); e = 0 gives delta = 1 (disabled).

Usage:  python tests/golden/make_exit_thresholds.py  [--quick]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import numpy as np  # noqa: E402

import oracle  # noqa: E402
from synth import configs, images, weights  # noqa: E402

PLAN = [("deit_s", 1.0, (0.0, 0.5, 0.9)),
        ("deit_s_384", 0.5, (0.5,)),
        ("deit_s_384", 1.0, (0.5,)),
        ("deit_s_384", 1.5, (0.5,))]


def thresholds(c_hat: np.ndarray, fractions):
    srt = np.sort(c_hat)[::-1]
    B = len(srt)
    out = {}
    for e in fractions:
        n = int(round(e * B))
        if n == 0:
            out[str(e)] = 1.0
        elif n >= B:
            out[str(e)] = float(srt[-1]) / 2
        else:
            out[str(e)] = float((np.float64(srt[n - 1]) + np.float64(srt[n])) / 2)
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--out", default=os.path.join(HERE, "exit_thresholds.json"))
    args = ap.parse_args()
    result = {"method": __doc__.split("Usage")[0].strip(), "workloads": []}
    for name, rho, fracs in PLAN:
        cfg = configs.get(name)
        W = weights.make_weights(cfg)
        imgs = images.make_images(cfg)
        t0 = time.time()
        _, eb, _, res = oracle.run(imgs, W, cfg, "bf16emu",
                                   delta=[1.0] * len(cfg["exits"]), rho=rho)
        c_hat = np.array([max(r["trace"][b]["c"] for b in cfg["exits"]) for r in res])
        th = thresholds(c_hat, fracs)
        result["workloads"].append(dict(workload=name, rho=rho, batch=cfg["batch"],
                                        thresholds=th,
                                        c_hat_sorted=[float(v) for v in np.sort(c_hat)[::-1]]))
        print(name, rho, th, f"{time.time() - t0:.1f}s", flush=True)
    with open(args.out, "w") as f:
        json.dump(result, f, indent=1)


if __name__ == "__main__":
    main()
