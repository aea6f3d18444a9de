"""Throughput of the staged adaptive ViT pipeline on one MI355X.

A step is one fusion_run over the whole batch (patch embedding, 12 blocks
with merge / exit check / prune / compaction, final head) with the images
already resident in HBM.  Default workload: DeiT-S shape, batch 256, bf16,
224x224 images, router strength 1; the headline line is taken at the
0 %-early-exit threshold, and the 50 % and 90 % settings (thresholds from
the oracle calibration in tests/golden/exit_thresholds.json) are reported
alongside.  Prints one JSON line.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

BF16_PEAK = 2.5e15   # MI355X dense bf16 MFMA, FLOP/s
HBM_PEAK = 8.0e12    # MI355X HBM3E, B/s


def executed_flops(cfg, counts, exit_block):
    """Algorithmic FLOPs the batch executed (per sample: patch embedding,
    24 T d^2 + 4 T^2 d per block run (mlp = 4d), the heads evaluated)."""
    d, mlp, C, L = cfg["d"], cfg["mlp"], cfg["C"], cfg["L"]
    T = counts.astype(np.float64)
    per_block = 2 * T * d * 3 * d + 2 * T * d * d + 4 * T * d * mlp + 4 * T * T * d
    f = per_block.sum()
    f += counts.shape[0] * 2.0 * cfg["N0"] * cfg["patch_dim"] * d
    for b in cfg["exits"]:
        f += 2.0 * d * C * (counts[:, b - 1] > 0).sum()
    f += 2.0 * d * C * (exit_block == L).sum()
    return float(f)


def kernel_work(cfg, counts):
    """Algorithmic FLOPs (matrix kernels) or bytes (memory-bound kernels) of
    every launch kind over one step, from the token counts."""
    d, mlp, H = cfg["d"], cfg["mlp"], cfg["H"]
    T = counts.astype(np.float64)
    live = T > 0
    M = T.sum(axis=0)                       # rows per block
    ns = live.sum(axis=0)                   # live samples per block
    w = {
        "gemm_qkv": ("flop", float((2 * M * d * 3 * d).sum())),
        "gemm_proj": ("flop", float((2 * M * d * d).sum())),
        "gemm_fc1_gelu": ("flop", float((2 * M * d * mlp).sum())),
        "gemm_fc2": ("flop", float((2 * M * mlp * d).sum())),
        "attention": ("flop", float((4 * T * T * d).sum())),
        "patch_embed": ("flop", 2.0 * counts.shape[0] * cfg["N0"] * cfg["patch_dim"] * d),
        # LayerNorm kernel: read fp32 rows, write bf16 rows; LN2 of every
        # block and LN1 of block 1 (later LN1s are written by the compaction)
        "layernorm": ("byte", float((M * d * (4 + 2)).sum() + M[0] * d * (4 + 2))),
    }
    # adapt: read the sample's fp32 rows and sizes, write the merged rows
    # back; compaction after block b: read and write the rows kept for block
    # b + 1 (x, size, origin) and write their LN1 (bf16)
    w["adapt"] = ("byte", float((M * (d * 4 + 8) * 2).sum()))
    w["compact"] = ("byte", float((M[1:] * ((d * 4 + 8) * 2 + d * 2)).sum()))
    return w


def measured_traffic(kernel):
    """HBM bytes per launch of `kernel` from the committed counter summary
    (profiles/traffic.json), or None if it was taken on other kernel source."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    entry = t.get("kernels", {}).get(kernel)
    if not entry:
        return None
    src = os.path.join(ROOT, "paper_2607_02612_amd", "csrc", entry["source"])
    with open(src, "rb") as f:
        digest = hashlib.sha256(f.read()).hexdigest()
    if digest != entry["source_sha256"]:
        return None
    return entry["bytes_per_launch"]


def cpu_baseline(cfg, W, imgs, n):
    """The oracle on the first n images (bounded sample), images/s."""
    from oracle import fusion_oracle as fo
    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:
        cores = os.cpu_count() or 1
    Wp = fo.prepare_weights(W, "bf16emu")
    fo.run_sample(imgs[0], Wp, cfg, "bf16emu")          # warm-up image
    t0 = time.perf_counter()
    for i in range(n):
        fo.run_sample(imgs[i], Wp, cfg, "bf16emu")
    dt = time.perf_counter() - t0
    return {"value": n / dt, "unit": "images/s", "cores": int(cores),
            "kind": "oracle",
            "sample": f"first {n} of the {imgs.shape[0]} DeiT-S images, bf16emu "
                      f"mode, exits disabled, merge and prune at rho=1 "
                      f"({dt:.1f} s wall)"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="deit_s")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--cpu-images", type=int, default=48)
    ap.add_argument("--headline-only", action="store_true",
                    help="time only the 0 %% early-exit setting (for profiler runs)")
    ap.add_argument("--calib-copy", action="store_true",
                    help="also run one 256 MiB device-to-device copy, whose HBM "
                         "counters calibrate FETCH_SIZE / WRITE_SIZE")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported "
              "(the path shards by sample with no exchange: run one process per GPU).",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2607_02612_amd import FusionModel
    from synth import blob, configs, images, weights

    cfg = configs.get(args.workload)
    W = weights.make_weights(cfg)
    imgs = images.make_images(cfg)
    B = cfg["batch"]
    with open(os.path.join(ROOT, "tests", "golden", "exit_thresholds.json")) as f:
        cal = json.load(f)
    th = {0.0: 1.0}
    for wl in cal["workloads"]:
        if wl["workload"] == args.workload and wl["rho"] == 1.0:
            th = {float(k): v for k, v in wl["thresholds"].items()}
    model = FusionModel(blob.pack(cfg, W), B)
    x = torch.from_numpy(imgs).cuda()
    out = model.alloc_outputs(B)

    def timed(delta):
        model.set_exit_thresholds([delta] * len(cfg["exits"]))
        for _ in range(args.warmup):
            model.run(x, out=out)
        torch.cuda.synchronize()
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0 = time.perf_counter()
        s.record()
        for _ in range(args.steps):
            model.run(x, out=out)
        e.record()
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        ms = s.elapsed_time(e) / args.steps
        counts = out[2].cpu().numpy()
        eb = out[1].cpu().numpy()
        fl = executed_flops(cfg, counts, eb)
        return dict(ms=ms, wall_ms=1e3 * wall / args.steps, img_s=B / (ms / 1e3),
                    flops=fl, pct_peak=100.0 * fl / (ms / 1e3) / BF16_PEAK,
                    early_exit=float((eb < cfg["L"]).mean()),
                    mean_tokens=float(counts[counts > 0].mean()), counts=counts)

    if args.calib_copy:
        src = torch.empty(64 << 20, dtype=torch.float32, device="cuda").fill_(1.0)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    sweep = {}
    for e_rate in sorted(th):
        if args.headline_only and e_rate != 0.0:
            continue
        sweep[e_rate] = timed(th[e_rate])
    head = sweep[0.0]

    # per-kernel timing (HIP events around each launch, separate pass)
    model.set_exit_thresholds([th[0.0]] * len(cfg["exits"]))
    model.profile_enable(True)
    for _ in range(args.steps):
        model.run(x, out=out)
    torch.cuda.synchronize()
    prof = model.profile_read()
    model.profile_enable(False)
    work = kernel_work(cfg, head["counts"])
    kernels = {}
    for k, (ms_tot, n) in prof.items():
        if n == 0:
            continue
        entry = {"ms_per_step": ms_tot / args.steps, "launches_per_step": n / args.steps}
        if k in work:
            kind, amount = work[k]
            rate = amount / (ms_tot / args.steps / 1e3)
            if kind == "flop":
                entry["tflops"] = rate / 1e12
                entry["frac_bf16_peak"] = rate / BF16_PEAK
            else:
                entry["gbps"] = rate / 1e9
                entry["frac_hbm_peak"] = rate / HBM_PEAK
        kernels[k] = entry
    flop_kernels = {k: v for k, v in kernels.items() if "tflops" in v}
    dom = max(flop_kernels, key=lambda k: flop_kernels[k]["ms_per_step"])
    dk = kernels[dom]
    roofline = {"kernel": dom, "bound": "mfma", "achieved": dk["tflops"],
                "peak": BF16_PEAK / 1e12, "unit": "TFLOP/s",
                "frac": dk["frac_bf16_peak"], "traffic": measured_traffic(dom)}

    line = {
        "metric": "images/sec at DeiT-S b=256 bf16 (1 GPU); % bf16 MFMA peak on executed FLOPs",
        "value": head["img_s"], "unit": "images/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": head["ms"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"{args.workload} batch {B} {cfg['img']}x{cfg['img']} "
                               f"({cfg['N0'] + 1} tokens), merge r={cfg['r']} every "
                               f"block, exit heads {list(cfg['exits'])}, prune "
                               f"keep {cfg['tau']} at {list(cfg['prunes'])}, rho=1, "
                               f"0% early exit",
                   "batch": B, "image": cfg["img"], "tokens": cfg["N0"] + 1,
                   "d": cfg["d"], "heads": cfg["H"], "layers": cfg["L"]},
        "pct_bf16_peak_executed": head["pct_peak"],
        "executed_gflop_per_image": head["flops"] / B / 1e9,
        "exit_sweep": {f"{int(100 * e)}%": {"threshold": th[e], "images_per_s": r["img_s"],
                                             "ms_per_step": r["ms"],
                                             "pct_bf16_peak_executed": r["pct_peak"],
                                             "measured_early_exit": r["early_exit"],
                                             "executed_gflop_per_image": r["flops"] / B / 1e9}
                       for e, r in sweep.items()},
        "roofline": roofline,
        "kernels": kernels,
    }
    if not args.no_cpu:
        line["cpu_baseline"] = cpu_baseline(cfg, W, imgs, args.cpu_images)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
