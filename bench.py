"""Throughput of the staged adaptive ViT pipeline on one MI355X.

A step is one fusion_run over the whole batch (patch embedding, 12 blocks
with merge / exit check / prune / compaction, final head) with the images
already resident in HBM.  Default workload: DeiT-S shape, batch 256, bf16,
224x224 images, router strength 1; the headline line is taken at the
0 %-early-exit threshold, and the 50 % and 90 % settings (thresholds from
the oracle calibration in tests/golden/exit_thresholds.json) are reported
alongside.  The K timed steps are kernel-by-kernel launches on one stream
(--graph: replays of the step captured as one HIP graph after the warm-up
steps); the headline setting is also timed in the other launch mode and
reported under "timing", with an event between consecutive steps for the
median and 10th / 90th percentile step times.

Also reported (same JSON line):
  paper     the Tab. I instantiation (DeiT-S, M = {3,5,7}, E = {8,10} with
            MLP heads, P = {9,10} with the learned scorer) under the
            balanced and power_save profiles and with adaptation off (plain
            DeiT-S on the same weights): images/s, exit rates, executed
            GFLOP/image and the reduction against dense DeiT-S, energy per
            image from the GPU's energy counter and 100 Hz power samples;
  ablation  single-mechanism and composed layer sets on one set of weights
            (Tab. VII): executed-FLOPs reduction and images/s;
  batch_sweep  images/s and ms/step against batch size for the profiles.
Prints one JSON line.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu]
                       [--no-paper] [--headline-only] [--graph]
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


def head_flops(cfg, b):
    """Matrix FLOPs of exit head b: 2 d C (linear) or 2 d h + 2 h C (MLP)."""
    d, C = cfg["d"], cfg["C"]
    kind = cfg["exit_kind"][cfg["exits"].index(b)]
    if kind == "linear":
        return 2.0 * d * C
    h = cfg["exit_hidden"]
    return 2.0 * d * h + 2.0 * h * C


def executed_flops(cfg, counts, exit_block):
    """Algorithmic FLOPs the batch executed (per sample: patch embedding,
    2 T d (3d + d + 2 mlp) + 4 T^2 d per block run, the heads evaluated)."""
    d, mlp, C, L = cfg["d"], cfg["mlp"], cfg["C"], cfg["L"]
    T = counts.astype(np.float64)
    per_block = 2 * T * d * 3 * d + 2 * T * d * d + 4 * T * d * mlp + 4 * T * T * d
    f = per_block.sum()
    f += counts.shape[0] * 2.0 * cfg["N0"] * cfg["patch_dim"] * d
    for b in cfg["exits"]:
        f += head_flops(cfg, b) * (counts[:, b - 1] > 0).sum()
    f += 2.0 * d * C * (exit_block == L).sum()
    return float(f)


def dense_flops(cfg):
    """FLOPs of the plain backbone on one image (no exit heads, no token
    reduction): the baseline of the FLOPs-reduction figures."""
    d, mlp, C, L, T = cfg["d"], cfg["mlp"], cfg["C"], cfg["L"], cfg["N0"] + 1
    blk = 2 * T * d * 3 * d + 2 * T * d * d + 4 * T * d * mlp + 4 * T * T * d
    return float(L * blk + 2 * cfg["N0"] * cfg["patch_dim"] * d + 2 * d * C)


def kernel_work(cfg, counts):
    """Algorithmic FLOPs and bytes of every launch kind over one step, from
    the token counts: each operand read once, each output written once (the
    fp32 residual stream read and written by the residual GEMMs).  Returns
    {kind: {"flop": F, "byte": B, "launches": n}}."""
    d, mlp, H = cfg["d"], cfg["mlp"], cfg["H"]
    T = counts.astype(np.float64)
    live = T > 0
    M = T.sum(axis=0)                       # rows per block
    nb = float((M > 0).sum())               # blocks run (one launch each)
    B, N0, pd = counts.shape[0], cfg["N0"], cfg["patch_dim"]
    w = {
        "gemm_qkv": {"flop": float((2 * M * d * 3 * d).sum()),
                     "byte": float((M * d * 2 + M * 3 * d * 2).sum() + nb * 3 * d * d * 2)},
        "gemm_proj": {"flop": float((2 * M * d * d).sum()),
                      "byte": float((M * d * 2 + M * d * 8).sum() + nb * d * d * 2)},
        "gemm_fc1_gelu": {"flop": float((2 * M * d * mlp).sum()),
                          "byte": float((M * d * 2 + M * mlp * 2).sum() + nb * mlp * d * 2)},
        "gemm_fc2": {"flop": float((2 * M * mlp * d).sum()),
                     "byte": float((M * mlp * 2 + M * d * 8).sum() + nb * d * mlp * 2)},
        # q, k, v read once (bf16), the output written once (bf16)
        "attention": {"flop": float((4 * T * T * d).sum()),
                      "byte": float((T * 3 * d * 2 + T * d * 2).sum())},
        "patch_embed": {"flop": 2.0 * B * N0 * pd * d,
                        "byte": B * N0 * (pd * 4 + pd * 2 + pd * 2 + d * 4) + d * pd * 2.0},
        # LayerNorm kernel: read fp32 rows, write bf16 rows; LN2 of every
        # block and LN1 of block 1 (later LN1s are written by the compaction)
        "layernorm": {"flop": 0.0, "byte": float((M * d * (4 + 2)).sum() + M[0] * d * (4 + 2))},
        # adapt: read the sample's fp32 rows and sizes, write the merged rows
        # back; compaction after block b: read the rows kept for block b + 1
        # (fp32 row, row id, size, origin), write their LN1 (bf16) and their
        # row id, size and origin (the fp32 rows themselves stay in place)
        "adapt": {"flop": 0.0, "byte": float((M * (d * 4 + 8) * 2).sum())},
        "compact": {"flop": 0.0, "byte": float((M[1:] * ((d * 4 + 12) + (d * 2 + 12))).sum())},
    }
    return w


def roofline_bound(work):
    """The roofline resource of a launch kind: "mfma" when its FLOPs take
    longer at the dense bf16 peak than its bytes at the HBM peak, else
    "hbm"."""
    return "mfma" if work["flop"] / BF16_PEAK >= work["byte"] / HBM_PEAK else "hbm"


def measured_traffic(kernel, workload):
    """HBM bytes per launch of `kernel` on `workload` from the committed
    counter summary (profiles/traffic.json, one entry per workload), or None
    if none was taken there or it was taken on other kernel source."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    entry = t.get("workloads", {}).get(workload, {}).get("kernels", {}).get(kernel)
    if not entry:
        return None
    src = os.path.join(ROOT, "paper_2607_02612_amd", "csrc", entry["source"])
    with open(src, "rb") as f:
        digest = hashlib.sha256(f.read()).hexdigest()
    if digest != entry["source_sha256"]:
        return None
    return entry["bytes_per_launch"]


def measured_peaks(torch):
    """What the box itself reaches, beside the vendor peaks: HBM as a 1 GiB
    device-to-device copy (bytes read + written over the copy time), MFMA as
    a 8192^3 bf16 GEMM through torch (the vendor library), best of 20."""
    src = torch.empty(256 << 20, dtype=torch.float32, device="cuda").fill_(1.0)
    dst = torch.empty_like(src)
    a = torch.randn(8192, 8192, device="cuda").to(torch.bfloat16)
    b = torch.randn(8192, 8192, device="cuda").to(torch.bfloat16)
    c = torch.empty(8192, 8192, device="cuda", dtype=torch.bfloat16)

    def best(fn, reps=20):
        for _ in range(3):
            fn()
        t = []
        for _ in range(reps):
            s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            s.record()
            fn()
            e.record()
            e.synchronize()
            t.append(s.elapsed_time(e) / 1e3)
        return min(t)

    t_copy = best(lambda: dst.copy_(src))
    t_mm = best(lambda: torch.matmul(a, b, out=c))
    del src, dst, a, b, c
    return {"hbm_copy_gbps": 2 * (1 << 30) / t_copy / 1e9,
            "bf16_gemm_tflops": 2 * 8192 ** 3 / t_mm / 1e12,
            "method": "1 GiB device copy; 8192^3 bf16 torch.matmul; best of 20"}


def cpu_baseline(cfg, W, imgs, n):
    """The oracle on the first n images (bounded sample), images/s."""
    from oracle import fusion_oracle as fo
    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:
        cores = os.cpu_count() or 1
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            model = next(l.split(":", 1)[1].strip() for l in f if l.startswith("model name"))
    except (OSError, StopIteration):
        pass

    def rate(mode, k):
        Wp = fo.prepare_weights(W, mode)
        fo.run_sample(imgs[0], Wp, cfg, mode)          # warm-up image
        t0 = time.perf_counter()
        for i in range(k):
            fo.run_sample(imgs[i], Wp, cfg, mode)
        return k / (time.perf_counter() - t0), time.perf_counter() - t0

    v, dt = rate("bf16emu", n)
    n32 = max(1, n // 4)
    v32, dt32 = rate("fp32", n32)
    return {"value": v, "unit": "images/s", "cores": int(cores),
            "kind": "oracle",
            "sample": f"first {n} of the {imgs.shape[0]} DeiT-S images, bf16emu "
                      f"mode, exits disabled, merge and prune at rho=1 "
                      f"({dt:.1f} s wall)",
            "fp32_mode": {"value": v32, "unit": "images/s",
                          "sample": f"first {n32} images, fp32 mode ({dt32:.1f} s wall)"},
            "host": {"cpu_model": model, "os_cpu_count": os.cpu_count()}}


class EnergyMeter:
    """GPU energy over a region, two ways: the difference of the device's
    energy accumulator, and power samples at 100 Hz (current socket power)
    integrated with the trapezoid rule, the sampling protocol of NVML-based
    measurements.  Reads only; the device is matched to torch's device 0 by
    PCI bus id.  ``error`` says why a reading is missing."""

    def __init__(self):
        self.ok, self.error, self.h = False, None, None
        try:
            import amdsmi
            import torch
            self.smi = amdsmi
            amdsmi.amdsmi_init()
            prop = torch.cuda.get_device_properties(0)
            want = (int(prop.pci_domain_id), int(prop.pci_bus_id), int(prop.pci_device_id))
            for h in amdsmi.amdsmi_get_processor_handles():
                bdf = amdsmi.amdsmi_get_gpu_device_bdf(h)      # dddd:bb:dd.f
                dom, bus, rest = bdf.split(":")
                dev = rest.split(".")[0]
                if (int(dom, 16), int(bus, 16), int(dev, 16)) == want:
                    self.h = h
            if self.h is None:
                self.error = f"no amd-smi device with PCI id {want}"
            else:
                self.ok = True
        except Exception as e:  # measurement is optional
            self.error = f"{type(e).__name__}: {e}"

    def _acc(self):
        e = self.smi.amdsmi_get_energy_count(self.h)
        return e["energy_accumulator"] * e["counter_resolution"] * 1e-6  # J

    def _power(self):
        p = self.smi.amdsmi_get_power_info(self.h)
        v = p.get("current_socket_power")
        if not isinstance(v, (int, float)):
            v = p.get("average_socket_power")
        return float(v) if isinstance(v, (int, float)) else None

    def measure(self, fn):
        """Run fn() (which synchronises the GPU) and return the energy."""
        import threading
        if not self.ok:
            return {"error": self.error}
        samples, stop = [], threading.Event()

        def sampler():
            while not stop.is_set():
                try:
                    w = self._power()
                except Exception:
                    w = None
                if w is not None:
                    samples.append((time.perf_counter(), w))
                stop.wait(0.01)

        th = threading.Thread(target=sampler, daemon=True)
        try:
            a0 = self._acc()
        except Exception as e:
            a0, self.error = None, f"energy counter: {e}"
        th.start()
        t0 = time.perf_counter()
        fn()
        t1 = time.perf_counter()
        stop.set()
        th.join()
        out = {"seconds": t1 - t0, "power_samples": len(samples)}
        if a0 is not None:
            out["joules_counter"] = self._acc() - a0
        if len(samples) >= 2:
            j = 0.0
            for (ta, wa), (tb, wb) in zip(samples, samples[1:]):
                j += 0.5 * (wa + wb) * (tb - ta)
            out["joules_sampled"] = j * (t1 - t0) / (samples[-1][0] - samples[0][0])
            out["mean_power_w"] = float(np.mean([w for _, w in samples]))
        return out


def progress(msg):
    """A progress line on stderr (the JSON line alone goes to stdout)."""
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def run_timed(model, x, out, steps, warmup, delta=None, rho=None):
    """Warm up, then time `steps` runs on the current stream with HIP events;
    returns ms per step and the last run's outputs (host)."""
    import torch
    if delta is not None:
        model.set_exit_thresholds(list(delta))
    if rho is not None:
        model.set_router_strength(rho)
    for _ in range(warmup):
        model.run(x, out=out)
    torch.cuda.synchronize()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s.record()
    for _ in range(steps):
        model.run(x, out=out)
    e.record()
    torch.cuda.synchronize()
    return s.elapsed_time(e) / steps, out[1].cpu().numpy(), out[2].cpu().numpy()


def summarize(cfg, B, ms, eb, counts):
    fl = executed_flops(cfg, counts, eb)
    exits = {str(b): float((eb == b).mean()) for b in cfg["exits"]}
    return {"images_per_s": B / (ms / 1e3), "ms_per_step": ms,
            "exit_rate": exits, "executed_gflop_per_image": fl / B / 1e9,
            "flops_reduction_vs_dense": 1.0 - fl / B / dense_flops(cfg),
            "pct_bf16_peak_executed": 100.0 * fl / (ms / 1e3) / BF16_PEAK,
            "mean_tokens_per_block": float(counts[counts > 0].mean())}


def paper_section(args, energy):
    """Tab. I instantiation under its profiles; plain DeiT-S (the backbone
    alone, same weights) as the baseline; the adaptive model with every
    mechanism inert (delta = 1, rho = 0) shows the cost of the machinery."""
    import torch
    from paper_2607_02612_amd import FusionModel
    from synth import blob, configs, images, weights
    cfg = configs.get("deit_s_paper")
    cfg_plain = configs.get("deit_s_paper", merges=(), exits=(), prunes=(),
                            exit_kind=(), delta=())
    W = weights.make_weights(cfg)
    imgs = images.make_images(cfg)
    B = cfg["batch"]
    models = {"adaptive": FusionModel(blob.pack(cfg, W), B),
              "plain": FusionModel(blob.pack(cfg_plain, W), B)}
    x = torch.from_numpy(imgs).cuda()
    settings = {name: dict(configs.profile_settings(name), model="adaptive")
                for name in configs.PROFILES}
    settings["adaptive_inert"] = dict(delta=(1.0, 1.0), rho=0.0, model="adaptive")
    settings["plain"] = dict(delta=None, rho=None, model="plain")
    cfg_of = {"adaptive": cfg, "plain": cfg_plain}

    def go(name, xb, steps, warmup):
        st = settings[name]
        mdl = models[st["model"]]
        ob = mdl.alloc_outputs(xb.shape[0])
        return run_timed(mdl, xb, ob, steps, warmup, st["delta"], st["rho"])

    res = {}
    for name, st in settings.items():
        ms, eb, cnt = go(name, x, args.steps, args.warmup)
        r = summarize(cfg_of[st["model"]], B, ms, eb, cnt)
        r.update(delta=None if st["delta"] is None else list(st["delta"]), rho=st["rho"])
        res[name] = r
        progress(f"paper setting {name}: {r['images_per_s']:.0f} images/s")
    for name in res:
        res[name]["speedup_vs_plain"] = res["plain"]["ms_per_step"] / res[name]["ms_per_step"]
    # energy: regions of about args.energy_seconds per setting, the settings
    # interleaved and the round repeated args.energy_reps times, so that
    # drifts of the board's power management fall on every setting alike;
    # mean and spread (min, max) per setting
    e_names = ["plain", "balanced", "power_save"]
    regions = {name: [] for name in e_names}
    for rep in range(args.energy_reps):
        for name in e_names:
            st = settings[name]
            mdl = models[st["model"]]
            ob = mdl.alloc_outputs(B)
            if st["delta"] is not None:
                mdl.set_exit_thresholds(list(st["delta"]))
            if st["rho"] is not None:
                mdl.set_router_strength(st["rho"])
            n = max(1, int(1e3 * args.energy_seconds / res[name]["ms_per_step"]))

            def loop():
                for _ in range(n):
                    mdl.run(x, out=ob)
                torch.cuda.synchronize()
            e = energy.measure(loop)
            if "joules_counter" in e:
                e["mj_per_image_counter"] = 1e3 * e["joules_counter"] / (n * B)
            if "joules_sampled" in e:
                e["mj_per_image_sampled"] = 1e3 * e["joules_sampled"] / (n * B)
            e["images"] = n * B
            e["images_per_s_in_region"] = n * B / e["seconds"] if "seconds" in e else None
            regions[name].append(e)
            progress(f"energy region {rep + 1}/{args.energy_reps} {name}: "
                     f"{e.get('mj_per_image_counter', float('nan')):.2f} mJ/image")
    for name in e_names:
        rs = regions[name]
        summ = {"regions": rs, "seconds_per_region": args.energy_seconds}
        for key in ("mj_per_image_counter", "mj_per_image_sampled", "images_per_s_in_region",
                    "mean_power_w"):
            v = [r[key] for r in rs if isinstance(r.get(key), (int, float))]
            if v:
                summ[key] = {"mean": float(np.mean(v)), "min": float(np.min(v)),
                             "max": float(np.max(v))}
        res[name]["energy"] = summ
    # a difference in energy per image is claimed only where the ranges of
    # the repeated regions do not overlap
    cmp = {}
    base = res["plain"]["energy"].get("mj_per_image_counter")
    for name in ("balanced", "power_save"):
        v = res[name]["energy"].get("mj_per_image_counter")
        if base and v:
            separated = v["max"] < base["min"] or v["min"] > base["max"]
            cmp[name] = {"saving_vs_plain": 1.0 - v["mean"] / base["mean"],
                         "ranges_separated": bool(separated)}
    energy_summary = {"method": "GPU energy accumulator (amd-smi) over each region; "
                                "settings interleaved, repeated; mean (min, max)",
                      "vs_plain": cmp}
    # batch sweep (Fig. 6 protocol: throughput and latency against batch)
    sweep = {}
    for b in (1, 8, 32, 64, 128, 256):
        xb = x[:b].contiguous()
        row = {}
        for name in settings:
            ms, _, _ = go(name, xb, max(10, args.steps // 2), 3)
            row[name] = {"images_per_s": b / (ms / 1e3), "ms_per_step": ms}
        for name in row:
            row[name]["speedup_vs_plain"] = row["plain"]["ms_per_step"] / row[name]["ms_per_step"]
        sweep[str(b)] = row
        progress(f"batch sweep {b} done")
    for mdl in models.values():
        mdl.close()
    return {"energy": energy_summary,
            "workload": f"deit_s_paper batch {B}: merge (fraction rule) at "
                        f"{list(cfg['merges'])}, exit heads {list(cfg['exits'])} "
                        f"({', '.join(cfg['exit_kind'])}, hidden {cfg['exit_hidden']}), "
                        f"learned prune keep {cfg['tau']} at {list(cfg['prunes'])}",
            "dense_gflop_per_image": dense_flops(cfg) / 1e9,
            "profiles": res, "batch_sweep": sweep}


def ablation_section(args):
    """Tab. VII layer-set variants on one set of weights (a superset draw:
    every tensor any variant reads)."""
    import torch
    from paper_2607_02612_amd import FusionModel
    from synth import blob, configs, images, weights
    sup = configs.get("deit_s_paper", prunes=configs.ABLATION_SUPERSET_PRUNES)
    W = weights.make_weights(sup)
    imgs = images.make_images(sup)
    B = sup["batch"]
    x = torch.from_numpy(imgs).cuda()
    rows = {}
    for name, over, prof in configs.ABLATION:
        cfg = configs.ablation_config("deit_s_paper", over)
        if cfg["merge_rule"] == "budget":
            Wc = weights.zero_routers(cfg, W)       # m = 1/2: r = r_b
        else:
            Wc = W
        st = configs.profile_settings(prof)
        delta = st["delta"][:len(cfg["exits"])]
        model = FusionModel(blob.pack(cfg, Wc), B)
        out = model.alloc_outputs(B)
        ms, eb, cnt = run_timed(model, x, out, args.steps, args.warmup,
                                delta if cfg["exits"] else None, st["rho"])
        r = summarize(cfg, B, ms, eb, cnt)
        r.update(merges=list(cfg["merges"]), exits=list(cfg["exits"]),
                 prunes=list(cfg["prunes"]), merge_rule=cfg["merge_rule"],
                 delta=list(delta), rho=st["rho"])
        rows[name] = r
        model.close()
    base = rows["plain"]["ms_per_step"]
    for r in rows.values():
        r["speedup_vs_plain"] = base / r["ms_per_step"]
    return rows


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="deit_s")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--cpu-images", type=int, default=256)
    ap.add_argument("--headline-only", action="store_true",
                    help="time only the 0 %% early-exit setting (for profiler runs)")
    ap.add_argument("--no-paper", action="store_true",
                    help="skip the Tab. I / Tab. VII / batch-sweep sections")
    ap.add_argument("--graph", action="store_true",
                    help="headline from replays of the step captured as one HIP "
                         "graph (default: kernel-by-kernel launches; the other "
                         "mode is timed too and reported under 'timing')")
    ap.add_argument("--energy-seconds", type=float, default=10.0,
                    help="length of each energy region (the paper section)")
    ap.add_argument("--energy-reps", type=int, default=3,
                    help="interleaved repetitions of the energy regions")
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
    th.setdefault(0.0, 1.0)  # delta = 1: no exit (the 0 % setting where none is calibrated)
    model = FusionModel(blob.pack(cfg, W), B)
    x = torch.from_numpy(imgs).cuda()
    out = model.alloc_outputs(B)

    def timed(delta, graph):
        # the thresholds are kernel arguments: set them, then capture the step
        model.set_exit_thresholds([delta] * len(cfg["exits"]))
        for _ in range(args.warmup):
            model.run(x, out=out)
        torch.cuda.synchronize()
        step = lambda: model.run(x, out=out)
        if graph:
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(graph):
                model.run(x, out=out)
            step = graph.replay
            step()
            torch.cuda.synchronize()
        # one event between consecutive steps: the mean over the K steps is
        # the first-to-last interval / K, and the per-step intervals give the
        # median and the 10th / 90th percentiles
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
        t0 = time.perf_counter()
        ev[0].record()
        for i in range(args.steps):
            step()
            ev[i + 1].record()
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        ms = ev[0].elapsed_time(ev[-1]) / args.steps
        per = np.array([ev[i].elapsed_time(ev[i + 1]) for i in range(args.steps)])
        counts = out[2].cpu().numpy()
        eb = out[1].cpu().numpy()
        fl = executed_flops(cfg, counts, eb)
        return dict(ms=ms, wall_ms=1e3 * wall / args.steps, img_s=B / (ms / 1e3),
                    step_ms={"median": float(np.median(per)),
                             "p10": float(np.percentile(per, 10)),
                             "p90": float(np.percentile(per, 90))},
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
        sweep[e_rate] = timed(th[e_rate], args.graph)
        progress(f"exit setting {int(100 * e_rate)}%: {sweep[e_rate]['img_s']:.0f} images/s")
    head = sweep[0.0]
    other = timed(th[0.0], not args.graph)

    # per-kernel timing (HIP events around each launch, separate pass)
    model.set_exit_thresholds([th[0.0]] * len(cfg["exits"]))
    model.profile_enable(True)
    for _ in range(args.steps):
        model.run(x, out=out)
    torch.cuda.synchronize()
    prof = model.profile_read()
    model.profile_enable(False)
    progress("per-kernel event pass done")
    work = kernel_work(cfg, head["counts"])
    kernels = {}
    for k, (ms_tot, n) in prof.items():
        if n == 0:
            continue
        entry = {"ms_per_step": ms_tot / args.steps, "launches_per_step": n / args.steps}
        if k in work:
            sec = ms_tot / args.steps / 1e3
            wk = work[k]
            if wk["flop"] > 0:
                entry["tflops"] = wk["flop"] / sec / 1e12
                entry["frac_bf16_peak"] = wk["flop"] / sec / BF16_PEAK
            entry["gbps"] = wk["byte"] / sec / 1e9
            entry["frac_hbm_peak"] = wk["byte"] / sec / HBM_PEAK
            entry["roofline_bound"] = roofline_bound(wk)
        kernels[k] = entry
    # the dominant kernel (most time per step among those with an algorithmic
    # work model), reported against the peak of its roofline resource
    dom = max((k for k in kernels if "roofline_bound" in kernels[k]),
              key=lambda k: kernels[k]["ms_per_step"])
    dk = kernels[dom]
    wk = work[dom]
    n_launch = max(1.0, dk["launches_per_step"])
    if "tflops" in dk:
        # a dense contraction (the token GEMMs, attention): on the MFMA roof,
        # with its HBM fraction on algorithmic bytes beside it
        roofline = {"kernel": dom, "bound": "mfma", "achieved": dk["tflops"],
                    "peak": BF16_PEAK / 1e12, "unit": "TFLOP/s",
                    "frac": dk["frac_bf16_peak"], "traffic": measured_traffic(dom, args.workload),
                    "hbm_gbps": dk["gbps"], "frac_hbm_peak": dk["frac_hbm_peak"],
                    "roof_binding_at_peaks": dk["roofline_bound"]}
    else:
        roofline = {"kernel": dom, "bound": "hbm", "achieved": dk["gbps"],
                    "peak": HBM_PEAK / 1e9, "unit": "GB/s",
                    "frac": dk["frac_hbm_peak"], "traffic": measured_traffic(dom, args.workload)}
    roofline["algorithmic_flop_per_launch"] = wk["flop"] / n_launch
    roofline["algorithmic_bytes_per_launch"] = wk["byte"] / n_launch
    roofline["mean_launch_us"] = dk["ms_per_step"] / n_launch * 1e3
    # the whole step on the roofline: executed FLOPs at the MFMA peak against
    # the algorithmic bytes of all kinds at the HBM peak
    step_bytes = sum(w["byte"] for w in work.values())
    step_roof = {"executed_gflop": head["flops"] / 1e9, "algorithmic_gbytes": step_bytes / 1e9,
                 "ms_at_mfma_peak": head["flops"] / BF16_PEAK * 1e3,
                 "ms_at_hbm_peak": step_bytes / HBM_PEAK * 1e3,
                 "ms_measured": head["ms"]}

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
        "timing": {"launch": "hip_graph" if args.graph else "eager",
                   "step_ms": head["step_ms"],
                   ("eager" if args.graph else "hip_graph"):
                       {"ms_per_step": other["ms"], "images_per_s": other["img_s"],
                        "step_ms": other["step_ms"]}},
        "pct_bf16_peak_executed": head["pct_peak"],
        "executed_gflop_per_image": head["flops"] / B / 1e9,
        "exit_sweep": {f"{int(100 * e)}%": {"threshold": th[e], "images_per_s": r["img_s"],
                                             "ms_per_step": r["ms"],
                                             "step_ms": r["step_ms"],
                                             "pct_bf16_peak_executed": r["pct_peak"],
                                             "measured_early_exit": r["early_exit"],
                                             "executed_gflop_per_image": r["flops"] / B / 1e9}
                       for e, r in sweep.items()},
        "roofline": roofline,
        "step_roofline": step_roof,
        "kernels": kernels,
    }
    if not args.headline_only:
        # (not in profiler runs: its copy would be taken for the counter
        # calibration copy)
        mp = measured_peaks(torch)
        line["measured_peaks"] = mp
        if roofline["unit"] == "GB/s":
            roofline["frac_of_measured"] = roofline["achieved"] / mp["hbm_copy_gbps"]
        else:
            roofline["frac_of_measured"] = roofline["achieved"] / mp["bf16_gemm_tflops"]
        if roofline["unit"] == "TFLOP/s":
            roofline["hbm_frac_of_measured_copy"] = roofline["hbm_gbps"] / mp["hbm_copy_gbps"]
        line["pct_measured_gemm_peak_executed"] = (
            100.0 * head["flops"] / (head["ms"] / 1e3) / (mp["bf16_gemm_tflops"] * 1e12))
    if not (args.no_paper or args.headline_only):
        model.close()
        energy = EnergyMeter()
        line["paper"] = paper_section(args, energy)
        progress("paper section done")
        line["ablation"] = ablation_section(args)
        progress("ablation section done")
    if not args.no_cpu:
        line["cpu_baseline"] = cpu_baseline(cfg, W, imgs, args.cpu_images)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
