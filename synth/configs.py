"""Workload definitions: backbone shapes, layer sets and adaptive settings.

These are plain data (no arithmetic of the method).  The five workloads are
DeiT-family shapes; the layer sets, merge counts and keep ratios are fixed
here once and read identically by the CPU oracle and by the weight-blob
writer (the blob carries them to the GPU library).

Layer sets (the paper's M, E, P of the Preliminaries, Sec. III-A) are 1-based
block indices.  ``r`` is the per-block merge budget r_b, ``tau`` the keep
ratio tau_b of Eq. 8, ``delta`` the default exit threshold per exit block
(Eq. 7).  ``exit_gain`` is the gain g of the exit/final head init,
N(0, (g/sqrt(d))^2), chosen so that confidences spread around the thresholds
with random backbones.  The gains were picked once by running the oracle
over the workload's first images: tiny 0.7, DeiT-Ti 2.7 and DeiT-B 4.0 put
the fixed thresholds (0.5 / 0.6) inside the confidence distribution (about
20-80 % early exits); DeiT-S (224 and 384) use 6.0, whose confidences spread
over roughly 0.3-0.95 so that thresholds set at exit-rate percentiles are
well separated.

Rules (strings, read by both sides through the blob header):
``merge_rule``  "budget"   -- r = clamp(floor(2 rho m r_b + 1/2), 0, N/2);
                "fraction" -- r = floor(rho m N / 2), at most N/2: the merge
                              ratio of Sec. III-C applied to the candidate
                              pairs, rescaled by the profile ratio of Eq. 5.
``prune_rule``  "cls_attn" -- token scores = head-mean CLS attention;
                "learned"  -- s_i = w . z_i + beta, a linear scorer h_b
                              (Eq. 8) with weights prune_w, prune_b.
``exit_kind``   per exit block: "linear" (LN + linear on CLS), "cls_mlp"
                (LN + 2-layer MLP on CLS) or "pool_mlp" (size-weighted mean
                of the patch tokens, then LN + 2-layer MLP); ``exit_hidden``
                is the MLP hidden width.

The ``*_paper`` workloads instantiate Tab. I: M = {3,5,7}, E = {8,10} with
a SpatialPool MLP head at block 8 and a CLS MLP head at block 10, P =
{9,10} with the learned scorer, delta = (0.8, 0.95), tau = 0.7, merge
ratios from the routers.  Hidden width 2d gives 2 x (d 2d + 2d C) ~ 2.1M
head parameters at DeiT-S, the total the paper states.  The router bias
-2 starts the merge ratio near sigmoid(-2) = 0.12 (about 11 of 98 pairs at
block 3), and ``exit_gain`` 60 puts about 85-90 % of the block-8
confidences above 0.8 with random backbones (the trained exit rate at
block 8 is about 89 %, Tab. VII).
"""
from __future__ import annotations

import copy

_BASE_DEIT = dict(img=224, patch=16, in_ch=3, L=12, C=1000, prop_attn=1,
                  precision="bf16", tau=0.7, exits=(4, 8), prunes=(4, 7, 10))

CONFIGS = {
    # 32x32 images, patch 4 -> 64 patches + CLS; fp32 end to end.
    "tiny": dict(index=1, img=32, patch=4, in_ch=3, d=64, H=2, L=4, mlp=256,
                 C=10, batch=8, precision="fp32", prop_attn=1,
                 merges=(1, 2, 3, 4), r=4, exits=(2,), delta=0.5,
                 prunes=(1, 2, 3, 4), tau=0.75, exit_gain=0.7),
    # DeiT-Ti shape: 196 patches + CLS, d=192, 3 heads.
    "deit_ti": dict(_BASE_DEIT, index=2, d=192, H=3, mlp=768, batch=64,
                    merges=tuple(range(1, 13)), r=8, delta=0.6,
                    exit_gain=2.7),
    # DeiT-S shape: d=384, 6 heads, batch 256 (the headline workload).
    "deit_s": dict(_BASE_DEIT, index=3, d=384, H=6, mlp=1536, batch=256,
                   merges=tuple(range(1, 13)), r=8, delta=0.6,
                   exit_gain=6.0),
    # DeiT-B shape: d=768, 12 heads.
    "deit_b": dict(_BASE_DEIT, index=4, d=768, H=12, mlp=3072, batch=256,
                   merges=tuple(range(1, 13)), r=12, delta=0.6,
                   exit_gain=4.0),
    # DeiT-S at 384x384: 576 patches + CLS, batch 64.
    "deit_s_384": dict(_BASE_DEIT, index=5, img=384, d=384, H=6, mlp=1536,
                       batch=64, merges=tuple(range(1, 13)), r=24,
                       delta=0.6, exit_gain=6.0),
    # Tab. I layer sets and rules at the tiny shape (fp32, parity workload).
    "tiny_paper": dict(index=6, img=32, patch=4, in_ch=3, d=64, H=2, L=4,
                       mlp=256, C=10, batch=16, precision="fp32",
                       prop_attn=1, merges=(1, 2), r=0, exits=(2, 3),
                       delta=(0.5, 0.6), prunes=(3, 4), tau=0.7,
                       exit_gain=3.0, merge_rule="fraction",
                       prune_rule="learned",
                       exit_kind=("pool_mlp", "cls_mlp"), exit_hidden=128,
                       router_bias=-1.0),
    # Tab. I: DeiT-S with the paper's layer sets, heads and rules.
    "deit_s_paper": dict(_BASE_DEIT, index=7, d=384, H=6, mlp=1536,
                         batch=256, merges=(3, 5, 7), r=0, exits=(8, 10),
                         delta=(0.8, 0.95), prunes=(9, 10), tau=0.7,
                         exit_gain=60.0, merge_rule="fraction",
                         prune_rule="learned",
                         exit_kind=("pool_mlp", "cls_mlp"), exit_hidden=768,
                         router_bias=-2.0),
}


# Operating profiles of the paper workloads (Sec. IV-A, Profiles; Tab. I):
# per profile the exit thresholds delta_b and the target keep ratio tau_tgt;
# the router strength is rho = (1 - tau_tgt) / (1 - tau_tgt(balanced)), the
# rescaling of Eq. 5, which also scales the prune keep ratios.  balanced is
# the reference profile of Tab. I.  The paper gives no power_save values;
# this one takes tau_tgt = 0.5 and thresholds lowered by 0.1 / 0.05.
PROFILES = {
    "balanced": dict(delta=(0.8, 0.95), tau_tgt=0.7),
    "power_save": dict(delta=(0.7, 0.9), tau_tgt=0.5),
}


# Tab. VII rows (Sec. IV-F, Ablation Study) as layer-set overrides of a
# Tab. I workload, each with the profile it runs under.  "parallel prune +
# exit" prunes at blocks that every sample reaches before the first exit
# head; "full sequential, fixed r" merges a fixed budget with zero routers
# (the budget rule at m = 1/2 merges exactly r pairs).  ABLATION is the
# DeiT-S (deit_s_paper) version, ABLATION_TINY the same compositions on the
# four-block tiny_paper shape.
ABLATION = [
    ("plain", dict(merges=(), exits=(), prunes=()), "balanced"),
    ("pruning only", dict(merges=(), exits=()), "balanced"),
    ("merging only", dict(exits=(), prunes=()), "balanced"),
    ("early exit only", dict(merges=(), prunes=()), "balanced"),
    ("parallel prune + exit", dict(merges=(), prunes=(3, 6, 9)), "balanced"),
    ("sequential exit -> prune", dict(merges=()), "balanced"),
    ("full sequential, fixed r=8 merges", dict(merge_rule="budget", r=8), "balanced"),
    ("full sequential, merge routers", dict(), "balanced"),
    ("full sequential, routers + power_save scaling", dict(), "power_save"),
]
ABLATION_SUPERSET_PRUNES = (3, 6, 9, 10)

ABLATION_TINY = [
    ("plain", dict(merges=(), exits=(), prunes=()), "balanced"),
    ("pruning only", dict(merges=(), exits=()), "balanced"),
    ("merging only", dict(exits=(), prunes=()), "balanced"),
    ("early exit only", dict(merges=(), prunes=()), "balanced"),
    ("parallel prune + exit", dict(merges=(), prunes=(1, 2)), "balanced"),
    ("sequential exit -> prune", dict(merges=()), "balanced"),
    ("full sequential, fixed r=4 merges", dict(merge_rule="budget", r=4), "balanced"),
    ("full sequential, merge routers", dict(), "balanced"),
    ("full sequential, routers + power_save scaling", dict(), "power_save"),
]
ABLATION_TINY_SUPERSET_PRUNES = (1, 2, 3, 4)


def ablation_config(base: str, over: dict, **extra) -> dict:
    """The workload of one ablation row (no exit heads: no kinds or
    thresholds either)."""
    o = dict(over)
    if "exits" in o and not o["exits"]:
        o.update(exit_kind=(), delta=())
    o.update(extra)
    return get(base, **o)


def profile_settings(name: str, ref: str = "balanced") -> dict:
    """delta and rho of a named profile (Eq. 5 ratio against ``ref``)."""
    p, r = PROFILES[name], PROFILES[ref]
    return dict(delta=tuple(p["delta"]),
                rho=(1.0 - p["tau_tgt"]) / (1.0 - r["tau_tgt"]))


def get(name: str, **overrides) -> dict:
    """Return a deep copy of workload ``name`` with derived sizes filled in."""
    cfg = copy.deepcopy(CONFIGS[name])
    cfg.update(overrides)
    cfg["name"] = name
    g = cfg["img"] // cfg["patch"]
    cfg["grid"] = g
    cfg["N0"] = g * g
    cfg["dh"] = cfg["d"] // cfg["H"]
    cfg["patch_dim"] = cfg["in_ch"] * cfg["patch"] * cfg["patch"]
    cfg.setdefault("merge_rule", "budget")
    cfg.setdefault("prune_rule", "cls_attn")
    cfg.setdefault("exit_hidden", 0)
    cfg.setdefault("router_bias", 0.0)
    if "exit_kind" not in cfg:
        cfg["exit_kind"] = tuple("linear" for _ in cfg["exits"])
    cfg["exit_kind"] = tuple(cfg["exit_kind"])
    if len(cfg["exit_kind"]) != len(cfg["exits"]):
        raise ValueError("one exit_kind per exit block")
    if isinstance(cfg.get("delta"), (int, float)):
        cfg["delta"] = tuple(float(cfg["delta"]) for _ in cfg["exits"])
    cfg["r_b"] = tuple(cfg["r"] if b in cfg["merges"] else 0
                       for b in range(1, cfg["L"] + 1))
    cfg["tau_b"] = tuple(cfg["tau"] if b in cfg["prunes"] else 1.0
                         for b in range(1, cfg["L"] + 1))
    return cfg
