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
}


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
    if isinstance(cfg.get("delta"), (int, float)):
        cfg["delta"] = tuple(float(cfg["delta"]) for _ in cfg["exits"])
    cfg["r_b"] = tuple(cfg["r"] if b in cfg["merges"] else 0
                       for b in range(1, cfg["L"] + 1))
    cfg["tau_b"] = tuple(cfg["tau"] if b in cfg["prunes"] else 1.0
                         for b in range(1, cfg["L"] + 1))
    return cfg
