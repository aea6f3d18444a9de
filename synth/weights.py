"""Seeded random weights for a DeiT-style backbone with Fusion's add-ons.

Pure data generation: every tensor is drawn from a NumPy PCG64 stream with a
fixed seed.  Nothing here evaluates the network.

Init (random-init backbone, N(0, 0.02) for cls, pos and every matrix):
  * ``affine="plain"``  -- biases 0, LayerNorm gamma 1 / beta 0.
  * ``affine="random"`` -- biases N(0, 0.05), gamma U(0.5, 1.5),
    beta N(0, 0.05); used by parity tests so that a misplaced bias or LN
    parameter cannot cancel out.
Exit heads and the final classifier use N(0, (g/sqrt(d))^2) with
g = cfg["exit_gain"], so that max-softmax confidences spread over (0, 1)
instead of sitting near 1/C; for MLP exit heads the first layer is
N(0, 1/d) (unit-scale hidden pre-activations) and the second
N(0, (g/sqrt(hidden))^2).  Router weights use ``router_std`` (0.02 by
default; a larger value spreads the per-sample merge counts) and the bias
``router_bias`` (the workload's value by default).  The learned pruning
scorer uses N(0, 1/d), bias 0 (plain) or N(0, 0.05) (random).

Tensor names, order and layouts are the ones the C library's blob parser
expects (see ``synth.blob``):
  cls[d], pos[N0+1, d], pe_w[d, C_in*p*p] with (c, ky, kx) order, pe_b[d];
  per block b: ln1_g, ln1_b, qkv_w[3d, d] (rows q|k|v, each head-major),
  qkv_b[3d], proj_w[d, d], proj_b, ln2_g, ln2_b, fc1_w[mlp, d], fc1_b,
  fc2_w[d, mlp], fc2_b;
  per merge block: router_w[d], router_b[1];
  per exit block: eln_g, eln_b, then ew[C, d], eb[C] ("linear") or
      ew1[hidden, d], eb1[hidden], ew2[C, hidden], eb2[C] (MLP kinds);
  per prune block with the learned scorer: prune_w[d], prune_b[1];
  final: norm_g, norm_b, head_w[C, d], head_b[C].
"""
from __future__ import annotations

import numpy as np


def tensor_specs(cfg: dict):
    """Ordered list of (name, shape) for a workload."""
    d, mlp, C, N0 = cfg["d"], cfg["mlp"], cfg["C"], cfg["N0"]
    specs = [("cls", (d,)), ("pos", (N0 + 1, d)),
             ("pe_w", (d, cfg["patch_dim"])), ("pe_b", (d,))]
    for b in range(1, cfg["L"] + 1):
        p = f"blk{b}."
        specs += [(p + "ln1_g", (d,)), (p + "ln1_b", (d,)),
                  (p + "qkv_w", (3 * d, d)), (p + "qkv_b", (3 * d,)),
                  (p + "proj_w", (d, d)), (p + "proj_b", (d,)),
                  (p + "ln2_g", (d,)), (p + "ln2_b", (d,)),
                  (p + "fc1_w", (mlp, d)), (p + "fc1_b", (mlp,)),
                  (p + "fc2_w", (d, mlp)), (p + "fc2_b", (d,))]
        if b in cfg["merges"]:
            specs += [(p + "router_w", (d,)), (p + "router_b", (1,))]
        if b in cfg["exits"]:
            kind = cfg["exit_kind"][cfg["exits"].index(b)]
            specs += [(p + "eln_g", (d,)), (p + "eln_b", (d,))]
            if kind == "linear":
                specs += [(p + "ew", (C, d)), (p + "eb", (C,))]
            else:
                hx = cfg["exit_hidden"]
                specs += [(p + "ew1", (hx, d)), (p + "eb1", (hx,)),
                          (p + "ew2", (C, hx)), (p + "eb2", (C,))]
        if b in cfg["prunes"] and cfg["prune_rule"] == "learned":
            specs += [(p + "prune_w", (d,)), (p + "prune_b", (1,))]
    specs += [("norm_g", (d,)), ("norm_b", (d,)),
              ("head_w", (C, d)), ("head_b", (C,))]
    return specs


def make_weights(cfg: dict, seed: int | None = None, affine: str = "plain",
                 router_std: float = 0.02, router_bias: float | None = None) -> dict:
    """Draw every tensor of ``tensor_specs(cfg)`` as float32."""
    if router_bias is None:
        router_bias = cfg.get("router_bias", 0.0)
    if seed is None:
        seed = cfg["index"]
    rng = np.random.Generator(np.random.PCG64(seed))
    d = cfg["d"]
    head_std = cfg["exit_gain"] / np.sqrt(d)
    out = {}
    for name, shape in tensor_specs(cfg):
        leaf = name.split(".")[-1]
        if leaf in ("ln1_g", "ln2_g", "eln_g", "norm_g"):
            if affine == "random":
                a = rng.uniform(0.5, 1.5, size=shape)
            else:
                a = np.ones(shape)
        elif leaf in ("ln1_b", "ln2_b", "eln_b", "norm_b", "pe_b", "qkv_b",
                      "proj_b", "fc1_b", "fc2_b", "eb", "eb1", "eb2", "head_b",
                      "prune_b"):
            if affine == "random":
                a = rng.normal(0.0, 0.05, size=shape)
            else:
                a = np.zeros(shape)
        elif leaf == "router_b":
            a = np.full(shape, router_bias)
        elif leaf == "router_w":
            a = rng.normal(0.0, router_std, size=shape)
        elif leaf in ("ew", "head_w"):
            a = rng.normal(0.0, head_std, size=shape)
        elif leaf in ("ew1", "prune_w"):
            a = rng.normal(0.0, 1.0 / np.sqrt(d), size=shape)
        elif leaf == "ew2":
            a = rng.normal(0.0, cfg["exit_gain"] / np.sqrt(shape[1]), size=shape)
        else:  # cls, pos, pe_w, qkv_w, proj_w, fc1_w, fc2_w
            a = rng.normal(0.0, 0.02, size=shape)
        out[name] = np.ascontiguousarray(a, dtype=np.float32)
    return out


def zero_routers(cfg: dict, weights: dict) -> dict:
    """Copy of ``weights`` with every merge router set to w = 0, beta = 0."""
    w = dict(weights)
    for b in cfg["merges"]:
        w[f"blk{b}.router_w"] = np.zeros_like(weights[f"blk{b}.router_w"])
        w[f"blk{b}.router_b"] = np.zeros_like(weights[f"blk{b}.router_b"])
    return w


def backbone_param_count(cfg: dict) -> int:
    """Parameters of the plain backbone (patch embed, blocks, final head)."""
    n = 0
    for name, shape in tensor_specs(cfg):
        leaf = name.split(".")[-1]
        if leaf.startswith("router") or leaf.startswith("prune") or leaf in (
                "eln_g", "eln_b", "ew", "eb", "ew1", "eb1", "ew2", "eb2"):
            continue
        n += int(np.prod(shape))
    return n


def exit_head_param_count(cfg: dict) -> int:
    """Parameters of the exit heads (LayerNorm included)."""
    n = 0
    for name, shape in tensor_specs(cfg):
        if name.split(".")[-1] in ("eln_g", "eln_b", "ew", "eb", "ew1", "eb1",
                                   "ew2", "eb2"):
            n += int(np.prod(shape))
    return n


def router_param_count(cfg: dict) -> int:
    n = 0
    for name, shape in tensor_specs(cfg):
        if name.split(".")[-1].startswith("router"):
            n += int(np.prod(shape))
    return n
