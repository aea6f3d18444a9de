"""Weight-blob writer for the C library (format only, no arithmetic).

Layout (little endian), mirrored by the parser in the library:

  offset 0   char[8]  magic "FUSNVIT\\0"
             u32      version (1)
             u32      header_bytes (offset of the tensor table)
             u32      img, patch, in_ch, d, heads, L, mlp, classes
             u32      prop_attn (0/1), precision (0 = fp32, 1 = bf16)
             u32      merge_mask, exit_mask, prune_mask (bit b-1 = block b)
             u32      r_b[32]
             f64      tau_b[32]
             f32      delta_b[32]   (default exit threshold, exit blocks)
             u32      merge_rule    (0 = budget, 1 = fraction)
             u32      prune_rule    (0 = CLS attention, 1 = learned scorer)
             u32      exit_kind[32] (exit blocks: 0 = linear, 1 = CLS MLP,
                                     2 = pooled MLP; 0 elsewhere)
             u32      exit_hidden   (hidden width of the MLP exit heads)
             u32      n_tensors
  header_bytes:      n_tensors entries of
             char[32] name (NUL padded), u32 ndim, u32 shape[4],
             u64 offset (from blob start, 64-byte aligned), u64 nbytes
  then       fp32 tensor data.
"""
from __future__ import annotations

import struct

import numpy as np

from .weights import tensor_specs

MAGIC = b"FUSNVIT\0"
VERSION = 2
MAX_L = 32
_HDR_FMT = "<8sII" + "I" * 8 + "II" + "III" + "I" * MAX_L + "d" * MAX_L \
           + "f" * MAX_L + "II" + "I" * MAX_L + "I" + "I"
MERGE_RULES = {"budget": 0, "fraction": 1}
PRUNE_RULES = {"cls_attn": 0, "learned": 1}
EXIT_KINDS = {"linear": 0, "cls_mlp": 1, "pool_mlp": 2}
_ENT_FMT = "<32sI4IQQ"
HEADER_BYTES = struct.calcsize(_HDR_FMT)
ENTRY_BYTES = struct.calcsize(_ENT_FMT)


def _mask(blocks) -> int:
    m = 0
    for b in blocks:
        m |= 1 << (b - 1)
    return m


def pack(cfg: dict, weights: dict) -> bytes:
    specs = tensor_specs(cfg)
    L = cfg["L"]
    r_b = list(cfg["r_b"]) + [0] * (MAX_L - L)
    tau_b = [float(t) for t in cfg["tau_b"]] + [1.0] * (MAX_L - L)
    delta_b = [1.0] * MAX_L
    for b, dl in zip(cfg["exits"], cfg["delta"]):
        delta_b[b - 1] = float(dl)
    exit_kind = [0] * MAX_L
    for b, k in zip(cfg["exits"], cfg["exit_kind"]):
        exit_kind[b - 1] = EXIT_KINDS[k]
    hdr = struct.pack(
        _HDR_FMT, MAGIC, VERSION, HEADER_BYTES,
        cfg["img"], cfg["patch"], cfg["in_ch"], cfg["d"], cfg["H"], L,
        cfg["mlp"], cfg["C"],
        int(cfg["prop_attn"]), 1 if cfg["precision"] == "bf16" else 0,
        _mask(cfg["merges"]), _mask(cfg["exits"]), _mask(cfg["prunes"]),
        *r_b, *tau_b, *delta_b, MERGE_RULES[cfg["merge_rule"]],
        PRUNE_RULES[cfg["prune_rule"]], *exit_kind, int(cfg["exit_hidden"]),
        len(specs))
    table_end = HEADER_BYTES + ENTRY_BYTES * len(specs)
    off = (table_end + 63) // 64 * 64
    entries, chunks = [], []
    for name, shape in specs:
        a = np.ascontiguousarray(weights[name], dtype="<f4")
        if tuple(a.shape) != tuple(shape):
            raise ValueError(f"{name}: shape {a.shape} != {shape}")
        shp = list(shape) + [0] * (4 - len(shape))
        entries.append(struct.pack(_ENT_FMT, name.encode(), len(shape), *shp,
                                   off, a.nbytes))
        chunks.append((off, a.tobytes()))
        off = (off + a.nbytes + 63) // 64 * 64
    buf = bytearray(off)
    buf[:HEADER_BYTES] = hdr
    buf[HEADER_BYTES:table_end] = b"".join(entries)
    for o, data in chunks:
        buf[o:o + len(data)] = data
    return bytes(buf)
