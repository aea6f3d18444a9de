"""Seeded synthetic images: low-frequency sinusoids plus Gaussian noise.

Per image i and channel c:
    x[c, y, x] = sum_{k=1..3} a_k sin(2 pi (fx_k x / W + fy_k y / H) + phi_k)
                 + sigma_i * eps
with a ~ U(0, 1), fx, fy ~ U(-4, 4) cycles per image, phi ~ U(0, 2 pi),
sigma_i ~ U(0, 1) per image and eps ~ N(0, 1).  Computed in float64 and
stored as float32 NCHW.
"""
from __future__ import annotations

import numpy as np


def make_images(cfg: dict, batch: int | None = None, seed: int | None = None,
                first: int = 0) -> np.ndarray:
    """Images ``first .. first+batch-1`` of the workload's seeded stream.

    Every image has its own generator (seed, image index), so image j is the
    same whatever batch it is drawn in.
    """
    if batch is None:
        batch = cfg["batch"]
    if seed is None:
        seed = 1000 + cfg["index"]
    C, S = cfg["in_ch"], cfg["img"]
    yy, xx = np.meshgrid(np.arange(S, dtype=np.float64),
                         np.arange(S, dtype=np.float64), indexing="ij")
    out = np.empty((batch, C, S, S), dtype=np.float32)
    for j in range(batch):
        rng = np.random.Generator(np.random.PCG64([seed, first + j]))
        sigma = rng.uniform(0.0, 1.0)
        for c in range(C):
            acc = np.zeros((S, S), dtype=np.float64)
            for _ in range(3):
                a = rng.uniform(0.0, 1.0)
                fx, fy = rng.uniform(-4.0, 4.0, size=2)
                phi = rng.uniform(0.0, 2.0 * np.pi)
                acc += a * np.sin(2.0 * np.pi * (fx * xx / S + fy * yy / S)
                                  + phi)
            acc += sigma * rng.standard_normal((S, S))
            out[j, c] = acc.astype(np.float32)
    return out
