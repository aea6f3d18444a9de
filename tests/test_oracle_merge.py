"""Pins for the oracle's bipartite soft matching and size-weighted merge
(Sec. III-C): invariants on every merge and brute force on tiny inputs."""
import itertools
import math

import numpy as np
import pytest

import oracle
from oracle import fusion_oracle as fo
from synth import configs, images, weights


def _state(rng, N, d, sizes=True):
    x = rng.standard_normal((N + 1, d)).astype(np.float32)
    s = (rng.integers(1, 5, N + 1).astype(np.float32) if sizes
         else np.ones(N + 1, np.float32))
    sc = rng.uniform(0, 1, N + 1).astype(np.float32)
    sc /= sc.sum()
    origin = np.arange(N + 1) * 3 + 7
    return x, s, sc, origin


def _merge(x, s, sc, origin, r):
    plan = fo.merge_plan(x, r)
    if r == 0:
        return plan, (x, s, sc, origin)
    return plan, fo.apply_merge(x, s, sc, origin, plan["A"], plan["B"],
                                plan["chosen"], plan["best"][plan["chosen"]])


@pytest.mark.parametrize("N,r", [(2, 1), (9, 3), (10, 5), (16, 4), (17, 8),
                                 (196, 8), (196, 98), (576, 24)])
def test_merge_invariants(N, r):
    rng = np.random.default_rng(N * 100 + r)
    x, s, sc, origin = _state(rng, N, 48)
    plan, (x2, s2, sc2, o2) = _merge(x, s, sc, origin, r)
    # count: N - r patch tokens plus CLS
    assert x2.shape[0] == N + 1 - r
    # CLS untouched and first
    assert np.array_equal(x2[0], x[0]) and o2[0] == origin[0]
    # total size preserved exactly (integer-valued float32)
    assert s2.sum(dtype=np.float64) == s.sum(dtype=np.float64)
    # size-weighted sum preserved, so the size-weighted mean is preserved
    tot = (s[:, None].astype(np.float64) * x).sum(0)
    tot2 = (s2[:, None].astype(np.float64) * x2).sum(0)
    np.testing.assert_allclose(tot2, tot, rtol=1e-6, atol=1e-5)
    # CLS scores add through the merge
    assert abs(sc2.sum(dtype=np.float64) - sc.sum(dtype=np.float64)) < 1e-6
    # survivors keep their relative order
    assert np.all(np.diff(o2) > 0)
    # each output is the size-weighted mean of its provenance group
    groups = {int(o): [int(o)] for o in o2}
    A, B = plan["A"], plan["B"]
    for a in plan["chosen"]:
        groups[int(origin[1 + B[plan["best"][a]]])].append(int(origin[1 + A[a]]))
    row_of = {int(o): i for i, o in enumerate(origin)}
    for i, o in enumerate(o2):
        rows = [row_of[g] for g in groups[int(o)]]
        w = s[rows].astype(np.float64)
        np.testing.assert_allclose(x2[i], (w[:, None] * x[rows]).sum(0) / w.sum(),
                                   rtol=1e-5, atol=1e-5)
        assert s2[i] == s[rows].sum()


def test_merge_r_zero_is_identity_and_r_max_merges_all_of_a():
    rng = np.random.default_rng(5)
    x, s, sc, origin = _state(rng, 20, 16)
    _, (x2, s2, sc2, o2) = _merge(x, s, sc, origin, 0)
    assert np.array_equal(x2, x) and np.array_equal(o2, origin)
    plan, (x3, s3, sc3, o3) = _merge(x, s, sc, origin, 10)
    A = plan["A"]
    assert set(o3.tolist()) == set(origin.tolist()) - {int(origin[1 + a]) for a in A}


def _py_cos(u, v):
    nu = math.sqrt(sum(float(t) * float(t) for t in u))
    nv = math.sqrt(sum(float(t) * float(t) for t in v))
    return sum(float(a) * float(b) for a, b in zip(u, v)) / (nu * nv)


@pytest.mark.parametrize("seed", range(12))
def test_merge_brute_force_tiny(seed):
    """Pure-Python loops: pairwise cosine, argmax, and an exhaustive search
    over all r-subsets of A maximising the summed best similarity."""
    rng = np.random.default_rng(100 + seed)
    N = int(rng.integers(3, 13))
    r = int(rng.integers(0, N // 2 + 1))
    x, s, sc, origin = _state(rng, N, 6)
    P = x[1:]
    A = list(range(0, N, 2))
    B = list(range(1, N, 2))
    best, bestsim = [], []
    for a in A:
        sims = [_py_cos(P[a], P[b]) for b in B]
        j = max(range(len(B)), key=lambda t: (sims[t], -t))
        best.append(j)
        bestsim.append(sims[j])
    subsets = list(itertools.combinations(range(len(A)), r))
    top = max(subsets, key=lambda c: sum(bestsim[i] for i in c))
    plan, (x2, s2, _, o2) = _merge(x, s, sc, origin, r)
    assert sorted(plan["chosen"].tolist()) == sorted(top)
    if r:
        assert plan["best"].tolist() == best
        np.testing.assert_allclose(plan["bestsim"], bestsim, rtol=1e-5, atol=1e-6)
    # merged values by explicit loops
    exp_rows = []
    chosen = set(top)
    for t in range(N + 1):
        if t == 0:
            exp_rows.append((x[0].astype(np.float64), s[0], origin[0]))
            continue
        j = t - 1
        if j % 2 == 0 and (j // 2) in chosen:
            continue
        num = s[t] * x[t].astype(np.float64)
        den = float(s[t])
        if j % 2 == 1:
            for i in sorted(chosen):
                if best[i] == j // 2:
                    num = num + s[1 + A[i]] * x[1 + A[i]].astype(np.float64)
                    den += float(s[1 + A[i]])
        exp_rows.append((num / den, den, origin[t]))
    assert len(exp_rows) == x2.shape[0]
    for (v, dn, o), xv, sv, ov in zip(exp_rows, x2, s2, o2):
        np.testing.assert_allclose(xv, v, rtol=1e-5, atol=1e-6)
        assert sv == dn and ov == o


def test_merge_ties_go_to_lowest_slots():
    d = 4
    base = np.array([1.0, 0.0, 0.0, 0.0], np.float32)
    # all patch tokens identical: every similarity ties at 1
    x = np.stack([np.full(d, 3.0, np.float32)] + [base] * 8)
    plan = fo.merge_plan(x, 2)
    assert plan["best"].tolist() == [0, 0, 0, 0]
    assert plan["chosen"].tolist() == [0, 1]


def test_merge_count_uses_floor_half_pairs():
    """The count never exceeds floor(N/2), the number of B tokens."""
    for N in range(0, 12):
        m, r, _ = fo.router(np.zeros(8, np.float32), np.zeros(8, np.float32),
                            50.0, 1.0, 100, N)
        assert r == N // 2


def test_oracle_run_merge_keeps_mean_through_pipeline():
    """Across a whole staged run (no prune at block 1) the size-weighted mean
    of block 1's output survives the merge."""
    cfg = configs.get("tiny")
    W = fo.prepare_weights(weights.make_weights(cfg), "fp32")
    img = images.make_images(cfg, batch=1)[0]
    x = fo.patch_embed(img, W, cfg, "fp32")
    s = np.ones(x.shape[0], np.float32)
    x, sc = fo.block(x, s, fo._b_weights(W, 1), cfg, "fp32", want_cls=True)
    plan, (x2, s2, sc2, _) = _merge(x, s, sc, np.arange(x.shape[0]), 4)
    np.testing.assert_allclose((s2[:, None] * x2).sum(0) / s2.sum(),
                               (s[:, None] * x).sum(0) / s.sum(), rtol=1e-5, atol=1e-6)
    assert abs(float(sc2.sum()) - 1.0) < 1e-5
