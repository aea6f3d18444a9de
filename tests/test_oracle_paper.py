"""Pins for the paper-faithful instantiation: the merge-ratio count of
Sec. III-C with the profile rescaling of Eq. 5, the learned pruning scorer
of Eq. 8, the 2-layer MLP exit heads (CLS and size-weighted spatial pool)
and the Tab. I layer sets."""
import json
import math
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from oracle import fusion_oracle as fo
from synth import blob, configs, images, weights

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden():
    with open(os.path.join(GOLDEN, "paper_counts.json")) as f:
        return json.load(f)


# ------------------------------------------------------------ Tab. I ------
def test_paper_workload_matches_table_one():
    g = _golden()
    cfg = configs.get("deit_s_paper")
    sets = g["paper_layer_sets_deit_s"]["value"]
    assert list(cfg["merges"]) == sets["merges"]
    assert list(cfg["exits"]) == sets["exits"]
    assert list(cfg["prunes"]) == sets["prunes"]
    assert list(cfg["delta"]) == sets["delta"]
    assert all(cfg["tau_b"][b - 1] == sets["tau"] for b in cfg["prunes"])
    assert cfg["exit_kind"] == ("pool_mlp", "cls_mlp")
    assert weights.router_param_count(cfg) == g["router_params_deit_s_3_layers"]["value"]
    n = weights.exit_head_param_count(cfg)
    assert abs(n - g["exit_head_params_deit_s_approx"]["value"]) < 0.05e6, n


# ---------------------------------------------- merge ratio (Sec. III-C) --
@pytest.mark.parametrize("p,N,rho,want", [
    # floor(m~ N / 2) worked by hand, m~ = rho m
    (0.25, 196, 1.0, 24),    # 0.25 * 98 = 24.5
    (0.25, 196, 2.0, 49),    # 0.5 * 98
    (0.25, 197, 1.0, 24),    # 0.25 * 98.5 = 24.625
    (0.1, 196, 1.0, 9),      # 9.8
    (0.1, 196, 0.5, 4),      # 4.9
    (0.75, 64, 1.0, 24),     # 0.75 * 32
    (0.9, 196, 1.5, 98),     # 1.35 * 98 > 98 -> all floor(N/2) pairs
    (0.9, 7, 16.0, 3),       # clamp at floor(7/2)
    (0.3, 196, 0.0, 0),      # rho = 0: nothing merges
    (0.3, 1, 1.0, 0),        # one patch token: no pair
])
def test_fraction_rule_closed_form(p, N, rho, want):
    beta = math.log(p / (1.0 - p))
    m, r, margin = fo.router(np.zeros(8, np.float32), np.zeros(8, np.float32),
                             beta, rho, 0, N, "fraction")
    assert abs(float(m) - p) < 1e-6
    assert r == want
    assert margin >= 0.0


def test_fraction_rule_margin_is_distance_in_count_units():
    # m = 0.2501 at N = 196: t = m * 98 = 24.51; the count changes when t
    # crosses 25 or 24, so the margin is the distance to the nearer one
    beta = math.log(0.2501 / 0.7499)
    m, r, margin = fo.router(np.zeros(4, np.float32), np.zeros(4, np.float32),
                             beta, 1.0, 0, 196, "fraction")
    assert r == 24
    t = float(m) * 98.0
    assert margin == pytest.approx(min(t - 24.0, 25.0 - t), rel=1e-9)


def test_fraction_rule_ignores_budget_and_budget_rule_is_unchanged():
    z = np.zeros(4, np.float32)
    _, r1, _ = fo.router(z, z, 0.0, 1.0, 8, 196, "fraction")
    _, r2, _ = fo.router(z, z, 0.0, 1.0, 50, 196, "fraction")
    assert r1 == r2 == 49                       # m = 1/2 -> floor(196 / 4)
    _, r3, _ = fo.router(z, z, 0.0, 1.0, 8, 196, "budget")
    assert r3 == 8


# ----------------------------------------------- learned scorer (Eq. 8) ---
@pytest.mark.parametrize("seed", range(4))
def test_learned_prune_brute_force(seed):
    """Top-k by w . z + beta, computed here with Python float loops."""
    rng = np.random.default_rng(seed)
    T, d = 1 + int(rng.integers(3, 12)), 6
    x = rng.normal(size=(T, d)).astype(np.float32)
    w = rng.normal(size=d).astype(np.float32)
    beta = float(rng.normal())
    sc = fo.learned_scores(x, w, beta)
    brute = [sum(float(w[j]) * float(x[t, j]) for j in range(d)) + beta
             for t in range(T)]
    np.testing.assert_allclose(sc, brute, rtol=1e-5, atol=1e-5)
    N = T - 1
    for k in range(N + 1):
        kept, margin, _ = fo.prune_plan(sc, k, unit=1.0)
        # every kept patch outscores every dropped one (scores are distinct)
        best = sorted(range(1, T), key=lambda t: -brute[t])[:k]
        assert sorted(1 + kept) == sorted(best)
        assert list(kept) == sorted(kept)
        if 0 < k < N:
            srt = sorted(brute[1:], reverse=True)
            assert margin == pytest.approx(srt[k - 1] - srt[k], abs=1e-5)


def test_learned_prune_invariant_to_bias_and_positive_scale():
    rng = np.random.default_rng(7)
    x = rng.normal(size=(30, 16)).astype(np.float32)
    w = rng.normal(size=16).astype(np.float32)
    k0, _, _ = fo.prune_plan(fo.learned_scores(x, w, 0.0), 12, unit=1.0)
    k1, _, _ = fo.prune_plan(fo.learned_scores(x, 4.0 * w, 3.0), 12, unit=1.0)
    assert np.array_equal(k0, k1)
    # negating w keeps the complement (no ties): the bottom tokens
    k2, _, _ = fo.prune_plan(fo.learned_scores(x, -w, 0.0), 29 - 12, unit=1.0)
    assert sorted(set(range(29)) - set(k0.tolist())) == k2.tolist()


def test_learned_rule_keeps_top_scores_in_order():
    """In the pipeline, a learned prune block keeps CLS plus the k = floor(
    tau N) patch tokens of highest w . z + beta, in their sequence order."""
    cfg = configs.get("tiny_paper", delta=(1.0, 1.0))
    W = weights.make_weights(cfg, affine="random")
    Wp = fo.prepare_weights(W, "fp32")
    img = images.make_images(cfg, batch=2)
    for i in range(2):
        out = fo.run_sample(img[i], Wp, cfg, "fp32")
        for b in cfg["prunes"]:
            tb = out["trace"][b]
            sc = tb["scores"]
            N, k = sc.shape[0] - 1, tb["k"]
            before = out["trace"][b]["ids_after_merge"] if "ids_after_merge" in tb \
                else (out["trace"][b - 1]["ids"] if b - 1 in out["trace"] else None)
            top = np.sort(np.argsort(-sc[1:], kind="stable")[:k])
            assert len(tb["ids"]) == k + 1
            if before is not None:
                assert np.array_equal(np.asarray(before)[1 + top], tb["ids"][1:])


# ---------------------------------------------------------- exit heads ----
def test_spatial_pool_closed_forms():
    rng = np.random.default_rng(1)
    x = rng.normal(size=(9, 5)).astype(np.float32)
    ones = np.ones(9, np.float32)
    np.testing.assert_allclose(fo.spatial_pool(x, ones), x[1:].mean(axis=0),
                               rtol=1e-6, atol=1e-7)
    # the CLS row takes no part
    y = x.copy()
    y[0] = 1e6
    assert np.array_equal(fo.spatial_pool(y, ones), fo.spatial_pool(x, ones))
    # integer sizes = repeating each row that many times
    s = np.array([1, 1, 2, 3, 1, 4, 1, 1, 2], np.float32)
    rep = np.repeat(x[1:], s[1:].astype(int), axis=0).mean(axis=0)
    np.testing.assert_allclose(fo.spatial_pool(x, s), rep, rtol=1e-5, atol=1e-6)
    # no patch tokens: the zero vector
    assert np.array_equal(fo.spatial_pool(x[:1], ones[:1]), np.zeros(5, np.float32))


@pytest.mark.parametrize("seed", range(3))
def test_spatial_pool_is_unchanged_by_merging(seed):
    """Size-weighted merging keeps sum_t s_t z_t and sum_t s_t, so the pooled
    vector before and after a merge agrees (up to rounding)."""
    rng = np.random.default_rng(seed)
    T, d = 21, 12
    x = rng.normal(size=(T, d)).astype(np.float32)
    s = rng.integers(1, 4, size=T).astype(np.float32)
    plan = fo.merge_plan(x, 6)
    dst = plan["best"][plan["chosen"]]
    x2, s2, _, _ = fo.apply_merge(x, s, None, np.arange(T), plan["A"], plan["B"],
                                  plan["chosen"], dst)
    assert x2.shape[0] == T - 6
    np.testing.assert_allclose(fo.spatial_pool(x2, s2), fo.spatial_pool(x, s),
                               rtol=2e-5, atol=2e-6)


def test_mlp_head_matches_torch_functional():
    rng = np.random.default_rng(5)
    d, h, C = 24, 40, 7
    v = rng.normal(size=d).astype(np.float32)
    g = rng.uniform(0.5, 1.5, d).astype(np.float32)
    b = rng.normal(0, 0.1, d).astype(np.float32)
    W1 = rng.normal(0, 0.3, (h, d)).astype(np.float32)
    b1 = rng.normal(0, 0.1, h).astype(np.float32)
    W2 = rng.normal(0, 0.3, (C, h)).astype(np.float32)
    b2 = rng.normal(0, 0.1, C).astype(np.float32)
    got = fo.mlp_head_logits(v, g, b, W1, b1, W2, b2, "fp32")
    t = lambda a: torch.from_numpy(a.astype(np.float64))
    y = F.layer_norm(t(v), (d,), t(g), t(b), eps=1e-6)
    ref = F.linear(F.gelu(F.linear(y, t(W1), t(b1))), t(W2), t(b2)).numpy()
    np.testing.assert_allclose(got, ref, rtol=1e-5, atol=1e-5)


def test_exit_kinds_read_the_right_token_set():
    cfg = configs.get("tiny_paper")
    W = fo.prepare_weights(weights.make_weights(cfg, affine="random"), "fp32")
    Wb = {k[len("blk2."):]: v for k, v in W.items() if k.startswith("blk2.")}
    rng = np.random.default_rng(0)
    x = rng.normal(size=(10, cfg["d"])).astype(np.float32)
    s = np.ones(10, np.float32)
    pool = fo.exit_logits(x, s, Wb, "pool_mlp", "fp32")
    clsh = fo.exit_logits(x, s, Wb, "cls_mlp", "fp32")
    y = x.copy()
    y[0] += 1.0           # CLS moves: the pooled head does not
    assert np.array_equal(fo.exit_logits(y, s, Wb, "pool_mlp", "fp32"), pool)
    assert not np.array_equal(fo.exit_logits(y, s, Wb, "cls_mlp", "fp32"), clsh)
    z = x.copy()
    z[3] += 1.0           # a patch moves: the CLS head does not
    assert np.array_equal(fo.exit_logits(z, s, Wb, "cls_mlp", "fp32"), clsh)
    assert not np.array_equal(fo.exit_logits(z, s, Wb, "pool_mlp", "fp32"), pool)


# ------------------------------------------------------ whole pipeline ----
@pytest.mark.parametrize("mode", ["fp32", "bf16emu"])
def test_paper_rules_disabled_are_plain_vit_bit_exact(mode):
    """delta = 1 and rho = 0: m~ = 0 merges nothing, tau' = 1 keeps all."""
    cfg = configs.get("tiny_paper")
    W = weights.make_weights(cfg, affine="random")
    img = images.make_images(cfg, batch=2)
    lg, eb, cnt, _ = oracle.run(img, W, cfg, mode, delta=[1.0, 1.0], rho=0.0)
    Wp = fo.prepare_weights(W, mode)
    for i in range(2):
        assert np.array_equal(lg[i], fo.plain_forward(img[i], Wp, cfg, mode))
        assert eb[i] == cfg["L"] and np.all(cnt[i] == cfg["N0"] + 1)


def test_paper_token_counts_follow_rules():
    cfg = configs.get("tiny_paper", delta=(1.0, 1.0))
    W = weights.make_weights(cfg)
    imgs = images.make_images(cfg, batch=4)
    _, _, cnt, res = oracle.run(imgs, W, cfg, "fp32")
    for i in range(4):
        tr = res[i]["trace"]
        T = cfg["N0"] + 1
        for b in range(1, cfg["L"] + 1):
            assert cnt[i][b - 1] == T
            N = T - 1
            if b in cfg["merges"]:
                m = tr[b]["m"]
                assert tr[b]["r"] == min(math.floor(float(m) * N * 0.5), N // 2)
                T -= tr[b]["r"]
                N = T - 1
            if b in cfg["prunes"]:
                assert tr[b]["k"] == math.floor(0.7 * N)
                T = 1 + tr[b]["k"]


def test_exit_trajectory_with_mlp_heads():
    """Every exited sample stops at the first exit head whose confidence
    reaches its threshold; the others pass every head below threshold."""
    cfg = configs.get("tiny_paper")
    W = weights.make_weights(cfg)
    imgs = images.make_images(cfg, batch=16)
    delta = (0.45, 0.6)
    lg, eb, _, res = oracle.run(imgs, W, cfg, "fp32", delta=delta)
    for i in range(16):
        tr = res[i]["trace"]
        seen = [b for b in cfg["exits"] if b in tr and "c" in tr[b]]
        for b in seen:
            dl = delta[cfg["exits"].index(b)]
            if b < eb[i]:
                assert tr[b]["c"] < dl
            else:
                assert b == eb[i] and tr[b]["c"] >= dl
                assert np.array_equal(lg[i], tr[b]["exit_logits"])
    assert len(set(eb.tolist())) >= 2


def test_executed_flops_mlp_heads():
    cfg = configs.get("deit_s_paper")
    cnt = np.full(12, 197)
    f_all = fo.executed_flops(cfg, cnt, 12)
    base = fo.executed_flops(configs.get("deit_s_paper", exits=(),
                                         exit_kind=(), delta=()), cnt, 12)
    hx, d, C = 768, 384, 1000
    assert f_all - base == 2 * (2 * d * hx + 2 * hx * C)


def test_blob_header_carries_rules():
    cfg = configs.get("deit_s_paper")
    W = weights.make_weights(cfg)
    b = blob.pack(cfg, W)
    import struct
    assert struct.unpack_from("<I", b, 8)[0] == 2
    assert blob.HEADER_BYTES == 724
    mr, pr = struct.unpack_from("<II", b, 580)
    kinds = struct.unpack_from("<32I", b, 588)
    hx, nt = struct.unpack_from("<II", b, 716)
    assert (mr, pr, hx) == (1, 1, 768)
    assert kinds[7] == 2 and kinds[9] == 1 and sum(kinds) == 3
    assert nt == len(weights.tensor_specs(cfg))


def test_full_prune_leaves_cls_and_empty_pool():
    """tau' = 0 at rho = 4 keeps no patch token; a pooled head after that
    pools the zero vector, whose LayerNorm is the LN bias."""
    cfg = configs.get("tiny_paper", exits=(2, 4), exit_kind=("cls_mlp", "pool_mlp"))
    W = weights.make_weights(cfg, affine="random")
    Wp = fo.prepare_weights(W, "fp32")
    img = images.make_images(cfg, batch=1)
    out = fo.run_sample(img[0], Wp, cfg, "fp32", delta=(1.0, 1.0), rho=4.0)
    assert out["token_counts"][3] == 1
    W4 = {k[len("blk4."):]: v for k, v in Wp.items() if k.startswith("blk4.")}
    y = W4["eln_b"][None, :]
    ref = (fo.gelu(y @ W4["ew1"].T + W4["eb1"]) @ W4["ew2"].T + W4["eb2"])[0]
    np.testing.assert_allclose(out["trace"][4]["exit_logits"], ref, rtol=1e-6, atol=1e-6)
