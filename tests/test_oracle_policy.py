"""Pins for the router (Eq. 4-5), exit rule (Eq. 6-7, Alg. 1), prune
(Eq. 8) and the staged ordering (Sec. III-B)."""
import json
import math
import os

import numpy as np
import pytest

import oracle
from oracle import fusion_oracle as fo
from synth import configs, images, weights

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden():
    with open(os.path.join(GOLDEN, "paper_counts.json")) as f:
        return json.load(f)


def test_router_param_count_matches_paper():
    """d + 1 parameters per merge layer; 1,155 for three DeiT-S layers."""
    g = _golden()
    cfg = configs.get("deit_s", merges=(3, 5, 7))
    assert weights.router_param_count(cfg) == g["router_params_deit_s_3_layers"]["value"]
    cfg1 = configs.get("deit_s", merges=(1,))
    assert weights.router_param_count(cfg1) == cfg["d"] + 1


def test_backbone_param_count_is_deit_s():
    """About 22M backbone parameters for DeiT-S (Table I)."""
    g = _golden()
    cfg = configs.get("deit_s")
    n = weights.backbone_param_count(cfg)
    assert n == 22050664
    assert abs(n - g["deit_s_backbone_params_approx"]["value"]) < 0.1e6


@pytest.mark.parametrize("rho", [0.0, 0.25, 0.5, 1.0, 1.5, 2.0])
@pytest.mark.parametrize("r_b", [4, 8, 12, 24])
def test_zero_router_gives_scaled_budget(rho, r_b):
    """w = 0, beta = 0 -> m = 1/2 exactly -> r = floor(rho r_b + 1/2)."""
    m, r, _ = fo.router(np.ones(16, np.float32), np.zeros(16, np.float32),
                        0.0, rho, r_b, 1000)
    assert m == np.float32(0.5)
    assert r == math.floor(rho * r_b + 0.5)
    if rho == 1.0:
        assert r == r_b


def test_router_sigmoid_and_margin():
    w = np.array([0.5, -0.25], np.float32)
    x = np.array([2.0, 4.0], np.float32)
    m, r, margin = fo.router(x, w, 0.3, 1.0, 8, 100)
    z = 0.5 * 2 - 0.25 * 4 + 0.3
    assert abs(float(m) - 1 / (1 + math.exp(-z))) < 1e-7
    t = 2 * float(m) * 8 + 0.5
    assert r == math.floor(t) and abs(margin - abs(t - round(t))) < 1e-12


@pytest.mark.parametrize("N", [0, 1, 5, 137, 196, 576])
@pytest.mark.parametrize("tau,rho", [(0.7, 1.0), (0.7, 0.0), (0.7, 0.5),
                                     (0.7, 1.5), (0.75, 1.0), (0.7, 4.0)])
def test_keep_count_closed_form(N, tau, rho):
    k = fo.keep_count(N, tau, rho)
    eff = min(1.0, max(0.0, 1.0 - rho * (1.0 - tau)))
    assert k == math.floor(eff * N)
    if rho == 0.0:
        assert k == N
    assert 0 <= k <= N


def test_prune_topk_is_full_stable_sort():
    rng = np.random.default_rng(3)
    for _ in range(50):
        N = int(rng.integers(1, 60))
        sc = rng.integers(0, 6, N + 1).astype(np.float32) / 7   # many ties
        k = int(rng.integers(0, N + 1))
        kept, _, _ = fo.prune_plan(sc, k)
        ref = sorted(range(N), key=lambda j: (-float(sc[1 + j]), j))[:k]
        assert kept.tolist() == sorted(ref)


def _run(cfg, W, imgs, **kw):
    return oracle.run(imgs, W, cfg, "fp32" if cfg["precision"] == "fp32" else "bf16emu", **kw)


def test_exit_trajectory_first_head_over_threshold():
    """exit_block = min{b in E : c_b >= delta_b}; exited logits are exactly
    head_b's logits from the run without exits (Alg. 1, exit branch)."""
    cfg = configs.get("deit_ti", batch=6)
    W = weights.make_weights(cfg)
    imgs = images.make_images(cfg, batch=6)
    _, eb0, cnt0, res0 = _run(cfg, W, imgs, delta=[1.0, 1.0])
    assert np.all(eb0 == cfg["L"])
    cs = np.array([[r["trace"][b]["c"] for b in cfg["exits"]] for r in res0])
    delta = float(np.median(cs.max(axis=1)))
    lg, eb, cnt, res = _run(cfg, W, imgs, delta=[delta, delta])
    n_exit = 0
    for i, r0 in enumerate(res0):
        fired = [b for b in cfg["exits"] if r0["trace"][b]["c"] >= np.float32(delta)]
        if fired:
            n_exit += 1
            b = fired[0]
            assert eb[i] == b
            assert np.array_equal(lg[i], r0["trace"][b]["exit_logits"])
            # no block after the exit ran
            assert np.all(cnt[i][b:] == 0) and np.all(cnt[i][:b] == cnt0[i][:b])
        else:
            assert eb[i] == cfg["L"]
            assert np.array_equal(lg[i], res0[i]["logits"])
    assert 0 < n_exit < 6


def test_threshold_zero_exits_everyone_at_first_head():
    cfg = configs.get("tiny")
    W = weights.make_weights(cfg)
    imgs = images.make_images(cfg, batch=4)
    _, eb, cnt, _ = _run(cfg, W, imgs, delta=[0.0])
    assert np.all(eb == cfg["exits"][0])


def test_prune_only_after_exit_check_and_only_for_continuing():
    """At a block in both E and P an exiting sample is not pruned, and its
    logits come from the merged-but-unpruned tokens."""
    cfg = configs.get("tiny")
    W = weights.make_weights(cfg)
    imgs = images.make_images(cfg, batch=4)
    _, eb, cnt, res = _run(cfg, W, imgs, delta=[0.0])
    for r in res:
        tb = r["trace"][2]
        assert tb["exit"] and "k" not in tb
        assert len(tb["ids_after_merge"]) == tb["T"] - tb["r"]


def test_disabled_router_scaling_means_no_merge_no_prune():
    cfg = configs.get("tiny")
    W = weights.make_weights(cfg)
    imgs = images.make_images(cfg, batch=2)
    _, eb, cnt, res = _run(cfg, W, imgs, delta=[1.0], rho=0.0)
    assert np.all(cnt == cfg["N0"] + 1)


def test_token_counts_follow_merge_and_prune_counts():
    cfg = configs.get("deit_ti")
    W = weights.make_weights(cfg)
    imgs = images.make_images(cfg, batch=2)
    _, eb, cnt, res = _run(cfg, W, imgs, delta=[1.0, 1.0])
    for i, r in enumerate(res):
        T = cfg["N0"] + 1
        for b in range(1, cfg["L"] + 1):
            assert cnt[i][b - 1] == T
            tb = r["trace"][b]
            T = T - tb["r"]
            if b in cfg["prunes"]:
                assert tb["k"] == fo.keep_count(T - 1, cfg["tau"], 1.0)
                T = 1 + tb["k"]
            assert len(tb["ids"]) == T


def test_prune_scores_sum_to_one_through_merge():
    cfg = configs.get("tiny")
    W = fo.prepare_weights(weights.make_weights(cfg), "fp32")
    img = images.make_images(cfg, batch=1)[0]
    x = fo.patch_embed(img, W, cfg, "fp32")
    s = np.ones(x.shape[0], np.float32)
    origin = np.arange(x.shape[0])
    for b in range(1, cfg["L"] + 1):
        x, sc = fo.block(x, s, fo._b_weights(W, b), cfg, "fp32", want_cls=True)
        assert abs(float(sc.sum(dtype=np.float64)) - 1.0) < 1e-5
        plan = fo.merge_plan(x, 4)
        x, s, sc, origin = fo.apply_merge(x, s, sc, origin, plan["A"], plan["B"],
                                          plan["chosen"], plan["best"][plan["chosen"]])
        assert abs(float(sc.sum(dtype=np.float64)) - 1.0) < 1e-5
