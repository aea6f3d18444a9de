"""Whole-pipeline properties of the oracle and of the shared generators."""
import numpy as np
import pytest

import oracle
from oracle import fusion_oracle as fo
from synth import blob, configs, images, weights


def _mode(cfg):
    return "fp32" if cfg["precision"] == "fp32" else "bf16emu"


def test_generators_are_deterministic_and_batch_independent():
    cfg = configs.get("deit_ti")
    a = images.make_images(cfg, batch=4)
    b = images.make_images(cfg, batch=2, first=2)
    assert np.array_equal(a[2:], b)
    w1 = weights.make_weights(cfg)
    w2 = weights.make_weights(cfg)
    assert all(np.array_equal(w1[k], w2[k]) for k in w1)
    assert blob.pack(cfg, w1) == blob.pack(cfg, w2)


def test_image_statistics_follow_recipe():
    cfg = configs.get("deit_s")
    x = images.make_images(cfg, batch=8)
    assert x.shape == (8, 3, 224, 224) and x.dtype == np.float32
    # three sinusoids of amplitude <= 1 plus noise of sigma <= 1
    assert np.abs(x).max() < 3 + 6
    assert 0.2 < x.std() < 2.5


def test_batch_permutation_and_sample_alone():
    cfg = configs.get("tiny")
    W = weights.make_weights(cfg)
    imgs = images.make_images(cfg, batch=5)
    lg, eb, cnt, _ = oracle.run(imgs, W, cfg, "fp32")
    perm = np.array([3, 0, 4, 1, 2])
    lg2, eb2, cnt2, _ = oracle.run(imgs[perm], W, cfg, "fp32")
    assert np.array_equal(lg2, lg[perm]) and np.array_equal(eb2, eb[perm])
    assert np.array_equal(cnt2, cnt[perm])
    lg3, eb3, cnt3, _ = oracle.run(imgs[2:3], W, cfg, "fp32")
    assert np.array_equal(lg3[0], lg[2]) and np.array_equal(cnt3[0], cnt[2])


def _follow_from(res, cfg):
    out = []
    for r in res:
        f = {}
        for b, tb in r["trace"].items():
            f[b] = dict(r=tb.get("r", 0), merge=tb.get("merge", {}),
                        exit=tb.get("exit", False),
                        ids=tb.get("ids", tb.get("ids_after_merge")))
        out.append(f)
    return out


def test_follow_mode_accepts_own_decisions_without_adoption():
    cfg = configs.get("deit_ti")
    W = weights.make_weights(cfg)
    imgs = images.make_images(cfg, batch=2)
    lg, eb, cnt, res = oracle.run(imgs, W, cfg, "bf16emu")
    lg2, eb2, cnt2, res2 = oracle.run(imgs, W, cfg, "bf16emu",
                                      follow=_follow_from(res, cfg))
    assert np.array_equal(lg, lg2) and np.array_equal(eb, eb2)
    assert all(len(r["adopted"]) == 0 for r in res2)


def test_follow_mode_rejects_decision_outside_margin():
    cfg = configs.get("tiny")
    W = weights.make_weights(cfg)
    imgs = images.make_images(cfg, batch=1)
    _, _, _, res = oracle.run(imgs, W, cfg, "fp32", delta=[1.0])
    f = _follow_from(res, cfg)
    # replace a merge source by the A token with the lowest best similarity
    tb = res[0]["trace"][1]
    x = fo.patch_embed(imgs[0], fo.prepare_weights(W, "fp32"), cfg, "fp32")
    xb, _ = fo.block(x, np.ones(x.shape[0], np.float32),
                     fo._b_weights(fo.prepare_weights(W, "fp32"), 1), cfg, "fp32")
    plan = fo.merge_plan(xb, tb["r"])
    worst = int(np.argmin(plan["bestsim"]))
    src = 1 + plan["A"][worst]
    bad = dict(tb["merge"])
    bad.pop(next(iter(bad)))
    bad[src] = 1 + plan["B"][plan["best"][worst]]
    f[0][1]["merge"] = bad
    with pytest.raises(fo.DecisionMismatch):
        oracle.run(imgs, W, cfg, "fp32", delta=[1.0], follow=f)
    # an exit decision far from the threshold cannot be overridden either
    f = _follow_from(res, cfg)
    f[0][2]["exit"] = True
    with pytest.raises(fo.DecisionMismatch):
        oracle.run(imgs, W, cfg, "fp32", delta=[1.0], follow=f)


def test_executed_flops_closed_form_deit_s():
    """24 T d^2 + 4 T^2 d per block; 197 tokens, 12 blocks, no reduction."""
    cfg = configs.get("deit_s")
    cnt = np.full(12, 197)
    f = fo.executed_flops(cfg, cnt, 12)
    dense = 12 * (24 * 197 * 384 ** 2 + 4 * 197 ** 2 * 384) \
        + 2 * 196 * 768 * 384 + 2 * 384 * 1000 * 3
    assert f == dense
    assert abs(f / 1e9 - 9.197) < 0.01
