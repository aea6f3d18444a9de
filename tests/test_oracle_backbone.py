"""Pins for the oracle's backbone (patch embed, blocks, heads) and rounding.

The plain ViT special case (threshold 1, router strength 0: no merge, no
exit, no prune) is checked against an independent forward pass built from
torch.nn.functional library routines (conv2d patch embedding, layer_norm,
multi_head_attention_forward, gelu, linear), so a dropped term, a wrong
patch order or a transposed weight in the oracle fails here.
"""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from oracle import fusion_oracle as fo
from synth import configs, images, weights


def _torch_vit(img, W, cfg, need_cls_attn=False):
    """fp32 DeiT-style forward from torch.nn.functional routines."""
    d, H, p = cfg["d"], cfg["H"], cfg["patch"]
    t = lambda a: torch.from_numpy(np.asarray(a, dtype=np.float32))
    x = torch.from_numpy(img)[None]
    pe = F.conv2d(x, t(W["pe_w"]).reshape(d, cfg["in_ch"], p, p), t(W["pe_b"]),
                  stride=p)
    tok = pe.flatten(2).transpose(1, 2)[0]               # [N0, d] raster order
    z = torch.cat([t(W["cls"])[None], tok], 0) + t(W["pos"])
    cls_attn = []
    for b in range(1, cfg["L"] + 1):
        g = lambda n: t(W[f"blk{b}.{n}"])
        h = F.layer_norm(z, (d,), g("ln1_g"), g("ln1_b"), eps=1e-6)[:, None, :]
        o, aw = F.multi_head_attention_forward(
            h, h, h, d, H, g("qkv_w"), g("qkv_b"), None, None, False, 0.0,
            g("proj_w"), g("proj_b"), training=False, need_weights=True,
            average_attn_weights=True)
        cls_attn.append(aw[0, 0].numpy())
        z = z + o[:, 0, :]
        h = F.layer_norm(z, (d,), g("ln2_g"), g("ln2_b"), eps=1e-6)
        z = z + F.linear(F.gelu(F.linear(h, g("fc1_w"), g("fc1_b"))),
                         g("fc2_w"), g("fc2_b"))
    y = F.layer_norm(z[0], (d,), t(W["norm_g"]), t(W["norm_b"]), eps=1e-6)
    out = F.linear(y, t(W["head_w"]), t(W["head_b"])).numpy()
    return (out, cls_attn) if need_cls_attn else out


@pytest.mark.parametrize("name,nimg", [("tiny", 3), ("deit_ti", 1)])
def test_plain_vit_matches_torch_functional(name, nimg):
    cfg = configs.get(name)
    W = weights.make_weights(cfg, affine="random")
    imgs = images.make_images(cfg, batch=nimg)
    Wp = fo.prepare_weights(W, "fp32")
    for i in range(nimg):
        ref = _torch_vit(imgs[i], W, cfg)
        got = fo.plain_forward(imgs[i], Wp, cfg, "fp32")
        np.testing.assert_allclose(got, ref, rtol=1e-5, atol=2e-5)


@pytest.mark.parametrize("name", ["tiny", "deit_ti"])
@pytest.mark.parametrize("mode", ["fp32", "bf16emu"])
def test_disabled_adaptation_is_plain_vit_bit_exact(name, mode):
    """delta = 1 and rho = 0 turn every adaptive step into an exact no-op."""
    cfg = configs.get(name)
    W = weights.make_weights(cfg, affine="random")
    img = images.make_images(cfg, batch=1)
    delta = [1.0] * len(cfg["exits"])
    lg, eb, cnt, _ = oracle.run(img, W, cfg, mode, delta=delta, rho=0.0)
    plain = fo.plain_forward(img[0], fo.prepare_weights(W, mode), cfg, mode)
    assert np.array_equal(lg[0], plain)
    assert eb[0] == cfg["L"]
    assert np.all(cnt[0] == cfg["N0"] + 1)


def test_cls_attention_matches_library_head_mean():
    """The prune score (head-mean CLS attention, unit sizes) equals the
    head-averaged attention weights torch returns."""
    cfg = configs.get("tiny")
    W = weights.make_weights(cfg, affine="random")
    img = images.make_images(cfg, batch=1)[0]
    _, ref_attn = _torch_vit(img, W, cfg, need_cls_attn=True)
    Wp = fo.prepare_weights(W, "fp32")
    x = fo.patch_embed(img, Wp, cfg, "fp32")
    s = np.ones(x.shape[0], np.float32)
    for b in range(1, cfg["L"] + 1):
        x, a = fo.block(x, s, fo._b_weights(Wp, b), cfg, "fp32", want_cls=True)
        np.testing.assert_allclose(a, ref_attn[b - 1], rtol=1e-5, atol=1e-7)
        assert abs(float(a.sum()) - 1.0) < 1e-5


def test_bf16_round_matches_torch_cast():
    rng = np.random.default_rng(0)
    a = np.concatenate([
        rng.standard_normal(100000).astype(np.float32) * 10.0,
        rng.standard_normal(1000).astype(np.float32) * 1e-38,   # subnormals
        np.array([0.0, -0.0, 1.0, 3.0e38, -3.0e38, np.inf, -np.inf],
                 dtype=np.float32)])
    # exact ties: bf16 value + half an ulp, both parities
    base = fo.bf16_round(rng.standard_normal(1000).astype(np.float32))
    ties = (base.view(np.uint32) | 0x8000).view(np.float32)
    a = np.concatenate([a, ties])
    ref = torch.from_numpy(a).to(torch.bfloat16).to(torch.float32).numpy()
    got = fo.bf16_round(a)
    assert np.array_equal(got.view(np.uint32), ref.view(np.uint32))


def test_layer_norm_and_gelu_match_library():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((7, 384)).astype(np.float32) * 3 + 1
    g = rng.uniform(0.5, 1.5, 384).astype(np.float32)
    b = rng.standard_normal(384).astype(np.float32)
    ref = F.layer_norm(torch.from_numpy(x), (384,), torch.from_numpy(g),
                       torch.from_numpy(b), eps=1e-6).numpy()
    np.testing.assert_allclose(fo.layer_norm(x, g, b), ref, rtol=1e-5, atol=1e-5)
    ref_g = F.gelu(torch.from_numpy(x)).numpy()
    np.testing.assert_allclose(fo.gelu(x), ref_g, rtol=1e-6, atol=1e-6)


def test_patchify_is_conv_order():
    cfg = configs.get("tiny")
    img = images.make_images(cfg, batch=1)[0]
    P = fo.patchify(img, cfg["patch"])
    p, g = cfg["patch"], cfg["grid"]
    # patch (gy, gx) raster index gy*g+gx; element (c, ky, kx)
    gy, gx, c, ky, kx = 3, 5, 2, 1, 3
    assert P[gy * g + gx, c * p * p + ky * p + kx] == img[c, gy * p + ky, gx * p + kx]


def test_max_softmax_matches_scipy():
    from scipy.special import softmax
    rng = np.random.default_rng(2)
    for _ in range(20):
        l = (rng.standard_normal(1000) * 5).astype(np.float32)
        assert abs(float(fo.max_softmax(l)) - softmax(l.astype(np.float64)).max()) < 1e-6


def test_bf16emu_rounds_stored_operands():
    """In bf16emu every stored matrix-product operand is bf16-representable,
    while the fp32 residual stream is not rounded."""
    cfg = configs.get("deit_ti")
    W = fo.prepare_weights(weights.make_weights(cfg, affine="random"), "bf16emu")
    for k in ("pe_w", "blk1.qkv_w", "blk1.fc2_w", "blk4.ew", "head_w"):
        assert np.array_equal(W[k], fo.bf16_round(W[k]))
    assert not np.array_equal(W["pos"], fo.bf16_round(W["pos"]))
    img = images.make_images(cfg, batch=1)[0]
    x32 = fo.patch_embed(img, fo.prepare_weights(weights.make_weights(cfg), "fp32"), cfg, "fp32")
    x16 = fo.patch_embed(img, W, cfg, "bf16emu")
    assert x32.shape == x16.shape
    # rounding changes the result by about one bf16 ulp of the operands
    Wf = fo.prepare_weights(weights.make_weights(cfg, affine="random"), "fp32")
    d = np.abs(fo.patch_embed(img, Wf, cfg, "fp32") - x16).max()
    assert 1e-5 < d < 5e-2


def test_bf16_contract_amplifies_summation_order_noise():
    """The fp32 path is insensitive to the accumulation order of the matrix
    products, while the bf16 rounding points turn that order into a visible
    logit drift: this is the floor the bf16 parity tolerance is derived
    from (tests/golden/noise_floor.json)."""
    import json
    import os
    cfg = configs.get("deit_ti")
    W = weights.make_weights(cfg)
    img = images.make_images(cfg, batch=1)[0]
    d = {}
    for mode in ("fp32", "bf16emu"):
        Wp = fo.prepare_weights(W, mode)
        a = fo.plain_forward(img, Wp, cfg, mode)
        with fo.accumulate("fp64"):
            b = fo.plain_forward(img, Wp, cfg, mode)
        d[mode] = float(np.abs(a - b).max())
    assert d["fp32"] < 1e-4
    assert d["bf16emu"] > 5e-3
    with open(os.path.join(os.path.dirname(__file__), "golden", "noise_floor.json")) as f:
        floor = {w["workload"]: w for w in json.load(f)["workloads"]}
    assert d["bf16emu"] <= floor["deit_ti"]["max_dlogit"] * 1.5
