"""Per-stage GPU parity of the backbone kernels against the oracle's stage
outputs: patch embedding, attention + projection residual, MLP residual
(fusion_debug_state stops the pipeline after a stage of block 1)."""
import numpy as np
import pytest

from oracle import fusion_oracle as fo
import parity_utils as pu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def _oracle_stage(cfg, Wp, img, stage, mode):
    x = fo.patch_embed(img, Wp, cfg, mode)
    if stage == 0:
        return x
    Wb = fo._b_weights(Wp, 1)
    s = np.ones(x.shape[0], np.float32)
    if stage == 1:
        O, _ = fo.attention(x, s, Wb, cfg, mode, False)
        return x + (O @ Wb["proj_w"].T + Wb["proj_b"])
    return fo.block(x, s, Wb, cfg, mode)[0]


@pytest.mark.parametrize("name,batch,tol", [("tiny", 8, 1e-4), ("deit_ti", 6, 2e-2),
                                            ("deit_s", 4, 2e-2), ("deit_b", 2, 2e-2),
                                            ("deit_s_384", 2, 2e-2)])
@pytest.mark.parametrize("stage", [0, 1, 2])
def test_block1_stage_parity(torch_cuda, name, batch, tol, stage):
    torch = torch_cuda
    cfg, W, imgs = pu.make(name, batch=batch, affine="random")
    print(f"[stage parity] {name} B={batch} stage={stage}", flush=True)
    model = pu.gpu_model(cfg, W, batch)
    xs, live = model.debug_state(torch.from_numpy(imgs).cuda(), 1, stage)
    assert list(live) == list(range(batch))
    mode = pu.mode_of(cfg)
    Wp = fo.prepare_weights(W, mode)
    worst = 0.0
    for i in range(batch):
        ref = _oracle_stage(cfg, Wp, imgs[i], stage, mode)
        assert xs[i].shape == ref.shape
        err = float(np.abs(xs[i] - ref).max())
        worst = max(worst, err)
        assert err <= tol, (i, err)
    print(f"  max |dx| = {worst:.3e}")
