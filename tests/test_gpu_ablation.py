"""GPU parity of the Tab. VII compositions (Sec. IV-F, Ablation Study):
single mechanisms (pruning only, merging only, early exit only), parallel
composition (pruning at blocks every sample reaches before the first exit
head), sequential exit -> prune, and the full sequential pipeline with fixed
merges, merge routers and profile scaling.  Each composition runs on one
superset weight draw, every sample is compared with the oracle (decisions
and logits, the same rules as the other parity tests), and the executed
FLOPs reduction against the dense backbone is printed beside the result
(the only Tab. VII column that synthetic weights can reproduce).
"""
import numpy as np
import pytest

from oracle import fusion_oracle as fo
from synth import configs, images, weights
import parity_utils as pu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def _dense_flops(cfg):
    d, mlp, C, L, T = cfg["d"], cfg["mlp"], cfg["C"], cfg["L"], cfg["N0"] + 1
    blk = 8 * T * d * d + 4 * T * d * mlp + 4 * T * T * d
    return L * blk + 2 * cfg["N0"] * cfg["patch_dim"] * d + 2 * d * C


def _flops_reduction(cfg, res):
    f = [fo.executed_flops(cfg, res["counts"][i], res["exit_block"][i])
         for i in range(len(res["exit_block"]))]
    return 1.0 - float(np.mean(f)) / _dense_flops(cfg)


def _settings(base, cfg, prof):
    """(delta, rho) of a profile: the Tab. I thresholds at DeiT-S; on the
    tiny shape the workload's own thresholds (lowered by 0.1 / 0.05 for
    power_save), with the profile's router strength."""
    st = configs.profile_settings(prof)
    if base == "tiny_paper" and cfg["exits"]:
        dl = tuple(configs.CONFIGS["tiny_paper"]["delta"])
        if prof == "power_save":
            dl = (dl[0] - 0.1, dl[1] - 0.05)
        delta = dl[:len(cfg["exits"])]
    else:
        delta = tuple(st["delta"][:len(cfg["exits"])])
    return (list(delta) if cfg["exits"] else None), st["rho"]


def _run_row(torch, base, rows, superset, name, batch=None):
    sup = configs.get(base, prunes=superset)
    W = weights.make_weights(sup)
    over, prof = next((o, p) for n, o, p in rows if n == name)
    cfg = configs.ablation_config(base, over)
    Wc = weights.zero_routers(cfg, W) if cfg["merge_rule"] == "budget" and cfg["merges"] else W
    imgs = images.make_images(sup, batch=batch)
    delta, rho = _settings(base, cfg, prof)
    print(f"[{base} ablation] {name}: M={cfg['merges']} E={cfg['exits']} "
          f"P={cfg['prunes']} delta={delta} rho={rho:.4f}", flush=True)
    m = pu.gpu_model(cfg, Wc, imgs.shape[0])
    res = pu.gpu_run(m, torch.from_numpy(imgs).cuda(), delta=delta, rho=rho)
    worst, adopted = pu.check_samples(cfg, Wc, imgs, res, range(imgs.shape[0]),
                                      delta=delta, rho=rho)
    red = _flops_reduction(cfg, res)
    exits = {int(b): int(c) for b, c in zip(*np.unique(res["exit_block"], return_counts=True))}
    print(f"  samples={imgs.shape[0]} max|dlogit|={worst:.3e} adoptions={len(adopted)} "
          f"FLOPs reduction={100 * red:.1f}% exit blocks={exits}", flush=True)
    pu.adoption_report(f"{base} {name}", adopted, imgs.shape[0])
    return cfg, res, red


@pytest.mark.parametrize("name", [n for n, _, _ in configs.ABLATION_TINY])
def test_tiny_paper_compositions_fp32(torch_cuda, name):
    cfg, res, red = _run_row(torch_cuda, "tiny_paper", configs.ABLATION_TINY,
                             configs.ABLATION_TINY_SUPERSET_PRUNES, name)
    if name == "plain":
        assert red == pytest.approx(0.0, abs=1e-12)
    if name == "parallel prune + exit":
        # pruning reaches every sample before the first exit head
        assert np.all(res["counts"][:, 1] < cfg["N0"] + 1)


@pytest.mark.parametrize("name", [n for n, _, _ in configs.ABLATION])
def test_deit_s_paper_compositions_bf16(torch_cuda, name):
    cfg, res, red = _run_row(torch_cuda, "deit_s_paper", configs.ABLATION,
                             configs.ABLATION_SUPERSET_PRUNES, name)
    if name == "plain":
        assert red == pytest.approx(0.0, abs=1e-12)
    if name == "parallel prune + exit":
        assert np.all(res["counts"][:, 7] < cfg["N0"] + 1)
