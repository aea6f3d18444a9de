"""Race proxy: no output of a run may depend on workspace state the run did
not write itself.  The model's floating-point workspace is filled with NaN
between two runs of the same batch; logits, exit blocks and token counts
must stay bit-identical (a stale read would turn them into NaN or change a
decision).  Covered on the headline workload and on the 384 x 384 workload
(long samples, chunked attention, the largest adapt size class), on the
timed (untraced) path and on the traced path."""
import numpy as np
import pytest

import parity_utils as pu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


@pytest.mark.parametrize("name,e,rho", [("deit_s", 0.5, 1.0), ("deit_s_384", 0.5, 1.0),
                                        ("deit_s_paper", None, 5.0 / 3.0)])
def test_nan_poisoned_workspace_gives_identical_outputs(torch_cuda, name, e, rho):
    torch = torch_cuda
    cfg, W, imgs = pu.make(name)
    if e is None:
        delta = [0.7, 0.9]
    else:
        d = pu.exit_thresholds(name, rho)[e]
        delta = [d, d]
    print(f"[race proxy] {name} batch {cfg['batch']} delta={delta} rho={rho:.4f}", flush=True)
    m = pu.gpu_model(cfg, W, cfg["batch"])
    x = torch.from_numpy(imgs).cuda()
    for traced in (False, True):
        ref = pu.gpu_run(m, x, delta=delta, rho=rho, traced=traced)
        assert np.isfinite(ref["logits"]).all()
        m.poison_workspace()
        got = pu.gpu_run(m, x, delta=delta, rho=rho, traced=traced)
        for k in ("logits", "exit_block", "counts"):
            assert np.array_equal(ref[k], got[k]), (traced, k)
        if traced:
            for k in ref["trace"]:
                assert np.array_equal(ref["trace"][k], got["trace"][k]), k
