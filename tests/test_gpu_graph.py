"""The whole forward captured as one HIP graph (how the benchmark times a
step): every replay gives the eager result bit for bit, with eager runs of
another batch and host synchronisations between the replays.  The forward
launches kernels only (no allocation, copy, memset or host wait between
them), and the exit thresholds and the router strength are kernel
arguments, fixed at capture."""
import pytest

import parity_utils as pu

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("workload,delta", [("deit_ti", 0.5), ("deit_s", 0.9)])
def test_graph_replays_match_eager(workload, delta):
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    cfg, W, imgs = pu.make(workload, affine="random", router_std=0.2)
    B = cfg["batch"]
    print(f"[graph] {workload} batch={B} delta={delta}", flush=True)
    m = pu.gpu_model(cfg, W, B)
    m.set_exit_thresholds([delta] * len(cfg["exits"]))
    xa = torch.from_numpy(imgs).cuda()
    xb = torch.flip(xa, dims=[0]).contiguous()  # a second batch: the same images reversed
    ref_a = [t.clone() for t in m.run(xa)]
    ref_b = [t.clone() for t in m.run(xb)]
    torch.cuda.synchronize()
    n_exit = int((ref_a[1] < cfg["L"]).sum())
    print(f"  eager: early exits {n_exit}/{B}", flush=True)

    out = m.alloc_outputs(B)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        m.run(xa, out=out)
    for rep in range(3):
        for t in out:
            t.zero_()
        g.replay()
        torch.cuda.synchronize()
        for name, t, r in zip(("logits", "exit_block", "token_counts"), out, ref_a):
            assert torch.equal(t, r), f"replay {rep}: {name} differs from the eager run"
        ob = m.run(xb)
        torch.cuda.synchronize()
        for name, t, r in zip(("logits", "exit_block", "token_counts"), ob, ref_b):
            assert torch.equal(t, r), f"eager run after replay {rep}: {name} differs"
    del g
    m.close()
