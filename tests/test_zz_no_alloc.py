"""fusion_test_merge_noalloc (scratch in the library's static device array,
no allocation) against fusion_test_merge (scratch allocated per call): the
same kernels on the same inputs must give bit-identical results, on two
calls in a row where the second is smaller (stale scratch contents of the
first call must not leak into the second)."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu


def _case(rng, lengths, d):
    cu = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int32)
    M = int(cu[-1])
    basis = rng.standard_normal((8, d))
    x = (rng.standard_normal((M, 8)) @ basis + 0.4 * rng.standard_normal((M, d))).astype(np.float32)
    size = rng.integers(1, 4, size=M).astype(np.float32)
    origin = np.concatenate([np.arange(T) for T in lengths]).astype(np.int32)
    r = np.array([(T - 1) // 2 if i % 3 else (T - 1) // 4 for i, T in enumerate(lengths)],
                 dtype=np.int32)
    return x, size, origin, cu, r


def test_merge_noalloc_equals_allocating_merge_on_two_calls():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_02612_amd import kernels
    rng = np.random.default_rng(2024)
    calls = [([197] * 64 + [100, 1, 2], 384),     # about 0.2 MiB of scratch
             ([1, 2, 17, 130, 5], 384)]           # smaller second call
    for lengths, d in calls:
        print(f"[noalloc] samples={len(lengths)} rows={sum(lengths)}", flush=True)
        x, size, origin, cu, r = _case(rng, lengths, d)
        T_ = lambda a: torch.from_numpy(a.copy()).cuda()
        xa, xb = T_(x), T_(x)
        oa, ma = kernels.merge(xa, T_(size), T_(origin), cu, r, max(lengths))
        ob, mb = kernels.merge(xb, T_(size), T_(origin), cu, r, max(lengths), noalloc=True)
        torch.cuda.synchronize()
        for k in oa:
            assert torch.equal(oa[k], ob[k]), k
        assert torch.equal(ma, mb)
        assert torch.equal(xa, xb)
        n = int(oa["counts"][0])
        assert n == len(lengths) and int(oa["counts"][1]) == int(cu[-1] - r.sum())


def test_merge_noalloc_capacity_error():
    """A call needing more than the static array is refused with
    FUSION_E_CAPACITY before anything is launched."""
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_02612_amd import FusionError, kernels
    lengths = [197] * 600                 # 118 200 rows: about 1.4 MiB of scratch
    cu = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int32)
    M = int(cu[-1])
    x = torch.zeros(M, 64, device="cuda")
    with pytest.raises(FusionError) as ei:
        kernels.merge(x, torch.ones(M, device="cuda"), torch.zeros(M, dtype=torch.int32, device="cuda"),
                      cu, np.zeros(len(lengths), np.int32), 197, noalloc=True)
    assert ei.value.code == -3
