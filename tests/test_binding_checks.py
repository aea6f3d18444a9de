"""Host-side argument checks of the Python binding (CPU): fusion_run's
buffers are validated before any launch, so a wrong-resolution batch or an
undersized output raises ValueError instead of reaching the kernels."""
import pytest
import torch

from paper_2607_02612_amd.model import check_run_args

INFO = dict(img=32, in_ch=3, classes=10, layers=4, n0=64, max_batch=8)
DEV = torch.device("cpu")


def _ok(B=4):
    images = torch.zeros(B, 3, 32, 32)
    out = (torch.zeros(B, 10), torch.zeros(B, dtype=torch.int32),
           torch.zeros(B, 4, dtype=torch.int32))
    trace = dict(r=torch.zeros(4, B, dtype=torch.int32), m=torch.zeros(4, B),
                 c=torch.zeros(4, B), merge_dst=torch.zeros(4, B, 65, dtype=torch.int32),
                 ids=torch.zeros(4, B, 65, dtype=torch.int32))
    return images, out, trace


def test_valid_arguments_pass():
    images, out, trace = _ok()
    assert check_run_args(INFO, DEV, images, out, trace) == 4
    assert check_run_args(INFO, DEV, images) == 4


@pytest.mark.parametrize("images", [
    torch.zeros(4, 3, 64, 64),                 # wrong resolution
    torch.zeros(4, 1, 32, 32),                 # wrong channel count
    torch.zeros(4, 3, 32, 32, dtype=torch.float16),
    torch.zeros(4, 3, 32, 64)[:, :, :, :32],   # not contiguous
    torch.zeros(3, 32, 32),                    # not a batch
    torch.zeros(0, 3, 32, 32),                 # empty batch
])
def test_bad_images_rejected(images):
    with pytest.raises(ValueError):
        check_run_args(INFO, DEV, images)


@pytest.mark.parametrize("k,bad", [
    (0, torch.zeros(3, 10)), (0, torch.zeros(4, 9)), (0, torch.zeros(4, 10, dtype=torch.float64)),
    (1, torch.zeros(4, dtype=torch.int64)), (1, torch.zeros(3, dtype=torch.int32)),
    (2, torch.zeros(4, 3, dtype=torch.int32)), (2, torch.zeros(4, 4)),
])
def test_bad_outputs_rejected(k, bad):
    images, out, _ = _ok()
    out = list(out)
    out[k] = bad
    with pytest.raises(ValueError):
        check_run_args(INFO, DEV, images, tuple(out))


@pytest.mark.parametrize("key,bad", [
    ("r", torch.zeros(4, 3, dtype=torch.int32)), ("m", torch.zeros(4, 4, dtype=torch.int32)),
    ("c", torch.zeros(3, 4)), ("merge_dst", torch.zeros(4, 4, 64, dtype=torch.int32)),
    ("ids", torch.zeros(4, 4, 65)),
])
def test_bad_trace_rejected(key, bad):
    images, out, trace = _ok()
    trace[key] = bad
    with pytest.raises(ValueError):
        check_run_args(INFO, DEV, images, out, trace)


def test_missing_trace_entry_and_wrong_device_rejected():
    images, out, trace = _ok()
    del trace["ids"]
    with pytest.raises(ValueError):
        check_run_args(INFO, DEV, images, out, trace)
    with pytest.raises(ValueError):
        check_run_args(INFO, torch.device("meta"), images)
