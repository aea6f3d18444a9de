"""Python binding of the C ABI: argument marshalling only.

Every step of the pipeline runs in libfusion.so's HIP kernels; PyTorch only
provides device memory (tensors passed as data pointers) and the stream.
"""
from __future__ import annotations

import ctypes
from ctypes import byref, c_double, c_float, c_int, c_int64, c_void_p

import torch

from . import _native
from ._native import FusionInfo, FusionTrace, check


def blob_inspect(blob: bytes) -> dict:
    info = FusionInfo()
    check(_native.lib().fusion_blob_inspect(blob, len(blob), byref(info)))
    return info.as_dict()


def _stream_ptr(stream) -> int:
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def _expect(t, name, shape, dtype, device):
    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{name} must be a tensor")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if t.dtype != dtype:
        raise ValueError(f"{name} has dtype {t.dtype}, expected {dtype}")
    if t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def check_run_args(info: dict, device: torch.device, images, out=None,
                   trace=None) -> int:
    """Host-side checks of fusion_run's buffers before any launch: a
    wrong-resolution batch or an undersized output would make the kernels
    read or write past the tensors.  Returns the batch size; raises
    ValueError on any mismatch."""
    if not isinstance(images, torch.Tensor) or images.dim() != 4:
        raise ValueError("images must be a 4-d tensor [batch, channels, side, side]")
    B = int(images.shape[0])
    if B < 1:
        raise ValueError("images holds no sample")
    # (a batch above max_batch is the library's FUSION_E_CAPACITY)
    S, C = info["img"], info["in_ch"]
    _expect(images, "images", (B, C, S, S), torch.float32, device)
    if out is not None:
        if len(out) != 3:
            raise ValueError("out must be (logits, exit_block, token_counts)")
        _expect(out[0], "logits", (B, info["classes"]), torch.float32, device)
        _expect(out[1], "exit_block", (B,), torch.int32, device)
        _expect(out[2], "token_counts", (B, info["layers"]), torch.int32, device)
    if trace is not None:
        L, T0 = info["layers"], info["n0"] + 1
        spec = {"r": ((L, B), torch.int32), "m": ((L, B), torch.float32),
                "c": ((L, B), torch.float32),
                "merge_dst": ((L, B, T0), torch.int32),
                "ids": ((L, B, T0), torch.int32)}
        for k, (shape, dt) in spec.items():
            if k not in trace:
                raise ValueError(f"trace lacks '{k}'")
            _expect(trace[k], f"trace['{k}']", shape, dt, device)
    return B


class FusionModel:
    """A model created from a weight blob on the current GPU."""

    def __init__(self, blob: bytes, max_batch: int):
        if not torch.cuda.is_available():
            raise RuntimeError("FusionModel needs a HIP GPU")
        self._lib = _native.lib()
        h = c_void_p()
        check(self._lib.fusion_model_create(blob, len(blob), int(max_batch),
                                            byref(h)))
        self._h = h
        self.device = torch.device("cuda", torch.cuda.current_device())
        self.info = self.get_info()

    def get_info(self) -> dict:
        info = FusionInfo()
        check(self._lib.fusion_model_info(self._h, byref(info)))
        return info.as_dict()

    def set_exit_thresholds(self, deltas):
        arr = (c_float * len(deltas))(*[float(v) for v in deltas])
        check(self._lib.fusion_set_exit_thresholds(self._h, arr, len(deltas)))

    def set_router_strength(self, rho: float):
        check(self._lib.fusion_set_router_strength(self._h, c_double(rho)))

    def alloc_outputs(self, batch: int):
        dev = self.device
        logits = torch.empty(batch, self.info["classes"], device=dev)
        exit_block = torch.empty(batch, dtype=torch.int32, device=dev)
        counts = torch.empty(batch, self.info["layers"], dtype=torch.int32, device=dev)
        return logits, exit_block, counts

    def alloc_trace(self, batch: int) -> dict:
        L, T0 = self.info["layers"], self.info["n0"] + 1
        dev = self.device
        return dict(r=torch.full((L, batch), -1, dtype=torch.int32, device=dev),
                    m=torch.full((L, batch), -1.0, device=dev),
                    c=torch.full((L, batch), -1.0, device=dev),
                    merge_dst=torch.full((L, batch, T0), -1, dtype=torch.int32, device=dev),
                    ids=torch.full((L, batch, T0), -1, dtype=torch.int32, device=dev))

    def run(self, images: torch.Tensor, out=None, trace: dict | None = None,
            stream=None):
        """Enqueue a run; returns (logits, exit_block, token_counts)."""
        B = check_run_args(self.info, self.device, images, out, trace)
        logits, exit_block, counts = out if out is not None else self.alloc_outputs(B)
        sp = _stream_ptr(stream)
        if trace is None:
            check(self._lib.fusion_run(self._h, images.data_ptr(), B,
                                       logits.data_ptr(), exit_block.data_ptr(),
                                       counts.data_ptr(), sp))
        else:
            t = FusionTrace(*(trace[k].data_ptr() for k in
                              ("r", "m", "c", "merge_dst", "ids")))
            check(self._lib.fusion_run_traced(self._h, images.data_ptr(), B,
                                              logits.data_ptr(),
                                              exit_block.data_ptr(),
                                              counts.data_ptr(), byref(t), sp))
        return logits, exit_block, counts

    def debug_state(self, images: torch.Tensor, block: int, stage: int):
        """Packed hidden states after (block, stage); see fusion_debug_state."""
        B = check_run_args(self.info, self.device, images)
        d, T0 = self.info["d"], self.info["n0"] + 1
        x = torch.zeros(B * T0, d, device="cuda")
        cu = torch.zeros(B + 1, dtype=torch.int32, device="cuda")
        live = torch.zeros(B, dtype=torch.int32, device="cuda")
        n = c_int(0)
        check(self._lib.fusion_debug_state(self._h, images.data_ptr(), B, block,
                                           stage, x.data_ptr(), cu.data_ptr(),
                                           live.data_ptr(), byref(n),
                                           _stream_ptr(None)))
        nl = n.value
        cu_h = cu[:nl + 1].cpu().numpy()
        x_h = x[:int(cu_h[-1])].cpu().numpy()
        live_h = live[:nl].cpu().numpy()
        return [x_h[cu_h[j]:cu_h[j + 1]] for j in range(nl)], live_h

    def poison_workspace(self, stream=None):
        """Fill the floating-point workspace with NaN (race proxy)."""
        check(self._lib.fusion_debug_poison_workspace(self._h, _stream_ptr(stream)))

    # ---- measurement
    def profile_enable(self, on: bool):
        check(self._lib.fusion_profile_enable(self._h, 1 if on else 0))

    def profile_read(self) -> dict:
        out = {}
        for k in range(self._lib.fusion_profile_kinds()):
            ms, n = c_double(0), c_int64(0)
            check(self._lib.fusion_profile_read(self._h, k, byref(ms), byref(n)))
            out[self._lib.fusion_profile_kind_name(k).decode()] = (ms.value, n.value)
        return out

    def close(self):
        if getattr(self, "_h", None):
            check(self._lib.fusion_model_destroy(self._h))
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
