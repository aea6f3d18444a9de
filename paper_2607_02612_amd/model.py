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


def _dev_f32(t: torch.Tensor, name: str):
    if not (t.is_cuda and t.dtype == torch.float32 and t.is_contiguous()):
        raise ValueError(f"{name} must be a contiguous float32 GPU tensor")


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
        dev = torch.device("cuda")
        logits = torch.empty(batch, self.info["classes"], device=dev)
        exit_block = torch.empty(batch, dtype=torch.int32, device=dev)
        counts = torch.empty(batch, self.info["layers"], dtype=torch.int32, device=dev)
        return logits, exit_block, counts

    def alloc_trace(self, batch: int) -> dict:
        L, T0 = self.info["layers"], self.info["n0"] + 1
        dev = torch.device("cuda")
        return dict(r=torch.full((L, batch), -1, dtype=torch.int32, device=dev),
                    m=torch.full((L, batch), -1.0, device=dev),
                    c=torch.full((L, batch), -1.0, device=dev),
                    merge_dst=torch.full((L, batch, T0), -1, dtype=torch.int32, device=dev),
                    ids=torch.full((L, batch, T0), -1, dtype=torch.int32, device=dev))

    def run(self, images: torch.Tensor, out=None, trace: dict | None = None,
            stream=None):
        """Enqueue a run; returns (logits, exit_block, token_counts)."""
        _dev_f32(images, "images")
        B = images.shape[0]
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
        _dev_f32(images, "images")
        B = images.shape[0]
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
