"""Python binding of the kernel-level entry points (fusion_test_* in
include/fusion.h): argument marshalling only.  Tensors are passed as device
pointers; the per-sample row offsets and merge counts are host arrays.

Each function runs one step of the pipeline with the library's HIP kernels
on caller-supplied packed ragged buffers and returns device tensors.
"""
from __future__ import annotations

import ctypes
from ctypes import byref, c_double, c_float

import numpy as np
import torch

from . import _native
from ._native import FusionPackedOut, FusionRagged, check

EPI = {"store": 0, "gelu": 1, "resid": 2, "f32": 3}


def _ptr(t):
    return None if t is None else t.data_ptr()


def _host_i32(a):
    a = np.ascontiguousarray(np.asarray(a, dtype=np.int32))
    return a, a.ctypes.data_as(ctypes.c_void_p)


def _stream():
    return torch.cuda.current_stream().cuda_stream


def _need(t, name, dtype):
    if not (isinstance(t, torch.Tensor) and t.is_cuda and t.dtype == dtype and t.is_contiguous()):
        raise ValueError(f"{name} must be a contiguous {dtype} GPU tensor")


def gemm(A, W, bias, epi, out, rows=None):
    """out <- epi(A W^T + bias).  A [M, K], W [N, K]: both bfloat16 (bf16
    path) or both float32; bias float32 [N]; out in the storage type
    (store / gelu) or float32 (resid / f32)."""
    prec = {torch.bfloat16: 1, torch.float32: 0}[A.dtype]
    _need(A, "A", A.dtype)
    _need(W, "W", A.dtype)
    _need(bias, "bias", torch.float32)
    _need(out, "out", out.dtype)
    if rows is not None:
        _need(rows, "rows", torch.int32)
    M, K = A.shape
    N = W.shape[0]
    if W.shape[1] != K or bias.shape[0] != N or out.shape[1] < N:
        raise ValueError("operand shapes do not match")
    if rows is None and out.shape[0] < M:
        raise ValueError("out has fewer rows than A")
    check(_native.lib().fusion_test_gemm(prec, A.data_ptr(), K, W.data_ptr(), N, K, M,
                                         bias.data_ptr(), EPI[epi], out.data_ptr(),
                                         out.shape[1], _ptr(rows), _stream()))
    return out


def attention(qkv, size, cu, heads, prop_attn=True, cls_tmax=None):
    """Per-sample MHSA over packed rows; returns (out [M, d] like qkv,
    cls_scores [B, heads, tmax] float32 or None)."""
    prec = {torch.bfloat16: 1, torch.float32: 0}[qkv.dtype]
    _need(qkv, "qkv", qkv.dtype)
    _need(size, "size", torch.float32)
    cu_h, cu_p = _host_i32(cu)
    B = len(cu_h) - 1
    M, d3 = qkv.shape
    if M != cu_h[-1] or size.shape[0] != M:
        raise ValueError("rows do not match the offsets")
    d = d3 // 3
    out = torch.zeros(M, d, dtype=qkv.dtype, device=qkv.device)
    cls = None
    if cls_tmax is not None:
        cls = torch.full((B, heads, cls_tmax), -1.0, device=qkv.device)
    check(_native.lib().fusion_test_attention(prec, qkv.data_ptr(), size.data_ptr(), cu_p, B,
                                              heads, d, int(bool(prop_attn)), out.data_ptr(),
                                              _ptr(cls), cls_tmax or 0, _stream()))
    return out, cls


def _ragged(x, size, origin, cu):
    _need(x, "x", torch.float32)
    _need(size, "size", torch.float32)
    _need(origin, "origin", torch.int32)
    cu_h, cu_p = _host_i32(cu)
    if x.shape[0] != cu_h[-1] or size.shape[0] != x.shape[0] or origin.shape[0] != x.shape[0]:
        raise ValueError("rows do not match the offsets")
    rg = FusionRagged(x.data_ptr(), size.data_ptr(), origin.data_ptr(), cu_p,
                      len(cu_h) - 1, x.shape[1])
    return rg, cu_h


def _packed(M, B, dev):
    o = dict(rows=torch.full((M,), -1, dtype=torch.int32, device=dev),
             size=torch.full((M,), -1.0, device=dev),
             origin=torch.full((M,), -1, dtype=torch.int32, device=dev),
             cu=torch.full((B + 1,), -1, dtype=torch.int32, device=dev),
             live=torch.full((B,), -1, dtype=torch.int32, device=dev),
             counts=torch.full((2,), -1, dtype=torch.int32, device=dev))
    po = FusionPackedOut(*(o[k].data_ptr() for k in ("rows", "size", "origin", "cu", "live",
                                                     "counts")))
    return o, po


def merge(x, size, origin, cu, r, id_stride, noalloc=False):
    """Bipartite merge of r[i] pairs per sample (x updated in place); returns
    (packed output dict, merge_dst [B, id_stride] int32).  noalloc: the
    variant whose scratch is the library's static device array."""
    rg, cu_h = _ragged(x, size, origin, cu)
    B = len(cu_h) - 1
    r_h, r_p = _host_i32(r)
    if len(r_h) != B:
        raise ValueError("one merge count per sample")
    o, po = _packed(x.shape[0], B, x.device)
    md = torch.full((B, id_stride), -1, dtype=torch.int32, device=x.device)
    fn = _native.lib().fusion_test_merge_noalloc if noalloc else _native.lib().fusion_test_merge
    check(fn(byref(rg), r_p, id_stride, md.data_ptr(), byref(po), _stream()))
    return o, md


def topk_compact(x, size, origin, cu, keep_ratio, scores=None, heads=1, prune_w=None,
                 prune_b=None, exit_logits=None, delta=1.0, ln=None, precision=1):
    """Exit check (optional), top-k prune and re-compaction; returns (packed
    output dict, logits, exit_block, ln_out)."""
    rg, cu_h = _ragged(x, size, origin, cu)
    B, M, d = len(cu_h) - 1, x.shape[0], x.shape[1]
    dev = x.device
    tmax = 0
    if scores is not None:
        _need(scores, "scores", torch.float32)
        if scores.shape[0] != B or scores.shape[1] != heads:
            raise ValueError("scores must be [batch, heads, tmax]")
        tmax = scores.shape[2]
    C = 0
    logits = exit_block = None
    if exit_logits is not None:
        _need(exit_logits, "exit_logits", torch.float32)
        C = exit_logits.shape[1]
        logits = torch.full((B, C), -7.0, device=dev)
        exit_block = torch.full((B,), -1, dtype=torch.int32, device=dev)
    ln_out = None
    ln_g = ln_b = None
    if ln is not None:
        ln_g, ln_b = ln
        ln_out = torch.zeros(M, d, dtype=torch.bfloat16 if precision == 1 else torch.float32,
                             device=dev)
    o, po = _packed(M, B, dev)
    check(_native.lib().fusion_test_topk_compact(
        byref(rg), _ptr(scores), heads, tmax, _ptr(prune_w), _ptr(prune_b), c_double(keep_ratio),
        _ptr(exit_logits), C, c_float(delta), _ptr(logits), _ptr(exit_block), precision,
        _ptr(ln_g), _ptr(ln_b), _ptr(ln_out), byref(po), _stream()))
    return o, logits, exit_block, ln_out
