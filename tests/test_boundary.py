"""C-ABI boundary checks that need no GPU: the library loads, exports every
declared entry point, and rejects malformed blobs and arguments on the host
with the documented status codes."""
import ctypes
import os
import re
import struct

import numpy as np
import pytest

from paper_2607_02612_amd import _native
from paper_2607_02612_amd.model import blob_inspect
from synth import blob, configs, weights

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    with open(os.path.join(ROOT, "include", "fusion.h")) as f:
        txt = f.read()
    return re.findall(r"FUSION_API\s+[\w\s\*]+?\b(fusion_\w+)\s*\(", txt)


def test_library_exports_every_declared_symbol():
    lib = _native.lib()
    names = _declared()
    assert len(names) >= 12
    for n in names:
        assert hasattr(lib, n), n
    assert {n for n, _, _ in _native.SIGNATURES} == set(names)


@pytest.fixture(scope="module")
def tiny_blob():
    cfg = configs.get("tiny")
    return cfg, blob.pack(cfg, weights.make_weights(cfg))


def test_blob_inspect_reads_header(tiny_blob):
    cfg, b = tiny_blob
    info = blob_inspect(b)
    assert info["d"] == cfg["d"] and info["layers"] == cfg["L"]
    assert info["n0"] == cfg["N0"] and info["classes"] == cfg["C"]
    assert info["exit_blocks"] == list(cfg["exits"])
    assert info["precision"] == 0
    assert info["r_b"] == list(cfg["r_b"])
    assert info["delta"] == pytest.approx(list(cfg["delta"]))
    cfg3 = configs.get("deit_s")
    info3 = blob_inspect(blob.pack(cfg3, weights.make_weights(cfg3)))
    assert info3["precision"] == 1 and info3["exit_blocks"] == [4, 8]
    assert info3["tau_b"][3] == 0.7 and info3["tau_b"][0] == 1.0


def _expect(code, b):
    lib = _native.lib()
    info = _native.FusionInfo()
    rc = lib.fusion_blob_inspect(b, len(b), ctypes.byref(info))
    assert rc == code, (rc, lib.fusion_last_error())
    assert lib.fusion_last_error().decode() != ""
    return lib.fusion_last_error().decode()


def test_corrupt_blobs_are_rejected(tiny_blob):
    cfg, b = tiny_blob
    E = -2
    _expect(E, b"\0" * 10)
    _expect(E, b"XXXXXXXX" + b[8:])                       # magic
    _expect(E, b[:8] + struct.pack("<I", 7) + b[12:])     # version
    _expect(E, b[:1000])                                   # truncated data
    # a tensor shape that disagrees with the header
    d_off = 16 + 4 * 3
    bad = bytearray(b)
    bad[d_off:d_off + 4] = struct.pack("<I", cfg["d"] * 2)
    assert "shape" in _expect(E, bytes(bad))
    # exit mask naming a block beyond L
    bad = bytearray(b)
    bad[60:64] = struct.pack("<I", 1 << 20)
    _expect(E, bytes(bad))
    # keep ratio outside [0, 1]
    bad = bytearray(b)
    bad[196:204] = struct.pack("<d", 1.5)
    _expect(E, bytes(bad))
    # tensor name out of order
    bad = bytearray(b)
    nm = blob.HEADER_BYTES
    bad[nm:nm + 3] = b"xyz"
    assert "expected tensor" in _expect(E, bytes(bad))


def test_create_rejects_bad_arguments_before_touching_device(tiny_blob):
    cfg, b = tiny_blob
    lib = _native.lib()
    h = ctypes.c_void_p()
    assert lib.fusion_model_create(b, len(b), 0, ctypes.byref(h)) == -1
    assert lib.fusion_model_create(b, len(b), 1 << 20, ctypes.byref(h)) == -1
    assert lib.fusion_model_create(b"junk" * 200, 800, 4, ctypes.byref(h)) == -2
    assert lib.fusion_model_create(None, 0, 4, ctypes.byref(h)) == -1
    assert lib.fusion_model_create(b, len(b), 4, None) == -1
    assert lib.fusion_model_destroy(None) == -1
    assert lib.fusion_set_router_strength(None, 1.0) == -1
    assert lib.fusion_run(None, None, 1, None, None, None, None) == -1


def test_bf16_shape_limits_are_checked():
    cfg = configs.get("deit_ti", mlp=700)   # not a multiple of 64
    b = blob.pack(cfg, weights.make_weights(cfg))
    assert "multiples of 64" in _expect(-2, b)


def test_profile_kind_names():
    lib = _native.lib()
    n = lib.fusion_profile_kinds()
    names = [lib.fusion_profile_kind_name(k).decode() for k in range(n)]
    assert "attention" in names and "adapt" in names and len(set(names)) == n


def test_blob_inspect_reads_paper_rules():
    cfg = configs.get("deit_s_paper")
    b = blob.pack(cfg, weights.make_weights(cfg))
    info = blob_inspect(b)
    assert info["merge_rule"] == 1 and info["prune_rule"] == 1
    assert info["exit_hidden"] == 768
    assert info["exit_kind"][7] == 2 and info["exit_kind"][9] == 1
    assert info["exit_blocks"] == [8, 10]
    assert info["delta"] == pytest.approx([0.8, 0.95])
    # an exit-head kind on a block that has no exit head
    bad = bytearray(b)
    bad[588:592] = struct.pack("<I", 1)
    assert "exit-head kind" in _expect(-2, bytes(bad))
    # hidden width that the bf16 GEMMs cannot tile
    bad = bytearray(b)
    bad[716:720] = struct.pack("<I", 700)
    assert "hidden width" in _expect(-2, bytes(bad))
    # unknown rules
    for off in (580, 584):
        bad = bytearray(b)
        bad[off:off + 4] = struct.pack("<I", 5)
        assert "rule" in _expect(-2, bytes(bad))


def _ragged_args(cu, d=64):
    cu = np.asarray(cu, dtype=np.int32)
    rg = _native.FusionRagged(8, 8, 8, cu.ctypes.data_as(ctypes.c_void_p), len(cu) - 1, d)
    po = _native.FusionPackedOut(8, 8, 8, 8, 8, 8)
    return cu, rg, po


@pytest.mark.parametrize("cu,r,d", [
    ([1, 5], [0], 64),            # offsets must start at 0
    ([0, 0], [0], 64),            # empty sample
    ([0, 641], [0], 64),          # more than 640 rows
    ([0, 5, 3], [0, 0], 64),      # decreasing offsets
    ([0, 5], [3], 64),            # r > floor(N/2)
    ([0, 5], [-1], 64),           # negative r
    ([0, 5], [1], 48),            # width not a multiple of 32
    ([0, 5], [1], 800),           # width beyond 768
])
def test_kernel_level_merge_rejects_bad_arguments_on_host(cu, r, d):
    """fusion_test_merge validates offsets, counts and width before any
    device call (the pointers here are never dereferenced)."""
    lib = _native.lib()
    cu, rg, po = _ragged_args(cu, d)
    r = np.asarray(r, dtype=np.int32)
    rc = lib.fusion_test_merge(ctypes.byref(rg), r.ctypes.data_as(ctypes.c_void_p), 8, None,
                               ctypes.byref(po), None)
    assert rc == -1, lib.fusion_last_error()
    assert lib.fusion_last_error().decode() != ""


def test_kernel_level_entry_points_reject_bad_arguments_on_host():
    lib = _native.lib()
    # GEMM: unknown precision / epilogue, bf16 K not a multiple of 32, row
    # map with a bf16 store epilogue
    assert lib.fusion_test_gemm(2, 8, 64, 8, 64, 64, 4, 8, 0, 8, 64, None, None) == -1
    assert lib.fusion_test_gemm(1, 8, 64, 8, 64, 64, 4, 8, 7, 8, 64, None, None) == -1
    assert lib.fusion_test_gemm(1, 8, 48, 8, 64, 48, 4, 8, 0, 8, 64, None, None) == -1
    assert lib.fusion_test_gemm(1, 8, 64, 8, 64, 64, 4, 8, 0, 8, 64, 8, None) == -1
    assert lib.fusion_test_gemm(1, None, 64, 8, 64, 64, 4, 8, 0, 8, 64, None, None) == -1
    # attention: bf16 needs 64-wide heads; tmax below the longest sample
    cu = np.array([0, 3, 10], dtype=np.int32)
    cp = cu.ctypes.data_as(ctypes.c_void_p)
    assert lib.fusion_test_attention(1, 8, 8, cp, 2, 4, 128, 1, 8, None, 0, None) == -1
    assert lib.fusion_test_attention(1, 8, 8, cp, 2, 2, 128, 1, 8, 8, 5, None) == -1
    # top-k: no score source, keep ratio outside [0, 1], exit without outputs
    cu, rg, po = _ragged_args([0, 4, 9])
    br = ctypes.byref
    assert lib.fusion_test_topk_compact(br(rg), None, 1, 9, None, None, 0.5, None, 0, 1.0,
                                        None, None, 1, None, None, None, br(po), None) == -1
    assert lib.fusion_test_topk_compact(br(rg), 8, 1, 9, None, None, 1.5, None, 0, 1.0,
                                        None, None, 1, None, None, None, br(po), None) == -1
    assert lib.fusion_test_topk_compact(br(rg), 8, 1, 9, None, None, 0.5, 8, 10, 0.5,
                                        None, None, 1, None, None, None, br(po), None) == -1
    assert lib.fusion_test_topk_compact(br(rg), 8, 1, 4, None, None, 0.5, None, 0, 1.0,
                                        None, None, 1, None, None, None, br(po), None) == -1


def test_noalloc_merge_refuses_oversized_calls_on_host():
    """fusion_test_merge_noalloc returns FUSION_E_CAPACITY when a call would
    need more scratch than the static array holds, before any device call."""
    lib = _native.lib()
    cu, rg, po = _ragged_args(np.arange(0, 197 * 700 + 1, 197))
    r = np.zeros(700, dtype=np.int32)
    rc = lib.fusion_test_merge_noalloc(ctypes.byref(rg), r.ctypes.data_as(ctypes.c_void_p), 197,
                                       None, ctypes.byref(po), None)
    assert rc == -3, lib.fusion_last_error()
    assert "scratch" in lib.fusion_last_error().decode()
