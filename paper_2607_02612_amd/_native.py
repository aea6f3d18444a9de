"""ctypes declarations of libfusion.so (the C ABI in include/fusion.h)."""
from __future__ import annotations

import ctypes
import os
from ctypes import (POINTER, c_char_p, c_double, c_float, c_int, c_int32,
                    c_int64, c_size_t, c_uint32, c_void_p)

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)),
                        "libfusion.so")
MAX_LAYERS = 32

STATUS = {0: "FUSION_OK", -1: "FUSION_E_INVALID_ARG", -2: "FUSION_E_BLOB",
          -3: "FUSION_E_CAPACITY", -4: "FUSION_E_OOM", -5: "FUSION_E_HIP",
          -6: "FUSION_E_STATE"}


class FusionInfo(ctypes.Structure):
    _fields_ = [("img", c_int32), ("patch", c_int32), ("in_ch", c_int32),
                ("d", c_int32), ("heads", c_int32), ("layers", c_int32),
                ("mlp", c_int32), ("classes", c_int32), ("n0", c_int32),
                ("precision", c_int32), ("prop_attn", c_int32),
                ("max_batch", c_int32), ("merge_mask", c_uint32),
                ("exit_mask", c_uint32), ("prune_mask", c_uint32),
                ("n_exit", c_int32), ("exit_blocks", c_int32 * MAX_LAYERS),
                ("r_b", c_int32 * MAX_LAYERS), ("tau_b", c_double * MAX_LAYERS),
                ("delta", c_float * MAX_LAYERS), ("rho", c_double),
                ("merge_rule", c_int32), ("prune_rule", c_int32),
                ("exit_kind", c_int32 * MAX_LAYERS), ("exit_hidden", c_int32)]

    def as_dict(self) -> dict:
        out = {}
        for name, _ in self._fields_:
            v = getattr(self, name)
            out[name] = list(v) if hasattr(v, "__len__") else v
        L = out["layers"]
        out["exit_blocks"] = out["exit_blocks"][:out["n_exit"]]
        out["delta"] = out["delta"][:out["n_exit"]]
        out["r_b"] = out["r_b"][:L]
        out["tau_b"] = out["tau_b"][:L]
        out["exit_kind"] = out["exit_kind"][:L]
        return out


class FusionTrace(ctypes.Structure):
    _fields_ = [("r", c_void_p), ("m", c_void_p), ("c", c_void_p),
                ("merge_dst", c_void_p), ("ids", c_void_p)]


class FusionRagged(ctypes.Structure):
    _fields_ = [("x", c_void_p), ("size", c_void_p), ("origin", c_void_p),
                ("cu", c_void_p), ("batch", c_int32), ("d", c_int32)]


class FusionPackedOut(ctypes.Structure):
    _fields_ = [("rows", c_void_p), ("size", c_void_p), ("origin", c_void_p),
                ("cu", c_void_p), ("live", c_void_p), ("counts", c_void_p)]


class FusionError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{STATUS.get(code, code)}: {msg}")
        self.code = code


# every exported entry point: (name, restype, argtypes)
SIGNATURES = [
    ("fusion_blob_inspect", c_int, [c_char_p, c_size_t, POINTER(FusionInfo)]),
    ("fusion_model_create", c_int, [c_char_p, c_size_t, c_int, POINTER(c_void_p)]),
    ("fusion_model_destroy", c_int, [c_void_p]),
    ("fusion_model_info", c_int, [c_void_p, POINTER(FusionInfo)]),
    ("fusion_set_exit_thresholds", c_int, [c_void_p, POINTER(c_float), c_int]),
    ("fusion_set_router_strength", c_int, [c_void_p, c_double]),
    ("fusion_run", c_int, [c_void_p, c_void_p, c_int, c_void_p, c_void_p,
                           c_void_p, c_void_p]),
    ("fusion_run_traced", c_int, [c_void_p, c_void_p, c_int, c_void_p,
                                  c_void_p, c_void_p, POINTER(FusionTrace),
                                  c_void_p]),
    ("fusion_debug_state", c_int, [c_void_p, c_void_p, c_int, c_int, c_int,
                                   c_void_p, c_void_p, c_void_p,
                                   POINTER(c_int), c_void_p]),
    ("fusion_debug_poison_workspace", c_int, [c_void_p, c_void_p]),
    ("fusion_profile_enable", c_int, [c_void_p, c_int]),
    ("fusion_profile_kinds", c_int, []),
    ("fusion_profile_kind_name", c_char_p, [c_int]),
    ("fusion_profile_read", c_int, [c_void_p, c_int, POINTER(c_double),
                                    POINTER(c_int64)]),
    ("fusion_test_gemm", c_int, [c_int, c_void_p, c_int, c_void_p, c_int, c_int,
                                 c_int, c_void_p, c_int, c_void_p, c_int, c_void_p,
                                 c_void_p]),
    ("fusion_test_attention", c_int, [c_int, c_void_p, c_void_p, c_void_p, c_int,
                                      c_int, c_int, c_int, c_void_p, c_void_p, c_int,
                                      c_void_p]),
    ("fusion_test_merge", c_int, [POINTER(FusionRagged), c_void_p, c_int, c_void_p,
                                  POINTER(FusionPackedOut), c_void_p]),
    ("fusion_test_merge_noalloc", c_int, [POINTER(FusionRagged), c_void_p, c_int, c_void_p,
                                          POINTER(FusionPackedOut), c_void_p]),
    ("fusion_test_topk_compact", c_int, [POINTER(FusionRagged), c_void_p, c_int, c_int,
                                         c_void_p, c_void_p, c_double, c_void_p, c_int,
                                         c_float, c_void_p, c_void_p, c_int, c_void_p,
                                         c_void_p, c_void_p, POINTER(FusionPackedOut),
                                         c_void_p]),
    ("fusion_last_error", c_char_p, []),
]

_LIB = None


def lib():
    """Load libfusion.so (built in-tree); raises if it has not been built."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is missing: build it with "
                "`python -m paper_2607_02612_amd.build` (hipcc, gfx950)")
        L = ctypes.CDLL(LIB_PATH)
        for name, res, args in SIGNATURES:
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _LIB = L
    return _LIB


def check(rc: int):
    if rc != 0:
        raise FusionError(rc, lib().fusion_last_error().decode())
