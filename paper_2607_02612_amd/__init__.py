"""MI355X (gfx950) implementation of Fusion's staged adaptive ViT inference.

The compute lives in libfusion.so (HIP kernels behind the C ABI declared in
include/fusion.h); this package only loads it and marshals arguments.
"""
from ._native import FusionError, LIB_PATH  # noqa: F401


def __getattr__(name):
    if name in ("FusionModel", "blob_inspect"):
        from . import model
        return getattr(model, name)
    raise AttributeError(name)
