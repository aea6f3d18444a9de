"""Seeded synthetic inputs shared by the CPU oracle's tests and the GPU path.

Holds only data generation (workload definitions, weights, images) and the
weight-blob writer; none of the method's arithmetic lives here.
"""
from . import configs, weights, images, blob  # noqa: F401
