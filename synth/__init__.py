"""Seeded synthetic workloads for the selective-upsampling step (inputs only)."""
from . import configs, generator  # noqa: F401
from .configs import Workload, keep_count  # noqa: F401
