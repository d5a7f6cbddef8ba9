"""Seeded synthetic workloads for the DFlow round: model shapes, weights,
prompts and acceptance-forcing schedules.

This package is input generation only.  It is shared by the CPU oracle and
the GPU path and contains none of the method's arithmetic.
"""
from .configs import CONFIGS, ModelDims, Workload, get_config  # noqa: F401
