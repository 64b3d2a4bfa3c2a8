"""Seeded synthetic workloads for the EasyBalance hot path.

Shared by the CPU oracle and the GPU path; holds input generation only
(shapes, seeds, distributions), none of the method's arithmetic.
"""
from .configs import CONFIGS, BY_NAME, Config, mini  # noqa: F401
