"""Seeded synthetic inputs shared by the CPU oracle and the device path.

Holds configurations and random draws only; none of the method's arithmetic.
"""
from . import configs, gen  # noqa: F401
from .configs import MoEConfig, CONFIGS, get  # noqa: F401
