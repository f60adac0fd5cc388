"""Workload definitions and seeded input generators.

This package holds the five synthetic workload shapes and the seeded random
draws that feed both the GPU library and the CPU oracle.  It contains none of
the method's arithmetic (no encoding, no NTT, no modular products): moduli
that a draw needs are passed in by the caller.
"""
from .configs import CONFIGS, Config, get  # noqa: F401
