"""Seeded synthetic workload descriptions shared by the oracle and the HIP path.

This package holds plain data only: configuration dictionaries with the
cluster shapes, tier distributions, arrival/length distributions and seeds.
It contains none of the scheduler's arithmetic.
"""
from .presets import PRESETS, preset, scaled, with_extensions  # noqa: F401
