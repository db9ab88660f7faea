"""Seeded synthetic inputs shared by the oracle side and the HIP side.

``values``  counter-based gradient values (host twin of the HIP generator)
``recipe``  workload shapes and per-unit, per-step scale streams
``layout``  placing a workload's units as segments of one device buffer
``gpu``     the HIP generator library (loaded on demand)

This package holds none of the controller's arithmetic.
"""
from . import recipe, values  # noqa: F401
