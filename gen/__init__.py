"""Seeded synthetic trace generators shared by the oracle tests, the GPU tests and the bench.

This package holds no arithmetic of the period-detection method: it only draws
piecewise-constant periodic power / utilisation / counter traces with noise,
spikes and per-repeat length jitter, in the shapes of the five workloads
(see ``gen.traces``).
"""
from .traces import (  # noqa: F401
    Workload,
    make_workload,
    planted_trace,
    WORKLOADS,
)
