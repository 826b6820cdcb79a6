"""Seeded synthetic workloads (shapes, region spans, keys, queries).

Shared by the CPU oracle and the device path; draws numbers only.
"""
from . import configs, generator  # noqa: F401
