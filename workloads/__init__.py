"""Seeded synthetic workloads for the StateKV per-frame video-prefill step.

This package holds the workload shapes and the deterministic input generators.
It contains none of the method's arithmetic (no attention, scoring or
selection): it only produces the Q/K/V bytes that both the CPU oracle and the
GPU library consume, so the two sides see identical inputs.
"""
from .configs import CONFIGS, WorkloadConfig, get_config  # noqa: F401
