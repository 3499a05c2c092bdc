"""Seeded synthetic inputs shared by the oracle, the tests and the benchmark.

This package draws random numbers and nothing else: it holds none of the
method's arithmetic (no ranking, quantization, packing or attention).
"""
from .configs import CONFIGS, WorkloadConfig, get_config
from . import synth

__all__ = ["CONFIGS", "WorkloadConfig", "get_config", "synth"]
