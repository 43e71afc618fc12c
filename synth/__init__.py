"""Seeded synthetic inputs shared by the oracle, the tests and the benchmark.

This package only draws numbers: model weights, initial noise, observation
tokens and their autoregressive evolution.  It contains none of the method's
arithmetic (no layers, no solver, no adaptation operator), so the CPU oracle
and the GPU path can both consume its output without sharing any code.
"""
from .workloads import WorkloadSpec, WORKLOADS, get_pair, get_workload
from .gen import (
    weight_manifest,
    make_weights,
    make_initial_noise,
    make_observations,
    make_remap_noise,
    bf16_round,
)

__all__ = [
    "WorkloadSpec",
    "WORKLOADS",
    "get_pair",
    "get_workload",
    "weight_manifest",
    "make_weights",
    "make_initial_noise",
    "make_observations",
    "make_remap_noise",
    "bf16_round",
]
