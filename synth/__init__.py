"""Seeded synthetic workloads for the large-sparse-target output layer.

This package only draws random inputs (initial V and U, minibatches of hidden
representations H and K-sparse targets). It contains none of the method's
arithmetic, so both the fp64 oracle and the GPU library can consume its arrays.
"""
from .workloads import (  # noqa: F401
    CONFIGS,
    Workload,
    WorkloadConfig,
    bounded_zipf_sampler,
    get_config,
)
