"""Seeded synthetic inputs shared by the oracle, the tests and the benchmark.

This package holds workload descriptions (shapes, sizes, distributions) and
random-number draws only.  It contains none of the training or aggregation
arithmetic: the oracle and the HIP library each implement that on their own.
"""
from .configs import CONFIGS, ConfigSpec, get_config, param_layout, param_count
from .gen import (
    init_params,
    make_acts,
    make_labels,
    make_lengths,
    make_local_vectors,
    make_global_vector,
    make_staleness,
    make_arrival_rates,
    make_arrival_counts,
    bf16_bits_from_f32,
    f32_from_bf16_bits,
    rng_for,
)

__all__ = [
    "CONFIGS", "ConfigSpec", "get_config", "param_layout", "param_count",
    "init_params", "make_acts", "make_labels", "make_lengths",
    "make_local_vectors", "make_global_vector", "make_staleness", "make_arrival_rates",
    "make_arrival_counts", "bf16_bits_from_f32", "f32_from_bf16_bits", "rng_for",
]
