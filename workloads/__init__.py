"""Seeded synthetic inputs shared by the GPU path's tests/bench and the CPU oracle.

This package holds only input generation: model presets (physical
parameters and sizes of the paper's benchmark networks), the counter-based
random generator used to draw initial membrane potentials, and the uint32
inverse-CDF table for the external Poisson drive. It holds none of the
method's arithmetic (no neuron update, plasticity or delivery).
"""

from .rng import splitmix64_mix, rng_u64, rng_u32, STREAM_GRAPH_PAIR, \
    STREAM_FANOUT, STREAM_INIT_V, STREAM_POISSON, STREAM_SPIKE
from .presets import Preset, PRESETS, preset, initial_state, poisson_cdf_table

__all__ = [
    "splitmix64_mix", "rng_u64", "rng_u32",
    "STREAM_GRAPH_PAIR", "STREAM_FANOUT", "STREAM_INIT_V", "STREAM_POISSON",
    "STREAM_SPIKE", "Preset", "PRESETS", "preset", "initial_state",
    "poisson_cdf_table",
]
