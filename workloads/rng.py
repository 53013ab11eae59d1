"""Counter-based random numbers (numpy), one of three independent implementations.

Definition (shared as a *specification*, not as code):

    key(stream, a, b) = stream << 58 | a << 24 | b     (stream < 64, a < 2^34, b < 2^24)
    x = seed XOR key
    z = x + 0x9E3779B97F4A7C15                          (mod 2^64)
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9
    z = (z ^ (z >> 27)) * 0x94D049BB133111EB
    out = z ^ (z >> 31)                                 (the SplitMix64 output of
                                                         Steele, Lea & Flood 2014)
    u32 = out >> 32

With seed XOR key = s, `out` is exactly the first value the published
SplitMix64 generator returns when seeded with s.

Streams: 0 Bernoulli graph pair (a=source, b=target), 1 fixed-fan-out target
(a=source, b=draw), 2 initial membrane potential (a=0, b=neuron), 3 external
Poisson drive (a=step, b=neuron), 4 Bernoulli source spikes (a=step, b=neuron).
The HIP library and the C oracle each implement the same definition on their
own; this module serves the input generators only.
"""

import numpy as np

STREAM_GRAPH_PAIR = 0
STREAM_FANOUT = 1
STREAM_INIT_V = 2
STREAM_POISSON = 3
STREAM_SPIKE = 4

_GAMMA = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)


def splitmix64_mix(x):
    """SplitMix64 output for state `x` (numpy uint64 array or scalar)."""
    x = np.asarray(x, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z = x + _GAMMA
        z = (z ^ (z >> np.uint64(30))) * _M1
        z = (z ^ (z >> np.uint64(27))) * _M2
    return z ^ (z >> np.uint64(31))


def rng_key(stream, a, b):
    a = np.asarray(a, dtype=np.uint64)
    b = np.asarray(b, dtype=np.uint64)
    if np.any(a >= np.uint64(1 << 34)) or np.any(b >= np.uint64(1 << 24)):
        raise ValueError("rng key field out of range (a < 2^34, b < 2^24)")
    if not 0 <= stream < 64:
        raise ValueError("stream must be in [0, 64)")
    return (np.uint64(stream) << np.uint64(58)) | (a << np.uint64(24)) | b


def rng_u64(seed, stream, a, b):
    return splitmix64_mix(np.uint64(seed) ^ rng_key(stream, a, b))


def rng_u32(seed, stream, a, b):
    return (rng_u64(seed, stream, a, b) >> np.uint64(32)).astype(np.uint32)
