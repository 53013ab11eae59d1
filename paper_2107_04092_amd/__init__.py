"""MI355X (gfx950) synapse pass of a clock-based SNN simulator.

Lazy + event-driven STDP over 64-bit firing histories and slice delivery with
LDS atomics, after Bautembach, Oikonomidis & Argyros, "Even Faster SNN
Simulation with Lazy+Event-driven Plasticity and Shared Atomics". The compute
path is the HIP library libsnn.so (C ABI in include/snn.h); `snn` is its thin
ctypes binding.
"""

from . import snn  # noqa: F401
