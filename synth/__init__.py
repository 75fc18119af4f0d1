"""Seeded synthetic inputs shared by the GPU path's tests and the oracle.

This package generates input arrays only (parameter replicas, per-mini-batch
gradients, the synthetic classification data of the MLP workload).  It holds
none of the method's arithmetic: no delays, masks, mixing matrices, gradient
accumulation or updates live here.

Every value is a pure function of (seed, stream, flat element index) through a
SplitMix64 counter (Steele, Lea and Flood, "Fast splittable pseudorandom number
generators", OOPSLA 2014) followed by integer-only shaping and one correctly
rounded fp32 multiply, so the NumPy generator in ``gen`` and the HIP fill kernel
in ``fill.hip`` produce bit-identical fp32 arrays, and any column window of a
tensor can be regenerated on the host without touching the device.
"""

from .gen import (  # noqa: F401
    NORMAL_STD_UNIT,
    normal_f32,
    normal_scale,
    splitmix_key,
    splitmix_words,
    uniform_f32,
    uniform_scale,
)
