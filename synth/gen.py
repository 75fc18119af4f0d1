"""NumPy side of the synthetic-input generator (bit-identical to ``fill.hip``).

Definition (shared, word for word, with the HIP kernel):

* ``fmix(z)``: the SplitMix64 output function
  ``z ^= z >> 30; z *= 0xBF58476D1CE4E5B9; z ^= z >> 27; z *= 0x94D049BB133111EB;
  z ^= z >> 31`` (all arithmetic mod 2**64).
* ``GAMMA = 0x9E3779B97F4A7C15`` (the SplitMix64 increment).
* stream key: ``key(seed, stream) = fmix(fmix(seed + GAMMA) + (stream + 1) * GAMMA)``.
* word of element ``e``: ``w(e) = fmix(key + (e + 1) * GAMMA)``, i.e. the e-th
  output of a SplitMix64 generator whose state starts at ``key``.
* approximately normal value: the four 16-bit fields of ``w`` summed (an
  Irwin-Hall sum of four discrete uniforms), centred by subtracting
  ``2 * 65535``, converted exactly to fp32 (|s| < 2**24) and multiplied in fp32
  by ``scale = fp32(std / sqrt((65536**2 - 1) / 3))``.  Mean 0, standard
  deviation ``std``, support +-3.46 std.
* uniform value on [-a, a): ``(w >> 40) - 2**23`` (exact in fp32) times
  ``scale = fp32(a / 2**23)``.

A single IEEE fp32 multiply of exact operands is correctly rounded on both the
host and gfx950, so the arrays agree bit for bit.
"""

from __future__ import annotations

import math

import numpy as np

_M64 = (1 << 64) - 1
GAMMA = 0x9E3779B97F4A7C15
_C1 = 0xBF58476D1CE4E5B9
_C2 = 0x94D049BB133111EB

# standard deviation of the centred sum of four uniform 16-bit integers
NORMAL_STD_UNIT = math.sqrt((65536.0 * 65536.0 - 1.0) / 3.0)


def _fmix_int(z: int) -> int:
    z &= _M64
    z ^= z >> 30
    z = (z * _C1) & _M64
    z ^= z >> 27
    z = (z * _C2) & _M64
    z ^= z >> 31
    return z


def splitmix_key(seed: int, stream: int) -> int:
    """Per-tensor key; ``stream`` separates tensors drawn from one seed."""
    k0 = _fmix_int((seed + GAMMA) & _M64)
    return _fmix_int((k0 + ((stream + 1) * GAMMA)) & _M64)


def _fmix_np(z: np.ndarray) -> np.ndarray:
    z = z ^ (z >> np.uint64(30))
    z = z * np.uint64(_C1)
    z = z ^ (z >> np.uint64(27))
    z = z * np.uint64(_C2)
    z = z ^ (z >> np.uint64(31))
    return z


def splitmix_words(seed: int, stream: int, index) -> np.ndarray:
    """64-bit words ``w(e)`` for the flat element indices ``index`` (array-like)."""
    e = np.asarray(index, dtype=np.uint64)
    key = np.uint64(splitmix_key(seed, stream))
    with np.errstate(over="ignore"):
        z = key + (e + np.uint64(1)) * np.uint64(GAMMA)
        return _fmix_np(z)


def normal_scale(std: float) -> np.float32:
    return np.float32(std / NORMAL_STD_UNIT)


def uniform_scale(half_width: float) -> np.float32:
    return np.float32(half_width / 8388608.0)


def normal_f32(seed: int, stream: int, index, std: float) -> np.ndarray:
    """Approximately N(0, std**2) fp32 values at flat indices ``index``."""
    w = splitmix_words(seed, stream, index)
    m16 = np.uint64(0xFFFF)
    s = ((w & m16) + ((w >> np.uint64(16)) & m16)
         + ((w >> np.uint64(32)) & m16) + (w >> np.uint64(48)))
    centred = s.astype(np.int64) - 131070
    return centred.astype(np.float32) * normal_scale(std)


def uniform_f32(seed: int, stream: int, index, half_width: float) -> np.ndarray:
    """Uniform fp32 values on [-half_width, half_width) at flat indices ``index``."""
    w = splitmix_words(seed, stream, index)
    centred = (w >> np.uint64(40)).astype(np.int64) - 8388608
    return centred.astype(np.float32) * uniform_scale(half_width)


def window_index(rows: int, P: int, c0: int, c1: int) -> np.ndarray:
    """Flat indices of columns [c0, c1) of every row of a row-major [rows, P] tensor."""
    r = np.arange(rows, dtype=np.int64)[:, None] * P
    c = np.arange(c0, c1, dtype=np.int64)[None, :]
    return (r + c).reshape(-1)
