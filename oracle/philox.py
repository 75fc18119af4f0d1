"""Philox4x64-10 (Salmon, Moraes, Dror and Shaw, "Parallel random numbers: as
easy as 1, 2, 3", SC'11), written out in plain Python integers.

A block maps a 256-bit counter (c0, c1, c2, c3) and a 128-bit key (k0, k1) to
four 64-bit words through ten rounds.  Each round multiplies c0 and c2 by the
two Philox multipliers, keeps the high and low halves of the 128-bit products
and xors the high halves with the other two counter words and the key; the key
is advanced by the two Weyl constants before every round but the first.

Conventions used by the simulated schedule (key = (seed, purpose)):

* purpose 1: per-mini-batch delays, counter (step, learner, mini-batch, 0)
* purpose 2: MATCHA base graph, counter (attempt, position, 0, 0)
* purpose 3: MATCHA matching activation, counter (step, matching, 0, 0)
* purpose 4: local shuffles of the MLP workload, counter (epoch, learner, position, 0)
* purpose 5: per-iteration random slow-down, counter (step, learner, 0, 0)

Pins: the all-zero block equals the published Random123 known answer, and
blocks agree with NumPy's independent ``numpy.random.Philox`` (tests).
"""

from __future__ import annotations

_MASK = (1 << 64) - 1
PHILOX_M0 = 0xD2E7470EE14C6C93
PHILOX_M1 = 0xCA5A826395121157
WEYL_0 = 0x9E3779B97F4A7C15
WEYL_1 = 0xBB67AE8584CAA73B

PURPOSE_DELAY = 1
PURPOSE_GRAPH = 2
PURPOSE_ACTIVATION = 3
PURPOSE_SHUFFLE = 4
PURPOSE_SLOWDOWN = 5


def block(counter, key, rounds: int = 10):
    """Four 64-bit output words of Philox4x64-``rounds`` for one counter."""
    c0, c1, c2, c3 = (int(x) & _MASK for x in counter)
    k0, k1 = (int(x) & _MASK for x in key)
    for r in range(rounds):
        if r > 0:
            k0 = (k0 + WEYL_0) & _MASK
            k1 = (k1 + WEYL_1) & _MASK
        prod0 = PHILOX_M0 * c0
        prod1 = PHILOX_M1 * c2
        hi0, lo0 = prod0 >> 64, prod0 & _MASK
        hi1, lo1 = prod1 >> 64, prod1 & _MASK
        c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
    return (c0, c1, c2, c3)


def word(seed: int, purpose: int, c0: int, c1: int = 0, c2: int = 0) -> int:
    """Word 0 of block(counter=(c0, c1, c2, 0), key=(seed, purpose))."""
    return block((c0, c1, c2, 0), (seed, purpose))[0]


def u01(w: int) -> float:
    """Map a 64-bit word to the open interval (0, 1): the top 52 bits plus a
    half unit, times 2**-52.  The sum needs 53 significant bits, so it is exact
    in fp64 and the result lies in [2**-53, 1 - 2**-53], never 0 or 1.  (With
    the top 53 bits the sum 2**53 - 0.5 would round to 2**53, giving u = 1.)"""
    return ((w >> 12) + 0.5) * (2.0 ** -52)


def bounded(w: int, k: int) -> int:
    """Integer in [0, k) by the multiply-shift map floor(w * k / 2**64)
    (Lemire, "Fast random integer generation in an interval", 2019, without
    the rejection step; the bias is at most k / 2**64)."""
    return (w * k) >> 64
