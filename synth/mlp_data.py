"""Synthetic data of the end-to-end MLP workload (CIFAR-shaped stand-in).

* inputs:  50,000 samples of 3072 values, approximately N(0, 1) (the generator
           of ``gen``), row-major [sample][feature].
* labels:  argmax (lowest index on ties) of a fixed random teacher network of
           the same architecture: weights N(0, 2 / fan_in), zero biases,
           computed once in fp64 on the host.  This is input generation; the
           trained network never sees the teacher.
* initial replica: the student's parameters, identical on every learner
           (Alg. 1/2 initialise all local models the same), weights and biases
           uniform on +-1/sqrt(fan_in), in the flat layout W1, b1, W2, b2.

CIFAR-10 itself is not available; these arrays have its shape (3072 inputs, 10
classes, 50,000 training samples).
"""

from __future__ import annotations

import math
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

from .gen import normal_f32, uniform_f32

N_SAMPLES = 50_000
D_IN, HIDDEN, CLASSES, BATCH = 3072, 512, 10, 32

STREAM_DATA = 10
STREAM_TEACHER_W1 = 11
STREAM_TEACHER_W2 = 12
STREAM_INIT = 13


def _threads():
    return max(1, min(16, len(os.sched_getaffinity(0))))


def inputs(seed: int, n_samples: int = N_SAMPLES, d_in: int = D_IN) -> np.ndarray:
    """[n_samples, d_in] fp32, generated in row chunks on several threads
    (NumPy's elementwise kernels release the GIL)."""
    out = np.empty((n_samples, d_in), dtype=np.float32)
    rows = max(1, (1 << 22) // d_in)

    def job(r0):
        r1 = min(n_samples, r0 + rows)
        idx = np.arange(r0 * d_in, r1 * d_in, dtype=np.int64)
        out[r0:r1] = normal_f32(seed, STREAM_DATA, idx, 1.0).reshape(r1 - r0, d_in)

    with ThreadPoolExecutor(_threads()) as ex:
        list(ex.map(job, range(0, n_samples, rows)))
    return out


def teacher_labels(seed: int, A: np.ndarray, hidden: int = HIDDEN, classes: int = CLASSES) -> np.ndarray:
    d_in = A.shape[1]
    W1 = normal_f32(seed, STREAM_TEACHER_W1, np.arange(d_in * hidden), math.sqrt(2.0 / d_in))
    W2 = normal_f32(seed, STREAM_TEACHER_W2, np.arange(hidden * classes), math.sqrt(2.0 / hidden))
    W1 = W1.reshape(d_in, hidden).astype(np.float64)
    W2 = W2.reshape(hidden, classes).astype(np.float64)
    labels = np.empty(A.shape[0], dtype=np.int32)
    step = 4096
    for r0 in range(0, A.shape[0], step):
        H = np.maximum(A[r0:r0 + step].astype(np.float64) @ W1, 0.0)
        labels[r0:r0 + step] = np.argmax(H @ W2, axis=1)
    return labels


def student_init(seed: int, d_in: int = D_IN, hidden: int = HIDDEN, classes: int = CLASSES) -> np.ndarray:
    """Flat fp32 parameters [W1, b1, W2, b2]."""
    a1, a2 = 1.0 / math.sqrt(d_in), 1.0 / math.sqrt(hidden)
    sizes = [(d_in * hidden, a1), (hidden, a1), (hidden * classes, a2), (classes, a2)]
    parts, start = [], 0
    for count, a in sizes:
        parts.append(uniform_f32(seed, STREAM_INIT, np.arange(start, start + count), a))
        start += count
    return np.concatenate(parts)
