"""CPU oracle for Non-blocking SGD (He & Dube, arXiv 2211.00889).

TEST INFRASTRUCTURE, NOT PRODUCT.  Only the test suite, the smoke check and
the benchmark's CPU-baseline leg may import or call anything here.  The GPU
library never does, and this package imports nothing from it: the two share no
code.  Inputs come from ``synth`` (seeded generators, none of the method's
arithmetic) or from the tests themselves.

Everything is plain, slow and written to be checked against the paper by eye:
fp64 arithmetic on fp32 inputs, explicit Python loops where the paper's
algorithm has loops, NumPy only as a library primitive (a matrix product, a
sum).  Modules:

* ``philox``   - Philox4x64-10 counter-based generator (Salmon et al., SC'11),
                 the random source of the simulated straggler delays and of
                 MATCHA's graph and activations.
* ``schedule`` - per-mini-batch delays, the terminal signal (deadline) and the
                 finished-mini-batch mask (Alg. 2, mini-batch loop; Lemma 1).
* ``mixing``   - mixing matrices: uniform (ring all-reduce, Eq. 4-5), ring
                 gossip (D-PSGD, Eq. 6) and MATCHA random matchings (Sec. 6.1).
* ``step``     - one Non-blocking step: accumulate finished mini-batches,
                 learning-rate scaling, momentum, mix and update (Alg. 2;
                 Sec. 3.2 bullets).
* ``mlp``      - the end-to-end two-layer MLP workload: forward/backward
                 per mini-batch, local shuffling (Alg. 1 initialisation),
                 training under any mixing kind.
* ``workload`` - drivers: a workload description mapped to the oracle's delay
                 model, mixing matrices and order; column windows of the
                 seeded inputs; several iterations of the step.

Parity pins for each function live in ``tests/test_oracle_*.py``; functions
with no pin say "parity unpinned" in their docstring.
"""

from . import mixing, mlp, philox, schedule, step, workload  # noqa: F401
