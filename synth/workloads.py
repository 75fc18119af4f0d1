"""The synthetic workloads: shapes, input distributions, delay models, mixing
kinds and hyper-parameters.  Plain data; both the GPU-path tests/bench and the
oracle read it, and each side maps the names to its own constants.

The paper trains CNNs on CIFAR-10/100 (Sec. 6.1); neither the datasets nor the
networks are available here, so flat parameter vectors sized like ResNet-18,
ResNet-50 and VGG-16 with Gaussian per-mini-batch gradients stand in for them.
Values never change the memory traffic of a step: the only data-dependent
control flow is the finished-mini-batch mask.
"""

from __future__ import annotations

import math
from dataclasses import dataclass, field, replace

# tensor streams of the input generator
STREAM_X = 1
STREAM_G = 2

MIX_THEN_STEP = "mix_then_step"
STEP_THEN_MIX = "step_then_mix"


@dataclass(frozen=True)
class DelaySpec:
    kind: str = "exp"          # "const" | "exp" | "lomax"
    base: float = 1.0
    param: float = 1.0         # exp: rate; lomax: shape
    slow_learner: int = -1     # -1: none; -2: random per iteration
    slow_factor: float = 1.0
    slow_prob: float = 0.0     # random slow-down only


@dataclass(frozen=True)
class Workload:
    name: str
    n: int
    m: int
    P: int
    mixing: str                # "uniform" | "ring" | "matcha"
    order: str
    delay: DelaySpec
    lr: float
    momentum: float
    steps: int
    seed: int = 0
    x_std: float = 1.0
    g_std: float = math.sqrt(1e-3)   # N(0, 1e-3) read as variance 1e-3
    matcha_degree: int = 3
    matcha_budget: float | None = None   # set: MATCHA's optimised p and alpha under this budget
    notes: str = ""
    extra: dict = field(default_factory=dict)

    def with_P(self, P: int) -> "Workload":
        return replace(self, P=P)

    def alg_bytes(self, sum_counts: int) -> int:
        """Algorithmic HBM bytes of one fused step: the finished gradient rows
        once, X and V read once and written once."""
        return 4 * self.P * (sum_counts + 4 * self.n)


TINY = Workload("tiny_n4_m4_P10k_allreduce", 4, 4, 10_000, "uniform", STEP_THEN_MIX,
                DelaySpec("exp", 1.0, 1.0), 0.1, 0.9, 10)
RESNET18_RING = Workload("resnet18_n8_m8_P11.2M_ring", 8, 8, 11_200_000, "ring", MIX_THEN_STEP,
                         DelaySpec("exp", 1.0, 1.0, slow_learner=7, slow_factor=3.0), 0.1, 0.9, 50)
RESNET50_MATCHA = Workload("resnet50_n16_m4_P23.5M_matcha", 16, 4, 23_500_000, "matcha",
                           MIX_THEN_STEP, DelaySpec("exp", 1.0, 0.5), 0.1, 0.9, 50)
VGG16_ALLREDUCE = Workload("vgg16_n8_m16_P138M_allreduce", 8, 16, 138_000_000, "uniform",
                           STEP_THEN_MIX, DelaySpec("lomax", 1.0, 1.5), 0.05, 0.9, 20)

RESNET50_MATCHA_OPT = replace(RESNET50_MATCHA, name="resnet50_n16_m4_P23.5M_matcha_optimised",
                              matcha_budget=0.5)

WORKLOADS = {w.name: w for w in (TINY, RESNET18_RING, RESNET50_MATCHA, VGG16_ALLREDUCE,
                                 RESNET50_MATCHA_OPT)}
ALIASES = {"tiny": TINY.name, "resnet18": RESNET18_RING.name, "resnet50": RESNET50_MATCHA.name,
           "vgg16": VGG16_ALLREDUCE.name, "resnet50opt": RESNET50_MATCHA_OPT.name}


def get(name: str) -> Workload:
    return WORKLOADS[ALIASES.get(name, name)]


@dataclass(frozen=True)
class MlpWorkload:
    """End-to-end workload: n learners train a d_in -> hidden (ReLU) ->
    classes softmax MLP by Non-blocking D-PSGD on a ring."""
    name: str
    n: int = 8
    m: int = 8
    batch: int = 32
    d_in: int = 3072
    hidden: int = 512
    classes: int = 10
    n_samples: int = 50_000
    mixing: str = "ring"
    order: str = MIX_THEN_STEP
    delay: DelaySpec = DelaySpec("exp", 1.0, 1.0)
    lr: float = 0.05
    momentum: float = 0.9
    steps: int = 200
    seed: int = 0
    eval_every: int = 10
    eval_samples: int = 4096
    eval_stride: int = 12      # evaluation subset: samples 0, 12, 24, ...
    matcha_degree: int = 3
    matcha_budget: float | None = None

    @property
    def P(self) -> int:
        return self.d_in * self.hidden + self.hidden + self.hidden * self.classes + self.classes

    @property
    def shard(self) -> int:
        return self.n_samples // self.n

    def eval_indices(self):
        import numpy as np

        return (np.arange(self.eval_samples, dtype=np.int64) * self.eval_stride).astype(np.int32)


MLP = MlpWorkload("mlp_n8_m8_b32_3072x512x10_ring")
MLP_TINY = MlpWorkload("mlp_tiny_n4_m4_b32_128x64x10_ring", n=4, m=4, d_in=128, hidden=64,
                       n_samples=4 * 640, steps=12, eval_every=4, eval_samples=256, eval_stride=10)


# The paper's heterogeneity model (Sec. 6.1): every iteration a random subset
# of learners is slowed by a random factor, the slowest taking up to twice as
# long as the fastest; mini-batch compute time otherwise constant.
MLP_HETERO = replace(MLP, name="mlp_n8_m8_b32_3072x512x10_ring_random_slowdown",
                     delay=DelaySpec("const", 1.0, 0.0, slow_learner=-2, slow_factor=2.0,
                                     slow_prob=0.5))


# The three mixing kinds the paper compares (Sec. 6.2): D-PSGD on the ring
# (above), MATCHA's random matchings of a 3-regular base graph (budget 0.5)
# and ring all-reduce, i.e. uniform W, stepping before the average (Eq. 4-5).
MIXINGS = {"ring": dict(mixing="ring", order=MIX_THEN_STEP),
           "matcha": dict(mixing="matcha", order=MIX_THEN_STEP),
           "uniform": dict(mixing="uniform", order=STEP_THEN_MIX)}


def mlp_with_mixing(wl: MlpWorkload, kind: str) -> MlpWorkload:
    """The MLP workload ``wl`` with another mixing kind (and its order)."""
    name = wl.name.replace("_ring", f"_{'allreduce' if kind == 'uniform' else kind}")
    return replace(wl, name=name, **MIXINGS[kind])
