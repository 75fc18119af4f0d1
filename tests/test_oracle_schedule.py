"""Pins for the simulated schedule: Lemma 1 / Thm 2 closed forms (App. A and B),
the Lomax tail, and the structural invariants of the mask."""

import math

import numpy as np
import pytest

from oracle import schedule
from oracle.schedule import DELAY_CONST, DELAY_EXP, DELAY_LOMAX, Delay


def _paper_sync_sum(n, lam):
    # App. B closed form: (n / lam) * sum_k C(n-1, k) (-1)^k / (k + 1)^2
    return (n / lam) * sum(math.comb(n - 1, k) * (-1) ** k / (k + 1) ** 2 for k in range(n))


@pytest.mark.parametrize("n", [2, 4, 8, 10, 16])
def test_paper_sum_is_harmonic_number(n):
    # E[max of n Exp(lam)] is H_n / lam (textbook); the paper's sum must agree
    H = sum(1.0 / k for k in range(1, n + 1))
    assert _paper_sync_sum(n, 1.0) == pytest.approx(H, rel=1e-9)


@pytest.mark.parametrize("n,lam", [(4, 1.0), (10, 0.5)])
def test_thm2_expected_iteration_times(n, lam):
    # One mini-batch per learner and no constant part: the terminal signal
    # comes at the minimum of n Exp(lam) times, E = 1 / (n lam) (Thm 2,
    # App. A); the blocking baseline waits for the maximum (App. B).
    d = Delay(DELAY_EXP, base=0.0, param=lam)
    draws = 6000
    T = np.empty(draws)
    S = np.empty(draws)
    for k in range(draws):
        s = schedule.sample_schedule(3, k, n, 1, d)
        T[k] = s["deadline"]
        S[k] = s["t_sync"]
    mean_min, sd_min = 1.0 / (n * lam), 1.0 / (n * lam)  # min is Exp(n lam)
    z = (T.mean() - mean_min) / (sd_min / math.sqrt(draws))
    assert abs(z) < 4.0
    var_max = sum(1.0 / (k * lam) ** 2 for k in range(1, n + 1))
    z = (S.mean() - _paper_sync_sum(n, lam)) / math.sqrt(var_max / draws)
    assert abs(z) < 4.0


def test_lomax_tail():
    # base 0: D itself, P(D > x) = (1 + x)^-shape
    d = Delay(DELAY_LOMAX, base=0.0, param=1.5)
    xs = np.array([schedule.minibatch_time(5, 0, 0, j, d) for j in range(20000)])
    for x in (0.5, 1.0, 3.0, 10.0):
        p = (1.0 + x) ** -1.5
        emp = (xs > x).mean()
        assert abs(emp - p) < 4.0 * math.sqrt(p * (1 - p) / xs.size)


def test_exp_mean_and_scale():
    d = Delay(DELAY_EXP, base=1.0, param=0.5, slow_learner=1, slow_factor=3.0)
    t0 = np.array([schedule.minibatch_time(9, k, 0, 0, d) for k in range(5000)])
    t1 = np.array([schedule.minibatch_time(9, k, 1, 0, d) for k in range(5000)])
    assert t0.min() > 1.0
    assert abs(t0.mean() - 3.0) < 4 * 2.0 / math.sqrt(5000)  # 1 + mean 1/0.5
    assert abs(t1.mean() - 9.0) < 4 * 6.0 / math.sqrt(5000)  # slowed x3


@pytest.mark.parametrize("kind", [DELAY_EXP, DELAY_LOMAX])
def test_mask_invariants(kind):
    d = Delay(kind, 1.0, 1.0 if kind == DELAY_EXP else 1.5, slow_learner=2, slow_factor=3.0)
    for step in range(40):
        s = schedule.sample_schedule(0, step, 6, 5, d)
        mask, counts = s["mask"], s["counts"]
        assert counts.min() >= 1 and counts.max() == 5  # the signaller finished all
        for i in range(6):
            assert list(mask[i]) == [1] * counts[i] + [0] * (5 - counts[i])
            # finished mini-batches end no later than the deadline, unless forced
            if counts[i] > 1 or s["finish"][i, 0] <= s["deadline"]:
                assert s["finish"][i, counts[i] - 1] <= s["deadline"]
            if counts[i] < 5:
                assert s["finish"][i, counts[i]] > s["deadline"]
        assert s["deadline"] == s["finish"][:, -1].min()
        assert s["t_sync"] == s["finish"][:, -1].max()
        assert s["t_step"] >= s["deadline"]


def test_const_delay_gives_full_mask():
    s = schedule.sample_schedule(0, 0, 5, 7, Delay(DELAY_CONST, base=1.0))
    assert s["mask"].all() and (s["counts"] == 7).all()


def test_huge_straggler_keeps_one_minibatch():
    d = Delay(DELAY_EXP, 1.0, 1.0, slow_learner=0, slow_factor=1e9)
    s = schedule.sample_schedule(0, 0, 4, 8, d)
    assert s["counts"][0] == 1
    assert s["t_step"] == s["finish"][0, 0] > s["deadline"]


def test_deterministic_in_seed_and_step():
    d = Delay(DELAY_EXP, 1.0, 1.0)
    a = schedule.sample_schedule(11, 4, 4, 4, d)
    b = schedule.sample_schedule(11, 4, 4, 4, d)
    c = schedule.sample_schedule(11, 5, 4, 4, d)
    assert np.array_equal(a["times"], b["times"])
    assert not np.array_equal(a["times"], c["times"])


def test_random_slowdown_model():
    # Sec. 6.1 heterogeneity: slowed nodes and slow-down rates change every
    # iteration, the slowest taking up to twice as long as the fastest
    from oracle.schedule import SLOW_RANDOM

    d = Delay(DELAY_CONST, base=1.0, slow_learner=SLOW_RANDOM, slow_factor=2.0, slow_prob=0.5)
    scales = np.array([[schedule.slowdown(3, k, i, d) for i in range(8)] for k in range(3000)])
    slowed = scales > 1.0
    assert abs(slowed.mean() - 0.5) < 4 * 0.5 / math.sqrt(scales.size)
    assert scales.min() >= 1.0 and scales.max() < 2.0
    s = scales[slowed]
    assert abs(s.mean() - 1.5) < 4 * (1 / math.sqrt(12)) / math.sqrt(s.size)  # uniform on (1, 2)
    # the slowed set changes between iterations
    assert not all(np.array_equal(slowed[k], slowed[k + 1]) for k in range(20))
    # with constant base times a learner's mini-batch time is exactly its scale
    sch = schedule.sample_schedule(3, 5, 8, 4, d)
    np.testing.assert_array_equal(sch["times"][:, 0], scales[5])
    assert sch["times"].max() / sch["times"].min() < 2.0


# ------------------------------------------------ Sec. 4.3 accounting (Thm 3-5, Cor. 1)
@pytest.mark.parametrize("n,m", [(1, 1), (4, 4), (8, 8), (16, 4)])
def test_accounting_equal_times(n, m):
    """Every learner as fast as the others: Y X_{1:P} = P, the Cor. 1 amount
    is the whole P B, and non-blocking has the blocking throughput (Thm 5 ratio
    1)."""
    s = schedule.sample_schedule(0, 3, n, m, Delay(DELAY_CONST, 1.5, 0.0))
    a = schedule.accounting(s["times"])
    assert a["x_first"] == a["x_last"] == 1.5 * m
    assert a["y"] * a["x_first"] == pytest.approx(n, rel=1e-15)
    assert a["data"] == pytest.approx(n * m, rel=1e-15)
    assert a["ratio"] == pytest.approx(1.0, rel=1e-15)
    assert a["throughput"] == pytest.approx(a["throughput_sync"], rel=1e-15)


@pytest.mark.parametrize("n,m,factor", [(8, 8, 2.0), (16, 4, 2.0), (5, 64, 3.0), (8, 16, 1.3)])
def test_accounting_constant_speed_bounds_finished_counts(n, m, factor):
    """Cor. 1 assumes each learner runs at a constant speed within the
    iteration.  DELAY_CONST with the random slow-down is exactly that (learner
    i's mini-batches all take s_i), so learner i finishes floor(m T / X_i) of
    them by T = X_{1:P}: the finished total lies in (data - P, data]."""
    d = Delay(DELAY_CONST, 1.0, 0.0, schedule.SLOW_RANDOM, factor, 0.5)
    for step in range(40):
        s = schedule.sample_schedule(11, step, n, m, d)
        a = schedule.accounting(s["times"])
        total = int(s["counts"].sum())
        assert a["data"] - n - 1e-9 < total <= a["data"] + 1e-9, step
        assert a["x_first"] == s["deadline"] and a["x_last"] == s["t_sync"]
        X = s["finish"][:, m - 1]
        for i in range(n):
            share = m * a["x_first"] / X[i]  # learner i's Cor. 1 share
            assert share - 1 - 1e-9 < s["counts"][i] <= share + 1e-9, (step, i)


@pytest.mark.parametrize("kind,param,slow,factor", [(DELAY_EXP, 1.0, -1, 1.0), (DELAY_LOMAX, 1.5, -1, 1.0),
                                                    (DELAY_EXP, 1.0, 7, 3.0)])
def test_accounting_invariants(kind, param, slow, factor):
    """Thm 5 is Thm 3 over Thm 4, at least 1 (no learner is slower than the
    slowest), and Y X_{1:P} lies between 1 (the fastest learner's own share)
    and P."""
    n, m = 8, 8
    for step in range(30):
        s = schedule.sample_schedule(2, step, n, m, Delay(kind, 1.0, param, slow, factor))
        a = schedule.accounting(s["times"])
        assert a["ratio"] == pytest.approx(a["throughput"] / a["throughput_sync"], rel=1e-14)
        assert a["ratio"] >= 1.0 - 1e-15
        yx = a["data"] / m
        assert 1.0 - 1e-12 <= yx <= n + 1e-12
        # Y itself: the per-learner throughputs added up, in any order
        X = s["finish"][:, m - 1]
        assert a["y"] == pytest.approx(float(np.sum(1.0 / X)), rel=1e-14)
