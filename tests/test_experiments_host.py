"""Host logic of the simulated time-to-loss comparison (no GPU)."""

import pytest

from paper_2211_00889_amd.experiments import time_to


def test_time_to_interpolates_between_evaluations():
    times = [0.0, 10.0, 20.0, 30.0]
    losses = [2.0, 1.5, 1.0, 0.9]
    assert time_to(times, losses, 2.5) == 0.0  # already below at the first evaluation
    assert time_to(times, losses, 1.5) == 10.0  # exactly at an evaluation
    assert time_to(times, losses, 1.25) == pytest.approx(15.0)
    assert time_to(times, losses, 0.95) == pytest.approx(25.0)
    assert time_to(times, losses, 0.5) is None  # never reached


def test_time_to_takes_the_first_crossing():
    # a loss that dips below the level, rises and dips again: the first crossing counts
    times = [0.0, 1.0, 2.0, 3.0]
    losses = [1.0, 0.4, 0.8, 0.2]
    assert time_to(times, losses, 0.5) == pytest.approx(0.5 / 0.6)  # between evaluations 0 and 1


def test_mlp_workloads_of_each_mixing_kind():
    from synth import workloads

    for base in (workloads.MLP, workloads.MLP_HETERO):
        ring = workloads.mlp_with_mixing(base, "ring")
        assert ring == base
        m = workloads.mlp_with_mixing(base, "matcha")
        u = workloads.mlp_with_mixing(base, "uniform")
        assert (m.mixing, m.order) == ("matcha", workloads.MIX_THEN_STEP) and "_matcha" in m.name
        assert (u.mixing, u.order) == ("uniform", workloads.STEP_THEN_MIX) and "_allreduce" in u.name
        assert len({base.name, m.name, u.name}) == 3
        assert m.delay == base.delay and u.n == base.n
