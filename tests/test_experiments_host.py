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
