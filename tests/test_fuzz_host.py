"""Property-based checks of the host entry points of the library (no GPU): for
random and invalid arguments every call either returns one of the documented
error statuses or succeeds with its invariants intact, and never crashes."""

import math

import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

import oracle
import paper_2211_00889_amd as nb
from paper_2211_00889_amd import _lib

SETTINGS = settings(max_examples=300, deadline=None, derandomize=True,
                    suppress_health_check=[HealthCheck.too_slow])
ERRORS = {_lib.E_ARG, _lib.E_SHAPE, _lib.E_UNSUPPORTED}
floats = st.one_of(st.floats(min_value=-4.0, max_value=8.0),
                   st.sampled_from([0.0, -0.0, math.inf, -math.inf, math.nan, 1e-300, 1e300]))


@SETTINGS
@given(seed=st.integers(0, 2**64 - 1), step=st.integers(0, 2**64 - 1), n=st.integers(-2, 20),
       m=st.integers(-2, 70), kind=st.integers(-1, 4), base=floats, param=floats,
       slow=st.integers(-4, 20), factor=floats, prob=floats)
def test_sample_mask_any_arguments(seed, step, n, m, kind, base, param, slow, factor, prob):
    try:
        mask, counts, times, timing = nb.sample_mask(seed, step, n, m, kind, base, param, slow,
                                                     factor, prob)
    except nb.NbsgdError as e:
        assert e.status in ERRORS
        return
    # accepted: the documented argument ranges hold and the schedule is consistent
    assert 1 <= n <= 16 and 1 <= m <= 64 and kind in (0, 1, 2) and base >= 0
    assert ((counts >= 1) & (counts <= m)).all()
    assert np.array_equal(mask, (np.arange(m)[None, :] < counts[:, None]).astype(np.uint8))
    assert (times >= 0).all()  # no NaN: the delay parameters are finite
    T, t_sync, t_step = timing
    assert T <= t_step <= t_sync
    d = oracle.schedule.Delay(kind, base, param, slow, factor, prob)
    s = oracle.schedule.sample_schedule(seed, step, n, m, d)
    assert np.array_equal(mask, s["mask"]) and np.array_equal(counts, s["counts"])


@SETTINGS
@given(seed=st.integers(0, 2**64 - 1), n=st.integers(-1, 20), degree=st.integers(-1, 8))
def test_matcha_create_any_arguments(seed, n, degree):
    try:
        g = nb.Matcha(seed, n, degree)
    except nb.NbsgdError as e:
        assert e.status in ERRORS
        # rejected: no simple connected degree-regular graph on n nodes exists,
        # or a simple pairing is too unlikely (about exp(-(d^2 - 1) / 4) per
        # attempt) for the pairing model's 100,000 attempts
        exists = (2 <= n <= 16 and 1 <= degree < n and (n * degree) % 2 == 0
                  and (degree > 1 or n == 2))
        assert not exists or (e.status == _lib.E_SHAPE and (degree >= 7 or 2 * degree >= n))
        return
    edges, M = g.matchings()
    assert len(edges) == n * degree // 2 and 1 <= M <= 2 * degree - 1
    W, active = g.w(seed % 97)
    assert 0 <= active <= M
    np.testing.assert_allclose(W.sum(axis=0), 1.0, atol=1e-6)
    np.testing.assert_allclose(W.sum(axis=1), 1.0, atol=1e-6)
    assert (W >= 0).all() and np.array_equal(W, W.T)
    g.close()


@SETTINGS
@given(P=st.one_of(st.integers(-5, 1 << 40), st.integers((1 << 20) - 2, (1 << 22) + 2)))
def test_row_stride_any_size(P):
    try:
        ld = nb.row_stride(P)
    except nb.NbsgdError as e:
        assert e.status == _lib.E_SHAPE and P < 0
        return
    u, s = 1 << 22, 1 << 20
    assert ld >= P >= 0
    if P <= s:
        assert ld == P
    elif P <= u:
        assert ld & (ld - 1) == 0 and ld < 2 * P
    else:
        k = ld // u
        assert ld % u == 0 and k & (k - 1) != 0 and ld - P < 2 * u


@SETTINGS
@given(d_in=st.integers(-1, 5000), hidden=st.integers(-1, 1100), classes=st.integers(-1, 20),
       batch=st.sampled_from([-1, 0, 16, 32, 64]))
def test_mlp_shape_any_arguments(d_in, hidden, classes, batch):
    try:
        P = nb.mlp_param_count(d_in, hidden, classes, batch)
    except nb.NbsgdError as e:
        assert e.status in ERRORS
        return
    assert batch == 32 and d_in % 128 == 0 and d_in >= 128 and hidden % 64 == 0
    assert 64 <= hidden <= 512 and 2 <= classes <= 16
    logical = d_in * hidden + hidden + hidden * classes + classes
    assert P == (logical + 3) // 4 * 4
    ws = nb.mlp_workspace_bytes(d_in, hidden, classes, 96, batch)
    assert ws >= 96 * (4 + 4 + hidden * 4 + hidden * 2)


@SETTINGS
@given(seed=st.integers(0, 2**64 - 1), step=st.integers(0, 10_000), n=st.integers(-1, 18),
       m=st.integers(-1, 66), b=st.integers(-1, 40), shard=st.integers(-1, 3000))
def test_minibatch_indices_any_arguments(seed, step, n, m, b, shard):
    try:
        idx = nb.minibatch_indices(seed, step, n, m, b, shard)
    except nb.NbsgdError as e:
        assert e.status in ERRORS
        return
    assert 1 <= n <= 16 and 1 <= m <= 64 and b >= 1 and shard >= m * b
    for i in range(n):
        row = idx[i].reshape(-1)
        assert len(set(row.tolist())) == row.size  # a window of one permutation
        assert ((row >= shard * i) & (row < shard * (i + 1))).all()


@pytest.mark.parametrize("n", [0, 17, -3])
def test_w_builders_reject_bad_n(n):
    for f in (nb.w_ring, nb.w_allreduce):
        with pytest.raises(nb.NbsgdError) as e:
            f(n)
        assert e.value.status in ERRORS
