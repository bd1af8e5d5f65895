"""Pins of the oracle's rolling cache (App. B.2): the epsilon form of alpha,
initialisation, shift-and-store, projection of a linear trajectory, and the
skip-step key/value sequence in which a non-keyframe's projected hidden state is
both its key and its value."""
import numpy as np
import pytest

import oracle


def test_alpha_endpoints_and_midpoint():
    eps = oracle.HIDDEN_EPS
    assert oracle.hidden_alpha(24.0, 21.0, 24.0) == 0.0                      # at t_before
    assert abs(oracle.hidden_alpha(24.0, 21.0, 21.0) - 3.0 / (3.0 + eps)) < 1e-16   # at t_after
    assert abs(oracle.hidden_alpha(24.0, 21.0, 22.5) - 1.5 / (3.0 + eps)) < 1e-16
    assert abs(oracle.hidden_alpha(0.9, 0.5, 0.6) - 0.3 / (0.4 + eps)) < 1e-15


def test_alpha_clamped_and_initial_state():
    assert oracle.hidden_alpha(24.0, 21.0, 30.0) == 0.0     # before the cached interval
    assert oracle.hidden_alpha(24.0, 21.0, 10.0) == 1.0     # after it
    # right after initialisation both slots hold one state at t_w: the quotient
    # (t_w - t) / eps is huge for any later step and clamps to 1
    assert oracle.hidden_alpha(30.0, 30.0, 29.0) == 1.0
    assert oracle.hidden_alpha(30.0, 30.0, 30.0) == 0.0
    with pytest.raises(ValueError):
        oracle.hidden_alpha(float("nan"), 1.0, 0.5)


def test_init_then_projection_returns_the_state():
    rng = np.random.default_rng(0)
    h = {f: rng.standard_normal((6, 4)) for f in (1, 3)}
    c = oracle.RollingCache()
    c.init([1, 3], h, 30.0)
    for t in (30.0, 29.0, 12.5):
        for f in (1, 3):
            assert np.array_equal(c.project(f, t), h[f])


def test_shift_and_store_sequence():
    rng = np.random.default_rng(1)
    h0, h1, h2 = (rng.standard_normal((5, 3)) for _ in range(3))
    c = oracle.RollingCache()
    c.init([2], {2: h0}, 24.0)
    c.shift_and_store([2], {2: h1}, 21.0)
    assert np.array_equal(c.h_before[2], h0) and np.array_equal(c.h_after[2], h1)
    assert (c.t_before[2], c.t_after[2]) == (24.0, 21.0)
    a = 1.0 / (3.0 + oracle.HIDDEN_EPS)
    assert np.allclose(c.project(2, 23.0), (1 - a) * h0 + a * h1, rtol=0, atol=1e-15)
    assert abs(a - 1.0 / 3.0) < 1e-8
    c.shift_and_store([2], {2: h2}, 18.0)
    assert np.array_equal(c.h_before[2], h1) and np.array_equal(c.h_after[2], h2)
    assert (c.t_before[2], c.t_after[2]) == (21.0, 18.0)


def test_linear_trajectory_is_reproduced():
    """h(t) = u + t w cached at t = 20 and 16 is recovered at any t in between,
    up to the epsilon term (relative 1e-8 / 4)."""
    rng = np.random.default_rng(2)
    u, w = rng.standard_normal((2, 7, 5))
    c = oracle.RollingCache()
    c.init([0], {0: u + 20.0 * w}, 20.0)
    c.shift_and_store([0], {0: u + 16.0 * w}, 16.0)
    for t in (20.0, 19.0, 17.5, 16.0):
        assert np.abs(c.project(0, t) - (u + t * w)).max() < 1e-7


def test_skip_step_kv():
    T, N, heads, d = 4, 3, 2, 4
    rng = np.random.default_rng(3)
    k = rng.standard_normal((T * N, heads, d))
    v = rng.standard_normal((T * N, heads, d))
    hb = {f: rng.standard_normal((N, heads * d)) for f in (1, 2)}
    ha = {f: rng.standard_normal((N, heads * d)) for f in (1, 2)}
    c = oracle.RollingCache()
    c.init([1, 2], hb, 24.0)
    c.shift_and_store([1, 2], ha, 21.0)
    K, V = oracle.skip_step_kv(k, v, c, [1, 2], 23.0, N)
    a = 1.0 / (3.0 + oracle.HIDDEN_EPS)
    for f in (0, 3):      # keyframes keep their keys and values
        assert np.array_equal(K[f * N:(f + 1) * N], k[f * N:(f + 1) * N])
        assert np.array_equal(V[f * N:(f + 1) * N], v[f * N:(f + 1) * N])
    for f in (1, 2):      # non-keyframes: key = value = projected hidden state
        exp = ((1 - a) * hb[f] + a * ha[f]).reshape(N, heads, d)
        assert np.allclose(K[f * N:(f + 1) * N], exp, rtol=0, atol=1e-15)
        assert np.array_equal(K[f * N:(f + 1) * N], V[f * N:(f + 1) * N])
    # inputs untouched
    assert not np.shares_memory(K, k) and not np.shares_memory(V, v)


def test_skip_step_attention_with_no_non_keyframes_is_plain():
    w_T, N, heads, d = 3, 4, 1, 8
    rng = np.random.default_rng(4)
    q, k, v = (rng.standard_normal((w_T * N, heads, d)) for _ in range(3))
    K, V = oracle.skip_step_kv(k, v, oracle.RollingCache(), [], 10.0, N)
    assert np.array_equal(K, k) and np.array_equal(V, v)
    a = oracle.keyframe_attention(q, K, V, [0, 2], N)
    b = oracle.keyframe_attention(q, k, v, [0, 2], N)
    assert np.array_equal(a, b)
