"""Pins for the oracle's latent trajectory projection, Eq. (3).

z_hat(tau) = (1 - alpha) z(t_start) + alpha z(t_end),
alpha = (t_start - tau) / (t_start - t_end).

Checked against: the endpoints (alpha = 0 at tau = t_start, alpha = 1 at
tau = t_end, App. B.2), the midpoint, exact reproduction of a linear trajectory
z(t) = u + t w (the projection is motivated by near-linear rectified-flow
trajectories, Sec. 3.2.4), equal snapshots (the state right after warm-up,
where both stored states coincide, App. B.2), keyframe planes passed through,
and the clamping reading for tau outside [t_end, t_start].
"""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2606_06309_amd import workloads
from parity import torch_bf16_to_f64

TINY = workloads.WORKLOADS["tiny"]


def _lat(B=2, dtype=torch.float32):
    return workloads.make_latents(TINY, B=B, dtype=dtype)


def _run(lat, ts, mask, B=2):
    Hl, Wl = TINY.latent_hw
    return oracle.project_latents(lat, B, TINY.latent_c, TINY.T, Hl, Wl, ts, mask)


def _slots(lat):
    x = lat.double().numpy() if lat.dtype != torch.bfloat16 else torch_bf16_to_f64(lat)
    return x[:, 0], x[:, 1]


NONE = np.zeros(TINY.T, np.uint8)
KF_MASK = oracle.keyframe_mask(TINY.keyframes, TINY.T)


def test_alpha_values():
    assert oracle.projection_alpha(24, 21, 23) == pytest.approx(1 / 3, abs=1e-16)
    assert oracle.projection_alpha(42, 40, 41) == 0.5
    assert oracle.projection_alpha(10, 5, 10) == 0.0
    assert oracle.projection_alpha(10, 5, 5) == 1.0
    # readings: clamp to [0, 1]; equal endpoints give 1
    assert oracle.projection_alpha(10, 5, 12) == 0.0
    assert oracle.projection_alpha(10, 5, 2) == 1.0
    assert oracle.projection_alpha(7, 7, 7) == 1.0
    # sigma-valued (non-integer) timesteps
    assert oracle.projection_alpha(0.8, 0.6, 0.75) == pytest.approx(0.25, abs=1e-15)
    with pytest.raises(ValueError):
        oracle.projection_alpha(math.nan, 1, 1)


def test_endpoints_are_exact():
    lat = _lat()
    z0, z1 = _slots(lat)
    assert np.array_equal(_run(lat, (24, 21, 24), NONE), z0)
    assert np.array_equal(_run(lat, (24, 21, 21), NONE), z1)


def test_midpoint():
    lat = _lat()
    z0, z1 = _slots(lat)
    out = _run(lat, (42, 40, 41), NONE)
    assert np.abs(out - (z0 + z1) / 2).max() < 1e-15


def test_linear_trajectory_is_reproduced():
    rng = np.random.default_rng(3)
    Hl, Wl = TINY.latent_hw
    shape = (1, TINY.latent_c, TINY.T, Hl, Wl)
    u = rng.standard_normal(shape)
    w = rng.standard_normal(shape)
    t_start, t_end = 0.9, 0.55
    lat = np.stack([u + t_start * w, u + t_end * w], axis=1)
    for tau in (0.9, 0.8, 0.7123, 0.55):
        out = oracle.project_latents(lat, 1, TINY.latent_c, TINY.T, Hl, Wl,
                                     (t_start, t_end, tau), NONE)
        assert np.abs(out - (u + tau * w)).max() < 1e-12


def test_equal_snapshots_are_a_fixed_point():
    lat = _lat()
    lat[:, 1] = lat[:, 0]
    z0, _ = _slots(lat)
    for ts in ((24, 21, 23), (30, 27, 28), (7, 7, 7)):
        out = _run(lat, ts, NONE)
        assert np.abs(out - z0).max() <= 1e-15 * max(1.0, np.abs(z0).max())


def test_keyframe_planes_take_the_current_state():
    lat = _lat()
    z0, z1 = _slots(lat)
    out = _run(lat, (24, 21, 23), KF_MASK)
    alpha = 1 / 3
    for f in range(TINY.T):
        if KF_MASK[f]:
            assert np.array_equal(out[:, :, f], z1[:, :, f])
        else:
            assert np.abs(out[:, :, f] - ((1 - alpha) * z0[:, :, f] + alpha * z1[:, :, f])).max() < 1e-15


def test_bf16_storage_is_widened_exactly():
    lat = _lat(dtype=torch.bfloat16)
    z0, z1 = _slots(lat)
    a = _run(lat, (24, 21, 23), KF_MASK)
    b = _run(np.stack([z0, z1], axis=1), (24, 21, 23), KF_MASK)
    assert np.array_equal(a, b)


def test_size_mismatch_is_rejected():
    lat = _lat()
    with pytest.raises(ValueError):
        oracle.project_latents(lat, 3, TINY.latent_c, TINY.T, 16, 16, (24, 21, 23), NONE)
    with pytest.raises(ValueError):
        _run(lat, (24, math.inf, 23), NONE)
