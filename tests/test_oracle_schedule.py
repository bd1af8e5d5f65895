"""Pins of the oracle's progressive asynchronous schedule (Eq. 2, Alg. 2):
hand-derived schedules, the paper's default configuration, agreement with
Alg. 2's printed membership test wherever that test is consistent, and the
invariants every schedule must satisfy."""
import itertools

import numpy as np
import pytest

import oracle


def test_eq2_boundaries():
    # T = 50, T_w = 8, T_mid = 25, strides 2 / 3 (the paper's defaults, T_mid = T/2)
    a = (50, 8, 25, 2, 3)
    assert oracle.skip_stride(42, *a) == 2        # first asynchronous step
    assert oracle.skip_stride(26, *a) == 2        # T_mid < t
    assert oracle.skip_stride(25, *a) == 3        # t <= T_mid
    assert oracle.skip_stride(1, *a) == 3
    with pytest.raises(ValueError):
        oracle.skip_stride(43, *a)                # warm-up


def test_hand_schedule_small():
    """T = 10, T_w = 2, T_mid = 4, strides 2 / 3, worked by hand from Alg. 2:
    warm-up at 10 and 9; the non-keyframes (at 8) step 8 -> 6 -> 4 with
    stride 2, then 4 -> 1 and 1 -> 0 with stride 3; in between they are
    projected on the interval they are crossing."""
    got = [(s["t"], s["phase"], s["n_skip"], s["nonkey_to"], s["t_start"], s["t_end"])
           for s in oracle.async_schedule(10, 2, 4, 2, 3)]
    assert got == [
        (10, "warmup", 1, 9, None, None),
        (9, "warmup", 1, 8, None, None),
        (8, "rhythmic", 2, 6, None, None),
        (7, "skip", 2, None, 8, 6),
        (6, "rhythmic", 2, 4, None, None),
        (5, "skip", 2, None, 6, 4),
        (4, "rhythmic", 3, 1, None, None),
        (3, "skip", 3, None, 4, 1),
        (2, "skip", 3, None, 4, 1),
        (1, "rhythmic", 3, 0, None, None),
    ]
    alphas = [s["alpha"] for s in oracle.async_schedule(10, 2, 4, 2, 3) if s["phase"] == "skip"]
    assert alphas == [0.5, 0.5, 1.0 / 3.0, 2.0 / 3.0]


def test_paper_default_configuration():
    """T = 50 steps, T_w = 8, strides 2 / 3 switching at T_mid = 25: 8 warm-up
    steps, Rhythmic Points 42, 40, ..., 26 (stride 2) then 24, 21, ..., 3
    (stride 3), every other step skipped."""
    sch = oracle.async_schedule(50, 8, 25, 2, 3)
    phases = [s["phase"] for s in sch]
    rp = [s["t"] for s in sch if s["phase"] == "rhythmic"]
    assert phases.count("warmup") == 8 and [s["t"] for s in sch[:8]] == list(range(50, 42, -1))
    assert rp == list(range(42, 25, -2)) + list(range(24, 0, -3))
    assert phases.count("skip") == 25 and len(sch) == 50
    # the last Rhythmic Point (3) takes the non-keyframes to 0
    assert sch[-3]["t"] == 3 and sch[-3]["nonkey_to"] == 0
    assert [(s["t_start"], s["t_end"]) for s in sch[-2:]] == [(3, 0), (3, 0)]


def _printed_rule_agrees(T, T_w, T_mid, ns, nl):
    for s in oracle.async_schedule(T, T_w, T_mid, ns, nl):
        if s["phase"] == "warmup":
            continue
        if (s["phase"] == "rhythmic") != oracle.alg2_nonkey_active(s["t"], T, T_w, T_mid, ns, nl):
            return False
    return True


def test_agrees_with_printed_rule_when_consistent():
    assert _printed_rule_agrees(50, 8, 25, 2, 3)
    # one stride throughout: the printed modulo test is exact
    for T, T_w, n in itertools.product([1, 2, 7, 20, 50], [0, 1, 3, 8], [1, 2, 3, 5]):
        if T_w <= T:
            for T_mid in (0, T // 2, T):
                assert _printed_rule_agrees(T, T_w, T_mid, n, n), (T, T_w, T_mid, n)


def test_printed_rule_breaks_where_stride_changes_off_a_rhythmic_point():
    """T_mid = 26: the non-keyframes step 28 -> 26 with stride 2, and 26 is
    not a multiple of 3 away from 42, so the printed test would skip them at
    26 (their state) and update them at 24 (not their state). The state-
    following schedule updates them at 26."""
    assert not oracle.alg2_nonkey_active(26, 50, 8, 26, 2, 3)
    assert oracle.alg2_nonkey_active(24, 50, 8, 26, 2, 3)
    sch = {s["t"]: s for s in oracle.async_schedule(50, 8, 26, 2, 3)}
    assert sch[26]["phase"] == "rhythmic" and sch[26]["nonkey_to"] == 23
    assert sch[24]["phase"] == "skip" and (sch[24]["t_start"], sch[24]["t_end"]) == (26, 23)
    assert not _printed_rule_agrees(50, 8, 26, 2, 3)


def _check_invariants(T, T_w, T_mid, ns, nl):
    sch = oracle.async_schedule(T, T_w, T_mid, ns, nl)
    assert [s["t"] for s in sch] == list(range(T, 0, -1))
    state, left = T, None
    for s in sch:
        t = s["t"]
        if t > T - T_w:
            assert s["phase"] == "warmup" and s["nonkey_to"] == t - 1
            state = t - 1
        elif s["phase"] == "rhythmic":
            assert state == t
            n = ns if t > T_mid else nl
            assert s["n_skip"] == n and s["nonkey_to"] == max(t - n, 0)
            left, state = t, s["nonkey_to"]
        else:
            assert s["phase"] == "skip" and state < t < left
            assert (s["t_start"], s["t_end"]) == (left, state)
            assert 0.0 < s["alpha"] < 1.0
            assert abs(s["alpha"] - oracle.projection_alpha(left, state, t)) < 1e-15
    assert state == 0          # every frame ends at z_0


def test_invariants_random_configurations():
    rng = np.random.default_rng(8)
    for _ in range(400):
        T = int(rng.integers(1, 80))
        T_w = int(rng.integers(0, T + 1))
        T_mid = int(rng.integers(0, T + 1))
        ns = int(rng.integers(1, 6))
        nl = int(rng.integers(ns, 9))
        _check_invariants(T, T_w, T_mid, ns, nl)


def test_degenerate_schedules():
    # stride 1: every asynchronous step is a Rhythmic Point (dense denoising)
    assert all(s["phase"] != "skip" for s in oracle.async_schedule(30, 4, 15, 1, 1))
    # warm-up over all steps
    assert all(s["phase"] == "warmup" for s in oracle.async_schedule(12, 12, 6, 2, 3))
    # no warm-up: the first step is a Rhythmic Point
    assert oracle.async_schedule(12, 0, 6, 2, 3)[0]["phase"] == "rhythmic"
    # a stride larger than the remaining steps jumps straight to 0
    sch = oracle.async_schedule(6, 2, 0, 9, 9)
    assert sch[2]["phase"] == "rhythmic" and sch[2]["nonkey_to"] == 0
    assert [s["phase"] for s in sch[3:]] == ["skip"] * 3
