"""Pins of the oracle's content-aware keyframe selection (Sec. 3.1, Eq. 1;
App. A, Alg. 1): the frame cosine similarity against library routines and
constructions with known answers, and the sequential scan against expected
outputs derived by hand from the algorithm's steps."""
import numpy as np
import pytest
import torch
from scipy.spatial import distance

import oracle


def _frames(x):
    """[B][C][T][H][W] -> [B][T][C*H*W] (frame vectors, channel after channel)."""
    B, C, T = x.shape[:3]
    return np.transpose(x.reshape(B, C, T, -1), (0, 2, 1, 3)).reshape(B, T, -1)


@pytest.mark.parametrize("dtype", [np.float32, np.float64])
def test_cosine_matches_torch_and_scipy(dtype):
    rng = np.random.default_rng(1)
    x = rng.standard_normal((2, 3, 7, 5, 6)).astype(dtype)
    sim = oracle.frame_cosine(x, 2, 3, 7, 5, 6)
    f = _frames(x.astype(np.float64))
    ft = torch.from_numpy(f)
    for b in range(2):
        for i in range(7):
            ref_t = torch.nn.functional.cosine_similarity(ft[b, i:i + 1], ft[b], dim=1).numpy()
            assert np.allclose(sim[b, i], ref_t, rtol=0, atol=1e-13)
            for j in range(7):
                assert abs(sim[b, i, j] - (1.0 - distance.cosine(f[b, i], f[b, j]))) < 1e-13


def test_cosine_bf16_reads_exact_bits():
    x = torch.randn(1, 2, 4, 3, 5, dtype=torch.float32).to(torch.bfloat16)
    sim = oracle.frame_cosine(x, 1, 2, 4, 3, 5)
    f = _frames(x.float().double().numpy())
    ref = torch.nn.functional.cosine_similarity(
        torch.from_numpy(f[0])[:, None, :], torch.from_numpy(f[0])[None, :, :], dim=2).numpy()
    assert np.allclose(sim[0], ref, rtol=0, atol=1e-13)


def test_cosine_frame_layout():
    """Frame f is nonzero only at one element of channel f % C, unique to it:
    the frames are orthogonal, so the matrix is the identity. Mixing up the
    channel and frame axes would make frames overlap."""
    B, C, T, H, W = 1, 3, 6, 2, 2
    x = np.zeros((B, C, T, H, W))
    for f in range(T):
        x[0, f % C, f, f // C, 0] = f + 1.0
    assert np.array_equal(oracle.frame_cosine(x, B, C, T, H, W)[0], np.eye(T))
    # the same frame vector spread over channels: frame f = scaled copy of frame 0
    y = np.zeros((B, C, T, H, W))
    base = np.arange(1, C * H * W + 1, dtype=np.float64).reshape(C, H, W)
    for f in range(T):
        y[0, :, f] = base * (f + 1) * (1 if f % 2 == 0 else -1)
    s = oracle.frame_cosine(y, B, C, T, H, W)[0]
    sign = np.array([1 if f % 2 == 0 else -1 for f in range(T)], dtype=np.float64)
    assert np.allclose(s, np.outer(sign, sign), atol=1e-15)


def test_cosine_invariants():
    rng = np.random.default_rng(2)
    x = rng.standard_normal((1, 4, 5, 3, 3))
    s = oracle.frame_cosine(x, 1, 4, 5, 3, 3)[0]
    assert np.allclose(np.diag(s), 1.0, atol=1e-15)
    assert np.allclose(s, s.T, atol=0)
    assert np.all(np.abs(s) <= 1.0 + 1e-15)
    # positive per-frame scaling leaves every similarity unchanged
    y = x * np.array([3.0, 0.25, 7.0, 1e-3, 2.0]).reshape(1, 1, 5, 1, 1)
    assert np.allclose(oracle.frame_cosine(y, 1, 4, 5, 3, 3)[0], s, atol=1e-14)
    # a zero frame has similarity 0 to every frame (norm clamped at 1e-8)
    z = x.copy()
    z[:, :, 2] = 0.0
    sz = oracle.frame_cosine(z, 1, 4, 5, 3, 3)[0]
    assert np.all(sz[2] == 0.0) and np.all(sz[:, 2] == 0.0)


# --- the sequential scan --------------------------------------------------------------

def _sim_from_last(T, values):
    """A [T][T] matrix whose entries are all 0.5 except those listed:
    values = {(i, j): s} sets sim[i][j] = sim[j][i] = s."""
    s = np.full((T, T), 0.5)
    np.fill_diagonal(s, 1.0)
    for (i, j), v in values.items():
        s[i, j] = s[j, i] = v
    return s


def test_identical_frames_select_only_the_first():
    assert oracle.select_keyframes_adaptive(np.ones((9, 9)), 0.9, 5, 0.1, 1.0, 1.0).tolist() == [0]


def test_budget_stops_the_scan():
    # every frame dissimilar; L_avg = 2.5; each selection has gap 1 <= 2.5 - 0.5,
    # so tau rises; the budget M = 4 ends the scan after frame 3
    got = oracle.select_keyframes_adaptive(np.zeros((10, 10)), 0.5, 4, 0.1, 0.5, 0.5)
    assert got.tolist() == [0, 1, 2, 3]


def test_scene_cuts_with_fixed_threshold():
    # groups [0..4], [5..9], [10..13]: 0.95 within a group, 0.1 across groups
    T = 14
    g = np.array([0] * 5 + [1] * 5 + [2] * 4)
    s = np.where(g[:, None] == g[None, :], 0.95, 0.1)
    assert oracle.select_keyframes_adaptive(s, 0.5, 10, 0.0, 0.0, 0.0).tolist() == [0, 5, 10]


def test_strict_comparison():
    s = _sim_from_last(6, {(3, 0): 0.3})
    # similarity exactly equal to the threshold does not select (Eq. 1 uses <)
    assert oracle.select_keyframes_adaptive(s, 0.3, 6, 0.0, 0.0, 0.0).tolist() == [0]
    assert oracle.select_keyframes_adaptive(s, 0.3 + 1e-12, 6, 0.0, 0.0, 0.0).tolist() == [0, 3]


def test_reference_is_the_most_recent_keyframe():
    # frame 5 is close to keyframe 0 but far from the most recent keyframe 3
    s = _sim_from_last(8, {(3, 0): 0.1, (5, 0): 0.99, (5, 3): 0.1})
    assert oracle.select_keyframes_adaptive(s, 0.3, 8, 0.0, 0.0, 0.0).tolist() == [0, 3, 5]


def test_threshold_adjustment_literal_and_intent():
    """T = 12, M = 3: L_avg = 4. Frame 6 is selected with gap 6 >= 4 + 1, so
    Alg. 1 lowers tau 0.5 -> 0.3 (the intent-consistent sign raises it to 0.7).
    Frame 8 has similarity 0.4 to keyframe 6: selected only with tau = 0.7."""
    T = 12
    vals = {(i, 0): 0.9 for i in range(1, 6)}
    vals[(6, 0)] = 0.1
    vals.update({(i, 6): 0.9 for i in range(7, 12)})
    vals[(8, 6)] = 0.4
    vals.update({(i, 8): 0.9 for i in range(9, 12)})
    s = _sim_from_last(T, vals)
    assert oracle.select_keyframes_adaptive(s, 0.5, 3, 0.2, 1.0, 1.0).tolist() == [0, 6]
    assert oracle.select_keyframes_adaptive(s, 0.5, 3, 0.2, 1.0, 1.0, intent_sign=True).tolist() == [0, 6, 8]


def test_small_gap_raises_threshold():
    """T = 10, M = 3: L_avg = 10/3. Frame 1 (gap 1 <= 10/3 - 2) is selected and
    tau rises 0.3 -> 0.5, so frame 2 (similarity 0.4 to frame 1) is selected and
    fills the budget; with the intent-consistent sign tau falls to 0.1, frame 2
    is passed over and frame 3 (similarity 0.05) is selected."""
    vals = {(1, 0): 0.2, (2, 1): 0.4, (3, 1): 0.05}
    vals.update({(i, 1): 0.9 for i in range(4, 10)})
    s = _sim_from_last(10, vals)
    assert oracle.select_keyframes_adaptive(s, 0.3, 3, 0.2, 2.0, 2.0).tolist() == [0, 1, 2]
    assert oracle.select_keyframes_adaptive(s, 0.3, 3, 0.2, 2.0, 2.0, intent_sign=True).tolist() == [0, 1, 3]


def test_expected_interval_is_a_real_quotient():
    """T = 10, M = 3: L_avg = 10/3. A gap of 4 lowers tau when delta_up = 0.6
    (4 >= 3.93) but not when delta_up = 0.7 (4 < 4.03)."""
    vals = {(i, 0): 0.9 for i in range(1, 4)}
    vals[(4, 0)] = 0.1
    vals[(5, 4)] = 0.25
    vals.update({(i, 4): 0.9 for i in range(6, 10)})
    s = _sim_from_last(10, vals)
    # tau 0.3 -> 0.2 with delta_up 0.6: frame 5 (0.25) is not selected
    assert oracle.select_keyframes_adaptive(s, 0.3, 3, 0.1, 0.6, 5.0).tolist() == [0, 4]
    # no adjustment with delta_up 0.7: frame 5 (0.25 < 0.3) is selected
    assert oracle.select_keyframes_adaptive(s, 0.3, 3, 0.1, 0.7, 5.0).tolist() == [0, 4, 5]


def test_single_frame_and_budget_one():
    assert oracle.select_keyframes_adaptive(np.ones((1, 1)), 0.5, 3, 0.1, 0.0, 0.0).tolist() == [0]
    assert oracle.select_keyframes_adaptive(np.zeros((5, 5)), 0.5, 1, 0.1, 0.0, 0.0).tolist() == [0]


def test_negative_control_plants_a_wrong_sign():
    """A scan that compares with >= instead of < must fail the cut pin."""
    T = 14
    g = np.array([0] * 5 + [1] * 5 + [2] * 4)
    s = np.where(g[:, None] == g[None, :], 0.95, 0.1)
    wrong = [0]
    last = 0
    for i in range(1, T):
        if s[i, last] >= 0.5:
            wrong.append(i)
            last = i
    assert wrong != oracle.select_keyframes_adaptive(s, 0.5, 10, 0.0, 0.0, 0.0).tolist()
