"""The seeded input generators the oracle and the GPU tests share: every named
workload has the shape, head layout, dtype and keyframe set its configuration
states (keyframe sets rebuilt from the stated policy: stride, uniform spacing,
or stride plus seeded extras), and the generators are deterministic, shaped as
documented and drawn with the stated scale."""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_06309_amd import workloads

W = workloads.WORKLOADS


@pytest.mark.parametrize("name,T,H,Wd,heads,d,dtype", [
    ("tiny", 5, 8, 8, 2, 64, "f32"),
    ("small", 13, 30, 52, 12, 128, "bf16"),
    ("480p", 21, 30, 52, 12, 128, "bf16"),
    ("720p", 21, 45, 80, 40, 128, "bf16"),
    ("long", 33, 45, 80, 24, 128, "bf16"),
    ("wan-1.3b", 21, 45, 80, 12, 128, "bf16"),
    ("cogvideox", 11, 48, 85, 48, 64, "bf16"),
])
def test_shapes(name, T, H, Wd, heads, d, dtype):
    w = W[name]
    assert (w.T, w.H, w.W, w.heads, w.head_dim, w.dtype) == (T, H, Wd, heads, d, dtype)
    assert w.N == H * Wd and w.S == T * H * Wd and w.M == len(w.keyframes)


def test_keyframe_sets_follow_the_stated_policies():
    assert W["tiny"].keyframes == (0, 2, 4)
    assert W["small"].keyframes == tuple(oracle.stride_keyframes(13, 3))             # every third frame
    assert W["480p"].keyframes == tuple(oracle.uniform_keyframes(21, 6))              # 6 evenly spaced, ends included
    assert W["720p"].keyframes == tuple(oracle.stride_keyframes(21, 4))               # first + every fourth
    base = set(oracle.stride_keyframes(33, 6).tolist())                                # ratio 1/6 ...
    extra = set(W["long"].keyframes) - base                                            # ... plus 2 seeded extras
    assert base <= set(W["long"].keyframes) and len(extra) == 2
    assert extra == {22, 31}
    assert W["long"].M == 8
    # the paper's two models with its default budget of 4 keyframes, evenly spaced
    assert W["wan-1.3b"].keyframes == tuple(oracle.uniform_keyframes(21, 4)) == (0, 7, 13, 20)
    assert W["cogvideox"].keyframes == tuple(oracle.uniform_keyframes(11, 4)) == (0, 3, 7, 10)
    assert W["wan-1.3b"].N == 3600 and W["cogvideox"].N == 4080


def test_small_workload_is_scaled():
    assert W["small"].qkv_scale == pytest.approx(1.0 / np.sqrt(128.0))
    assert all(W[n].qkv_scale == 1.0 for n in ("tiny", "480p", "720p", "long", "wan-1.3b", "cogvideox"))


def test_qkv_deterministic_shaped_and_scaled():
    w = workloads.custom(3, 8, 8, 2, 64, (0, 2), dtype="bf16", seed=7)
    q1, k1, v1 = workloads.make_qkv(w)
    q2, k2, v2 = workloads.make_qkv(w)
    assert q1.shape == (w.S, 2, 64) and q1.dtype == torch.bfloat16
    assert torch.equal(q1, q2) and torch.equal(k1, k2) and torch.equal(v1, v2)
    assert not torch.equal(q1, k1) and not torch.equal(k1, v1)
    q3, _, _ = workloads.make_qkv(w, seed=8)
    assert not torch.equal(q1, q3)
    qs, _, _ = workloads.make_qkv(w, scale=0.25)
    assert float(qs.float().std()) == pytest.approx(0.25 * float(q1.float().std()), rel=0.02)
    assert abs(float(q1.float().std()) - 1.0) < 0.1


def test_latents_two_independent_slots():
    lat = workloads.make_latents(W["tiny"], B=2)
    assert lat.shape == (2, 2, 4, 5, 16, 16) and lat.dtype == torch.float32
    assert not torch.equal(lat[:, 0], lat[:, 1])
    assert torch.equal(lat, workloads.make_latents(W["tiny"], B=2))


@pytest.mark.parametrize("name", ["small", "long", "cogvideox"])
def test_sample_rows_cover_the_edges(name):
    w = W[name]
    rows = workloads.sample_rows(w, per_head=64)
    Mq = w.M * w.N
    assert np.all(np.diff(rows) > 0) and rows[0] >= 0 and rows[-1] == Mq - 1
    for m in range(w.M):
        assert m * w.N in rows and m * w.N + w.N - 1 in rows
    assert rows.size >= 64
