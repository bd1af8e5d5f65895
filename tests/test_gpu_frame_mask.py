"""GPU parity of attention under a frame-level key/value mask
(rf_frame_attention) against the oracle's frame_attention, through the C ABI:
keyframe-only and other key/value frame lists on shapes whose frames are and
are not multiples of the key tile, every element; masked frames filled with
NaN (never read, so the output is unchanged bit for bit); the all-frames list
equal to rf_keyframe_attention; sampled rows at 33 x 45 x 80, 24 heads."""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_06309_amd import workloads
from parity import assert_parity, torch_bf16_to_f64

pytestmark = pytest.mark.gpu

rf = pytest.importorskip("paper_2606_06309_amd.binding")


def _f64(t):
    return torch_bf16_to_f64(t) if t.dtype == torch.bfloat16 else t.detach().cpu().double().numpy()


def _bits(t):
    t = t.detach().cpu().contiguous()
    return t.view(torch.int16 if t.dtype == torch.bfloat16 else torch.int32).numpy()


CASES = [
    # (workload, query frames, key/value frames)
    (workloads.WORKLOADS["tiny"], (0, 2, 4), (0, 2, 4)),                                   # fp32, N = 64
    (workloads.custom(5, 10, 13, 3, 128, (0, 2, 4), dtype="f32", seed=41), (0, 2, 4), (1, 4)),   # N = 130
    (workloads.custom(5, 10, 13, 3, 128, (0, 2, 4), dtype="bf16", seed=42), (0, 2, 4), (0, 2, 4)),
    (workloads.custom(5, 10, 13, 3, 64, (0, 2, 4), dtype="bf16", seed=43), (0, 2, 4), (0, 1, 3)),
    (workloads.custom(7, 5, 7, 2, 128, (0, 3, 6), dtype="bf16", seed=44), (0, 3, 6), (6,)),        # N = 35 < tile
    (workloads.custom(6, 8, 16, 2, 128, (0, 5), dtype="bf16", seed=45), (0, 5), (0, 1, 2, 3, 4)),  # N = 128
    (workloads.custom(9, 6, 10, 2, 128, (1, 4, 8), dtype="bf16", seed=46), (1, 4, 8), (0, 8)),     # frames far apart
    (workloads.custom(4, 12, 15, 2, 128, (0, 1, 2, 3), dtype="bf16", seed=47), (0, 1, 2, 3), (2,)),  # full queries
]


def _ids(c):
    w, qf, kvf = c
    return f"{w.name}_T{w.T}_N{w.N}_d{w.head_dim}_{w.dtype}_kv{'-'.join(map(str, kvf))}"


@pytest.mark.parametrize("case", CASES, ids=_ids)
def test_parity_every_element(case):
    w, qf, kvf = case
    print(f"[case] frame mask {_ids(case)}", flush=True)
    q, k, v = workloads.make_qkv(w, device="cuda")
    out = rf.rf_frame_attention(q, k, v, qf, kvf, w.T, w.H, w.W)
    torch.cuda.synchronize()
    ref = oracle.frame_attention(q.cpu(), k.cpu(), v.cpu(), qf, kvf, w.N)
    assert_parity(_f64(out), ref, "f32" if w.dtype == "f32" else "bf16", _ids(case))


@pytest.mark.parametrize("case", CASES[1:5], ids=_ids)
def test_masked_frames_are_never_read(case):
    w, qf, kvf = case
    q, k, v = workloads.make_qkv(w, device="cuda")
    base = rf.rf_frame_attention(q, k, v, qf, kvf, w.T, w.H, w.W)
    k2, v2 = k.clone(), v.clone()
    for f in range(w.T):
        if f not in kvf:
            k2[f * w.N:(f + 1) * w.N] = float("nan")
            v2[f * w.N:(f + 1) * w.N] = float("nan")
    got = rf.rf_frame_attention(q, k2, v2, qf, kvf, w.T, w.H, w.W)
    torch.cuda.synchronize()
    assert np.array_equal(_bits(got), _bits(base))
    assert bool(torch.isfinite(got.float()).all())


@pytest.mark.parametrize("case", [CASES[0], CASES[2]], ids=_ids)
def test_all_frames_is_keyframe_attention(case):
    w, qf, _ = case
    q, k, v = workloads.make_qkv(w, device="cuda")
    a = rf.rf_frame_attention(q, k, v, qf, list(range(w.T)), w.T, w.H, w.W)
    b = rf.rf_keyframe_attention(q, k, v, qf, w.T, w.H, w.W)
    torch.cuda.synchronize()
    assert np.array_equal(_bits(a), _bits(b))


def test_long_workload_keyframe_only_sampled():
    """33 frames of 45 x 80 tokens, 24 heads: the keyframes' queries over the
    keyframes' keys only (the keyframe-only ablation), sampled rows and heads."""
    w = workloads.WORKLOADS["long"]
    print("[case] frame mask long keyframe-only", flush=True)
    q, k, v = workloads.make_qkv(w, device="cuda")
    out = rf.rf_frame_attention(q, k, v, w.keyframes, w.keyframes, w.T, w.H, w.W)
    torch.cuda.synchronize()
    rows = workloads.sample_rows(w, 48)
    heads = np.array([0, 11, 23])
    got = _f64(out[torch.as_tensor(rows, device="cuda")])[:, heads]
    ref = oracle.frame_attention(q.cpu(), k.cpu(), v.cpu(), w.keyframes, w.keyframes, w.N,
                                 rows=rows, heads=heads)
    assert_parity(got, ref, "bf16", "long keyframe-only sampled")


def test_errors():
    w = CASES[2][0]
    q, k, v = workloads.make_qkv(w, device="cuda")
    for kvf, status in [((), rf.RF_ERR_INVALID_ARG), ((2, 1), rf.RF_ERR_INVALID_ARG),
                        ((0, 5), rf.RF_ERR_RANGE)]:
        with pytest.raises(rf.RhymeFlowError) as e:
            rf.rf_frame_attention(q, k, v, (0, 2), kvf, w.T, w.H, w.W)
        assert e.value.status == status
