"""The largest frame counts the ABI accepts (RF_MAX_FRAMES = 256 frames, id
lists of up to 256 entries carried in kernel arguments), through every GPU
entry point, against the oracle: attention (keyframe-query, all-frame, split
tail, frame-masked), projection, gather/scatter and the rolling cache."""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_06309_amd import workloads
from parity import assert_parity, torch_bf16_to_f64

pytestmark = pytest.mark.gpu

rf = pytest.importorskip("paper_2606_06309_amd.binding")

T = rf.RF_MAX_FRAMES


def _f64(t):
    return torch_bf16_to_f64(t) if t.dtype == torch.bfloat16 else t.detach().cpu().double().numpy()


def _bits(t):
    t = t.detach().cpu().contiguous()
    return t.view(torch.int16 if t.dtype == torch.bfloat16 else torch.int32).numpy()


KF = tuple(sorted(set(range(0, T, 3)) | {T - 1}))          # 87 keyframes, the last frame among them


@pytest.mark.parametrize("d", [64, 128])
def test_attention_256_frames(d):
    # 256 frames of 2 x 4 tokens: S = 2,048 keys, 696 keyframe query rows
    w = workloads.custom(T, 2, 4, 2, d, KF, dtype="bf16", seed=61)
    print(f"[case] 256 frames d={d} M={w.M}", flush=True)
    q, k, v = workloads.make_qkv(w, device="cuda")
    ref = oracle.keyframe_attention(q.cpu(), k.cpu(), v.cpu(), KF, w.N)
    out = rf.rf_keyframe_attention(q, k, v, KF, T, w.H, w.W)
    out_ws = rf.rf_keyframe_attention_ws(q, k, v, KF, T, w.H, w.W)
    torch.cuda.synchronize()
    assert_parity(_f64(out), ref, "bf16", "256 frames")
    assert_parity(_f64(out_ws), ref, "bf16", "256 frames, split tail")


def test_all_frame_and_frame_mask_256():
    w = workloads.custom(T, 2, 4, 1, 64, KF, dtype="bf16", seed=62)
    q, k, v = workloads.make_qkv(w, device="cuda")
    every = list(range(T))
    out = rf.rf_keyframe_attention(q, k, v, every, T, w.H, w.W)
    kv = [f for f in every if f != 100]                     # 255 key/value frames
    fm = rf.rf_frame_attention(q, k, v, KF, kv, T, w.H, w.W)
    torch.cuda.synchronize()
    rows = np.arange(0, T * w.N, 7)
    ref = oracle.keyframe_attention(q.cpu(), k.cpu(), v.cpu(), every, w.N, rows=rows)
    assert_parity(_f64(out)[rows], ref, "bf16", "all 256 frames")
    ref2 = oracle.frame_attention(q.cpu(), k.cpu(), v.cpu(), KF, kv, w.N)
    assert_parity(_f64(fm), ref2, "bf16", "255 key/value frames")


def test_projection_gather_scatter_256():
    w = workloads.Workload("f256", 63, T, 2, 4, 1, 64, "f32", KF, 1.0, 2, (3, 8))
    lat = workloads.make_latents(w, B=2, device="cuda")
    mask = oracle.keyframe_mask(KF, T)
    out = rf.rf_project_latents(lat, (24.0, 21.0, 23.0), mask)
    torch.cuda.synchronize()
    ref = oracle.project_latents(lat.cpu(), 2, 2, T, 3, 8, (24.0, 21.0, 23.0), mask)
    assert_parity(_f64(out), ref, "f32", "projection 256 frames")
    ids = list(range(T))
    src = torch.randn((T * 5, 16), device="cuda")
    g = rf.rf_gather_frames(src, ids, T, 5)
    back = torch.zeros_like(src)
    rf.rf_scatter_frames(g, back, ids, T, 5)
    torch.cuda.synchronize()
    assert torch.equal(g, src) and torch.equal(back, src)


def test_rolling_cache_255_frames():
    w = workloads.custom(T, 2, 4, 2, 64, (0,), dtype="bf16", seed=64)
    nk = list(range(1, T))                                  # 255 cached frames, slots up to 509
    D = w.heads * w.head_dim
    el = 2
    store = torch.empty(rf.rf_cache_store_bytes(len(nk), w.N, D, torch.bfloat16) // el,
                        dtype=torch.bfloat16, device="cuda")
    h0 = workloads.make_hidden(w, 0, device="cuda")
    h1 = workloads.make_hidden(w, 1, device="cuda")
    c = rf.rf_cache_init(nk, T, w.N, D, torch.bfloat16, 30.0, store=store, h_full=h0)
    rf.rf_cache_shift_store(c, 27.0, store=store, h_full=h1)
    k = torch.zeros((w.S, w.heads, w.head_dim), dtype=torch.bfloat16, device="cuda")
    v = torch.zeros_like(k)
    rf.rf_cache_project_kv(c, store, k, v, 28.0)
    torch.cuda.synchronize()
    a = oracle.hidden_alpha(30.0, 27.0, 28.0)
    hb, ha = _f64(h0).reshape(T, -1), _f64(h1).reshape(T, -1)
    kf = _f64(k).reshape(T, -1)
    exp = (1 - a) * hb[1:] + a * ha[1:]
    bound = 2.0 ** -8 * np.abs(exp) + 2.0 ** -21 * np.maximum(np.abs(hb[1:]), np.abs(ha[1:]))
    assert (np.abs(kf[1:] - exp) <= bound).all()
    assert not kf[0].any()                                   # the keyframe's rows are untouched
    assert np.array_equal(_bits(k)[w.N:], _bits(v)[w.N:])


# --- the device's geometry: the split plan follows its compute units ---------------

def test_plan_follows_the_device():
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    plan = rf.rf_attention_plan(8, 33, 33, 45, 80, 24, 128, rf.RF_BF16)
    assert plan["compute_units"] == cus
    assert plan == rf.rf_attention_plan(8, 33, 33, 45, 80, 24, 128, rf.RF_BF16, cus)
    assert plan["whole_tiles"] % cus == 0 or plan["parts"] == 0
    assert rf.rf_attention_workspace(8, 33, 33, 45, 80, 24, 128, rf.RF_BF16) == plan["workspace_bytes"]


def test_too_small_workspace_is_rejected_before_launch():
    """A workspace smaller than the current device's plan needs is refused
    (checked after the device query, before anything is launched): the output
    buffer keeps its sentinel."""
    w = workloads.custom(8, 16, 16, 2, 128, (0, 5), dtype="bf16", seed=51)
    need = rf.rf_attention_workspace(w.M, w.T, w.T, w.H, w.W, w.heads, w.head_dim, rf.RF_BF16)
    assert need > 0
    q, k, v = workloads.make_qkv(w, device="cuda")
    out = torch.full((w.M * w.N, w.heads, w.head_dim), 7.0, dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(need - 16, dtype=torch.uint8, device="cuda")
    with pytest.raises(rf.RhymeFlowError) as e:
        rf.rf_keyframe_attention_ws(q, k, v, w.keyframes, w.T, w.H, w.W, out=out, workspace=ws)
    assert e.value.status == rf.RF_ERR_INVALID_ARG and "needed" in str(e.value)
    torch.cuda.synchronize()
    assert bool((out == 7.0).all())
