"""GPU parity of the latent trajectory projection (Eq. 3) and of the frame
gather/scatter, through the C ABI, against the oracle."""
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
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy()
    if t.dtype == torch.float32:
        return t.view(torch.int32).numpy()
    return t.numpy()


def _project_case(w, B=1, dtype=torch.float32, ts=None, mask=None):
    print(f"[case] projection {w.name} B={B} dtype={dtype}", flush=True)
    lat = workloads.make_latents(w, B=B, device="cuda", dtype=dtype)
    ts = w.timesteps if ts is None else ts
    mask = oracle.keyframe_mask(w.keyframes, w.T) if mask is None else mask
    out = rf.rf_project_latents(lat, ts, mask)
    torch.cuda.synchronize()
    Hl, Wl = w.latent_hw
    ref = oracle.project_latents(lat.cpu(), B, w.latent_c, w.T, Hl, Wl, ts, mask)
    return lat, out, ref, mask


@pytest.mark.parametrize("name", ["tiny", "480p"])
def test_projection_fp32(name):
    w = workloads.WORKLOADS[name]
    lat, out, ref, mask = _project_case(w, B=2)
    assert_parity(_f64(out), ref, "f32", name)
    # keyframe planes are the current state, bit for bit
    o, l1 = _bits(out), _bits(lat[:, 1])
    for f in range(w.T):
        if mask[f]:
            assert np.array_equal(o[:, :, f], l1[:, :, f])


def test_projection_bf16():
    w = workloads.WORKLOADS["480p"]
    lat, out, ref, _ = _project_case(w, dtype=torch.bfloat16)
    assert_parity(_f64(out), ref, "bf16", "480p bf16")


def test_projection_endpoints_bit_exact():
    w = workloads.WORKLOADS["tiny"]
    none = np.zeros(w.T, np.uint8)
    lat = workloads.make_latents(w, B=1, device="cuda")
    a = rf.rf_project_latents(lat, (24, 21, 24), none)
    b = rf.rf_project_latents(lat, (24, 21, 21), none)
    assert torch.equal(a, lat[:, 0]) and torch.equal(b, lat[:, 1])


def test_projection_scalar_path_and_clamp():
    # plane of 5 x 7 = 35 elements (not a multiple of the 16-byte vector)
    w = workloads.Workload("odd", 7, 4, 1, 1, 1, 64, "f32", (0, 3), 1.0, 3, (5, 7))
    for ts in [(10.0, 5.0, 7.5), (10.0, 5.0, 12.0), (0.8, 0.55, 0.6123), (3.0, 3.0, 3.0)]:
        for dt in (torch.float32, torch.bfloat16):
            _, out, ref, _ = _project_case(w, B=3, dtype=dt, ts=ts)
            assert_parity(_f64(out), ref, "f32" if dt == torch.float32 else "bf16", f"odd {ts}")


def test_projection_in_place_on_slot1():
    w = workloads.WORKLOADS["tiny"]
    lat = workloads.make_latents(w, B=1, device="cuda")
    mask = oracle.keyframe_mask(w.keyframes, w.T)
    Hl, Wl = w.latent_hw
    ref = oracle.project_latents(lat.cpu(), 1, w.latent_c, w.T, Hl, Wl, w.timesteps, mask)
    key_before = _bits(lat[:, 1])
    out = rf.rf_project_latents(lat, w.timesteps, mask, out=lat[:, 1])
    torch.cuda.synchronize()
    assert out.data_ptr() == lat[:, 1].data_ptr()
    assert_parity(_f64(lat[:, 1]), ref, "f32", "in place")
    after = _bits(lat[:, 1])
    for f in range(w.T):
        if mask[f]:
            assert np.array_equal(after[:, :, f], key_before[:, :, f])


def test_projection_linear_trajectory():
    w = workloads.WORKLOADS["tiny"]
    g = torch.Generator(device="cuda").manual_seed(5)
    Hl, Wl = w.latent_hw
    u = torch.randn((1, w.latent_c, w.T, Hl, Wl), generator=g, device="cuda")
    d = torch.randn((1, w.latent_c, w.T, Hl, Wl), generator=g, device="cuda")
    lat = torch.stack([u + 0.9 * d, u + 0.5 * d], dim=1).contiguous()
    out = rf.rf_project_latents(lat, (0.9, 0.5, 0.6), np.zeros(w.T, np.uint8))
    exact = (u.double() + 0.6 * d.double()).cpu().numpy()
    assert np.abs(out.double().cpu().numpy() - exact).max() < 1e-5


# --- gather / scatter ------------------------------------------------------------------

def _random_bits(rows, cols, seed):
    g = torch.Generator(device="cuda").manual_seed(seed)
    return torch.randint(-32768, 32767, (rows, cols), generator=g, device="cuda",
                         dtype=torch.int32).to(torch.int16)


@pytest.mark.parametrize("name", ["small", "480p"])
def test_gather_bit_exact(name):
    w = workloads.WORKLOADS[name]
    print(f"[case] gather {name}", flush=True)
    src = _random_bits(w.S, w.heads * w.head_dim, 41)
    out = rf.rf_gather_frames(src, w.keyframes, w.T, w.N)
    torch.cuda.synchronize()
    exp = oracle.gather_frames(src.cpu().numpy(), w.keyframes, w.N)
    assert np.array_equal(out.cpu().numpy(), exp)


def test_scatter_bit_exact_and_leaves_other_rows():
    w = workloads.WORKLOADS["480p"]
    print("[case] scatter 480p", flush=True)
    compact = _random_bits(w.M * w.N, w.heads * w.head_dim, 42)
    dst = torch.full((w.S, w.heads * w.head_dim), 0x5A5A, dtype=torch.int16, device="cuda")
    before = dst.cpu().numpy()
    rf.rf_scatter_frames(compact, dst, w.keyframes, w.T, w.N)
    torch.cuda.synchronize()
    exp = oracle.scatter_frames(compact.cpu().numpy(), before, w.keyframes, w.N)
    assert np.array_equal(dst.cpu().numpy(), exp)


def test_gather_scatter_round_trip_long_full_size():
    w = workloads.WORKLOADS["long"]
    print("[case] gather/scatter long", flush=True)
    src = _random_bits(w.S, w.heads * w.head_dim, 43)
    compact = rf.rf_gather_frames(src, w.keyframes, w.T, w.N)
    dst = torch.zeros_like(src)
    rf.rf_scatter_frames(compact, dst, w.keyframes, w.T, w.N)
    torch.cuda.synchronize()
    tok = torch.from_numpy(oracle.rowmap(w.keyframes, w.N)).cuda()
    assert torch.equal(compact, src.index_select(0, tok))
    assert torch.equal(dst.index_select(0, tok), compact)
    mask = torch.ones(w.S, dtype=torch.bool, device="cuda")
    mask[tok] = False
    assert int(dst[mask].abs().sum()) == 0


def test_attention_then_scatter_pipeline():
    """One skip step: project non-keyframe latents, keyframe-query attention,
    scatter the keyframe rows into the full-sequence output."""
    w = workloads.custom(5, 10, 13, 2, 128, (0, 2, 4), dtype="bf16", seed=44)
    q, k, v = workloads.make_qkv(w, device="cuda")
    full = torch.zeros((w.S, w.heads, w.head_dim), dtype=torch.bfloat16, device="cuda")
    out = rf.rf_keyframe_attention(q, k, v, w.keyframes, w.T, w.H, w.W)
    rf.rf_scatter_frames(out, full, w.keyframes, w.T, w.N)
    torch.cuda.synchronize()
    ref = oracle.keyframe_attention(q.cpu(), k.cpu(), v.cpu(), w.keyframes, w.N)
    tok = oracle.rowmap(w.keyframes, w.N)
    got = torch_bf16_to_f64(full)
    assert_parity(got[tok], ref, "bf16", "pipeline")
    others = np.setdiff1d(np.arange(w.S), tok)
    assert np.all(got[others] == 0)


# --- workgroup boundaries of the launch shapes -------------------------------------------
# The copy runs one wave per 1 KB (64 vectors of 16 bytes), the projection 256 vectors per
# workgroup: frames and planes just under, at and over those sizes, and tiny ones.

@pytest.mark.parametrize("rows,row_bytes", [(1, 16), (3, 16), (63, 16), (64, 16), (65, 16), (2, 1024),
                                            (1, 1040), (127, 16)])
def test_gather_scatter_frame_sizes_around_a_workgroup(rows, row_bytes):
    T = 256
    ids = list(range(0, T - 1, 3)) + [T - 1]   # every third frame and the last one
    print(f"[case] gather/scatter rows={rows} row_bytes={row_bytes} T={T} M={len(ids)}", flush=True)
    cols = row_bytes // 2
    src = _random_bits(T * rows, cols, 45 + rows)
    out = rf.rf_gather_frames(src, ids, T, rows)
    dst = torch.full((T * rows, cols), 0x5A5A, dtype=torch.int16, device="cuda")
    before = dst.cpu().numpy()
    rf.rf_scatter_frames(out, dst, ids, T, rows)
    torch.cuda.synchronize()
    exp = oracle.gather_frames(src.cpu().numpy(), ids, rows)
    assert np.array_equal(out.cpu().numpy(), exp)
    assert np.array_equal(dst.cpu().numpy(), oracle.scatter_frames(exp, before, ids, rows))


@pytest.mark.parametrize("plane", [4, 1020, 1024, 1028, 2048 + 4])
def test_projection_planes_around_a_workgroup(plane):
    """fp32 planes of plane elements (4 per vector): 256 vectors per workgroup."""
    B, C, T = 2, 3, 5
    print(f"[case] projection plane={plane}", flush=True)
    g = torch.Generator(device="cuda").manual_seed(plane)
    lat = torch.randn((B, 2, C, T, 1, plane), generator=g, device="cuda")
    mask = np.array([1, 0, 0, 1, 0], dtype=np.uint8)
    ts = (24.0, 21.0, 23.0)
    out = rf.rf_project_latents(lat, ts, mask)
    torch.cuda.synchronize()
    exp = oracle.project_latents(lat.cpu(), B, C, T, 1, plane, ts, mask)
    assert_parity(_f64(out), exp, "f32", f"plane {plane}")
    # keyframe planes are slot 1 bit for bit
    assert torch.equal(out[:, :, 0], lat[:, 1, :, 0]) and torch.equal(out[:, :, 3], lat[:, 1, :, 3])
