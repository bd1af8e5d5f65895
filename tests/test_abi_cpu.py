"""The C ABI on a host without a GPU: the library loads, exports every symbol
the header declares, the host-only keyframe calls agree bit for bit with the
oracle, and every invalid argument is rejected before any HIP call."""
import ctypes
import math
import os
import re

import numpy as np
import pytest
import torch

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "rhymeflow.h")

rf = pytest.importorskip("paper_2606_06309_amd.binding")
lib = rf.lib

_i32p = ctypes.POINTER(ctypes.c_int32)
_u8p = ctypes.POINTER(ctypes.c_uint8)


def _header_text():
    with open(HEADER) as f:
        return f.read()


def test_every_declared_symbol_is_exported():
    text = _header_text()
    declared = set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(rf_\w+)\s*\(", text, re.M))
    assert {"rf_keyframe_attention", "rf_project_latents", "rf_select_keyframes"} <= declared
    assert declared == set(rf.EXPORTED)
    for name in declared:
        assert hasattr(lib, name), name


def test_header_constants_match_binding():
    text = _header_text()
    assert int(re.search(r"#define RF_ABI_VERSION (\d+)", text).group(1)) == rf.abi_version()
    assert int(re.search(r"#define RF_MAX_FRAMES (\d+)", text).group(1)) == rf.RF_MAX_FRAMES
    for name in ["RF_OK", "RF_ERR_INVALID_ARG", "RF_ERR_UNSUPPORTED", "RF_ERR_RANGE", "RF_ERR_HIP",
                 "RF_BF16", "RF_F32"]:
        val = int(re.search(name + r"\s*=\s*(-?\d+)", text).group(1))
        assert getattr(rf, name) == val, name


def test_status_strings():
    for code, name in [(0, "RF_OK"), (-1, "RF_ERR_INVALID_ARG"), (-2, "RF_ERR_UNSUPPORTED"),
                       (-3, "RF_ERR_RANGE"), (-4, "RF_ERR_HIP")]:
        assert lib.rf_status_string(code).decode() == name
    assert lib.rf_status_string(7).decode() == "RF_UNKNOWN_STATUS"


# --- host-only keyframe calls: bit-exact against the oracle -------------------------

def test_select_matches_oracle_exhaustively():
    rng = np.random.default_rng(5)
    for T in list(range(1, 12)) + [33, 256]:
        for _ in range(40):
            n = int(rng.integers(0, min(T, 8) + 1))
            ids = rng.integers(0, T, size=n).tolist()
            for force in (True, False):
                if not force and not ids:
                    continue
                got, mask = rf.rf_select_keyframes(ids, T, force_first=force)
                exp = oracle.select_keyframes(ids, T, force_first=force)
                assert got.tolist() == exp.tolist()
                assert mask.tolist() == oracle.keyframe_mask(exp, T).tolist()


def test_policies_match_oracle():
    for T in range(1, 60):
        for k in range(1, T + 2):
            assert rf.rf_keyframes_stride(T, k).tolist() == oracle.stride_keyframes(T, k).tolist()
        for M in range(1, T + 1):
            assert rf.rf_keyframes_uniform(T, M).tolist() == oracle.uniform_keyframes(T, M).tolist()


@pytest.mark.parametrize("call", [
    lambda: rf.rf_select_keyframes([5], 5),
    lambda: rf.rf_select_keyframes([-1], 5),
    lambda: rf.rf_select_keyframes([0], 257),
    lambda: rf.rf_select_keyframes([], 4, force_first=False),
    lambda: rf.rf_keyframes_stride(5, 0),
    lambda: rf.rf_keyframes_stride(0, 1),
    lambda: rf.rf_keyframes_uniform(5, 6),
    lambda: rf.rf_keyframes_uniform(5, 0),
])
def test_keyframe_call_errors(call):
    with pytest.raises(rf.RhymeFlowError) as e:
        call()
    assert e.value.status in (rf.RF_ERR_INVALID_ARG, rf.RF_ERR_RANGE)
    assert lib.rf_last_error().decode()


def test_select_null_outputs():
    ids = (ctypes.c_int32 * 1)(0)
    n = ctypes.c_int32()
    assert lib.rf_select_keyframes(ids, 1, 4, 0, None, ctypes.byref(n), None) == rf.RF_ERR_INVALID_ARG
    out = (ctypes.c_int32 * 4)()
    assert lib.rf_select_keyframes(ids, 1, 4, 0x10, out, ctypes.byref(n), None) == rf.RF_ERR_INVALID_ARG


# --- device calls: rejected before any HIP call ------------------------------------

A = 0x10000000   # fake, 16-byte aligned addresses; never dereferenced
B_ = 0x20000000
C_ = 0x30000000
O_ = 0x40000000


def _attn(q=A, k=B_, v=C_, out=O_, ids=(0, 2, 4), M=None, T=5, H=8, W=8, heads=2, d=64,
          dtype=rf.RF_BF16):
    arr = (ctypes.c_int32 * max(1, len(ids)))(*ids)
    M = len(ids) if M is None else M
    return lib.rf_keyframe_attention(q, k, v, out, arr if ids is not None else None, M, T, H, W,
                                     heads, d, dtype, None)


@pytest.mark.parametrize("kwargs,status", [
    (dict(q=0), rf.RF_ERR_INVALID_ARG),
    (dict(out=0), rf.RF_ERR_INVALID_ARG),
    (dict(H=0), rf.RF_ERR_INVALID_ARG),
    (dict(heads=-1), rf.RF_ERR_INVALID_ARG),
    (dict(ids=(0, 4, 2)), rf.RF_ERR_INVALID_ARG),
    (dict(ids=(0, 2, 2)), rf.RF_ERR_INVALID_ARG),
    (dict(ids=(0, 5)), rf.RF_ERR_RANGE),
    (dict(ids=(-1, 2)), rf.RF_ERR_RANGE),
    (dict(ids=(0,), M=0), rf.RF_ERR_INVALID_ARG),
    (dict(ids=(0, 1, 2, 3, 4, 5), T=5), rf.RF_ERR_RANGE),
    (dict(T=257, ids=(0,)), rf.RF_ERR_RANGE),
    (dict(d=96), rf.RF_ERR_UNSUPPORTED),
    (dict(d=256), rf.RF_ERR_UNSUPPORTED),
    (dict(dtype=7), rf.RF_ERR_UNSUPPORTED),
    (dict(q=A + 8), rf.RF_ERR_UNSUPPORTED),
    (dict(out=A + 1024), rf.RF_ERR_INVALID_ARG),       # out overlaps q
])
def test_attention_validation(kwargs, status):
    assert _attn(**kwargs) == status
    assert lib.rf_last_error().decode().startswith("rf_keyframe_attention")


def _fattn(q=A, k=B_, v=C_, out=O_, ids=(0, 2, 4), kv=(0, 2, 4), T=5, H=8, W=8, heads=2, d=64,
           dtype=rf.RF_BF16):
    arr = (ctypes.c_int32 * max(1, len(ids)))(*ids)
    kva = (ctypes.c_int32 * max(1, len(kv)))(*kv) if kv is not None else None
    return lib.rf_frame_attention(q, k, v, out, arr, len(ids), kva, 0 if kv is None else len(kv), T, H, W,
                                  heads, d, dtype, None, 0, None)


@pytest.mark.parametrize("kwargs,status", [
    (dict(kv=None), rf.RF_ERR_INVALID_ARG),
    (dict(kv=()), rf.RF_ERR_INVALID_ARG),
    (dict(kv=(2, 2)), rf.RF_ERR_INVALID_ARG),
    (dict(kv=(3, 1)), rf.RF_ERR_INVALID_ARG),
    (dict(kv=(0, 5)), rf.RF_ERR_RANGE),
    (dict(kv=(0, 1, 2, 3, 4, 5)), rf.RF_ERR_RANGE),
    (dict(ids=(4, 1)), rf.RF_ERR_INVALID_ARG),
    (dict(d=96), rf.RF_ERR_UNSUPPORTED),
    (dict(k=B_ + 8), rf.RF_ERR_UNSUPPORTED),
    (dict(out=A + 64), rf.RF_ERR_INVALID_ARG),
])
def test_frame_attention_validation(kwargs, status):
    assert _fattn(**kwargs) == status
    assert lib.rf_last_error().decode().startswith("rf_frame_attention")


def test_attention_workspace_sizes():
    # 2,712 tiles of 256 rows at 33 x 45 x 80, 24 heads: 152 beyond 10 rounds, split in 5
    assert rf.rf_attention_workspace(8, 33, 33, 45, 80, 24, 128, rf.RF_BF16, 256) == 152 * 5 * 256 * (128 * 4 + 8)
    # 40 heads, 6 keyframes of 45 x 80: 3,400 tiles, 72 beyond 13 rounds, split in 7
    assert rf.rf_attention_workspace(6, 21, 21, 45, 80, 40, 128, rf.RF_BF16, 256) == 72 * 7 * 256 * 520
    # whole rounds need nothing; fp32 never splits; too few key tiles to split
    assert rf.rf_attention_workspace(8, 33, 33, 48, 64, 24, 128, rf.RF_BF16, 256) == 0
    assert rf.rf_attention_workspace(8, 33, 33, 45, 80, 24, 128, rf.RF_F32, 256) == 0
    assert rf.rf_attention_workspace(3, 5, 5, 8, 8, 2, 64, rf.RF_BF16, 256) == 0
    n = ctypes.c_int64(0)
    for args, status in [((0, 5, 5, 8, 8, 2, 64, 0, 256), rf.RF_ERR_INVALID_ARG),
                         ((6, 5, 5, 8, 8, 2, 64, 0, 256), rf.RF_ERR_RANGE),
                         ((2, 5, 5, 8, 8, 2, 96, 0, 256), rf.RF_ERR_UNSUPPORTED),
                         ((2, 5, 300, 8, 8, 2, 64, 0, 256), rf.RF_ERR_RANGE),
                         ((2, 5, 5, 8, 8, 2, 64, 0, -1), rf.RF_ERR_RANGE),
                         ((2, 5, 5, 8, 8, 2, 64, 0, 65537), rf.RF_ERR_RANGE)]:
        assert lib.rf_attention_workspace(*args, ctypes.byref(n)) == status
    assert lib.rf_attention_workspace(2, 5, 5, 8, 8, 2, 64, 0, 256, None) == rf.RF_ERR_INVALID_ARG


# The split plan of the long workload (33 frames of 45 x 80, 24 heads x 128, 8
# keyframes: 28,800 query rows = 113 tiles of 256 per head, 2,712 tiles; 118,800
# keys = 1,857 tiles of 64) on three device sizes, worked by hand. s parts of
# each of the t tail tiles take ceil(t * s / CUs) / s rounds (s = 1: one round);
# the smallest s of the least cost wins, parts need >= 8 key tiles, s <= 8.
#   256 CUs: t = 2712 - 10 * 256 = 152; s = 2..8 cost 1, 2/3, 3/4, 3/5, 2/3, 5/7, 5/8 -> s = 5, 372 key tiles a part
#   128 CUs: t = 2712 - 21 * 128 = 24; s = 5 fits 120 parts in one round (1/5); s = 6..8 need two -> s = 5
#    80 CUs: t = 2712 - 33 * 80 = 72; every s needs s rounds (72 s / 80 > s - 1) -> cost 1, no split
LONG_PLANS = {
    256: dict(tiles=2712, whole_tiles=2560, tail_tiles=152, parts=5, key_tiles_per_part=372,
              workspace_bytes=152 * 5 * 256 * 520, compute_units=256),
    128: dict(tiles=2712, whole_tiles=2688, tail_tiles=24, parts=5, key_tiles_per_part=372,
              workspace_bytes=24 * 5 * 256 * 520, compute_units=128),
    80: dict(tiles=2712, whole_tiles=2712, tail_tiles=0, parts=0, key_tiles_per_part=0,
             workspace_bytes=0, compute_units=80),
}


@pytest.mark.parametrize("cus", sorted(LONG_PLANS))
def test_attention_plan_by_compute_units(cus):
    plan = rf.rf_attention_plan(8, 33, 33, 45, 80, 24, 128, rf.RF_BF16, cus)
    assert plan == LONG_PLANS[cus]
    assert rf.rf_attention_workspace(8, 33, 33, 45, 80, 24, 128, rf.RF_BF16, cus) == plan["workspace_bytes"]


def test_attention_plan_head_dim_64_and_fp32():
    # the CogVideoX-v1.5 shape (11 frames of 48 x 85, 48 heads x 64, 4 keyframes): 16,320 rows =
    # 64 tiles per head, 3,072 tiles = 12 whole rounds of 256: nothing to split; on 100 CUs
    # 72 tiles remain, 44,880 keys are 351 tiles of 128: s = 4 puts 288 parts in 3 rounds (3/4)
    assert rf.rf_attention_plan(4, 11, 11, 48, 85, 48, 64, rf.RF_BF16, 256)["parts"] == 0
    p = rf.rf_attention_plan(4, 11, 11, 48, 85, 48, 64, rf.RF_BF16, 100)
    assert (p["tail_tiles"], p["parts"], p["key_tiles_per_part"]) == (72, 4, 88)
    assert p["workspace_bytes"] == 72 * 4 * 256 * (64 * 4 + 8)
    f = rf.rf_attention_plan(4, 11, 11, 48, 85, 48, 64, rf.RF_F32, 256)
    assert f == dict(tiles=0, whole_tiles=0, tail_tiles=0, parts=0, key_tiles_per_part=0,
                     workspace_bytes=0, compute_units=256)


def test_attention_plan_of_the_current_device_needs_one():
    if _gpu_present():
        pytest.skip("a device is present")
    n = ctypes.c_int64(0)
    assert lib.rf_attention_workspace(8, 33, 33, 45, 80, 24, 128, rf.RF_BF16, 0, ctypes.byref(n)) == rf.RF_ERR_HIP
    assert "cannot query" in lib.rf_last_error().decode()


def _gpu_present():
    try:
        return torch.cuda.is_available()
    except Exception:
        return False


def _attn_ws(ws=0x50000000, ws_bytes=1 << 30, T=8, H=16, W=16, heads=2, d=128, ids=(0, 5), out=O_):
    arr = (ctypes.c_int32 * len(ids))(*ids)
    return lib.rf_keyframe_attention_ws(A, B_, C_, out, arr, len(ids), T, H, W, heads, d, rf.RF_BF16,
                                        ws, ws_bytes, None)


@pytest.mark.parametrize("kwargs,status", [
    (dict(ws=0), rf.RF_ERR_INVALID_ARG),
    (dict(ws_bytes=-1), rf.RF_ERR_INVALID_ARG),
    (dict(ws=0x50000008), rf.RF_ERR_UNSUPPORTED),
    (dict(ws=A + 64), rf.RF_ERR_INVALID_ARG),          # workspace inside q
    (dict(ws=O_ - 64), rf.RF_ERR_INVALID_ARG),         # workspace running into out
])
def test_attention_ws_validation(kwargs, status):
    # (a workspace smaller than the device's plan needs is checked after the device
    # query; its GPU test is in tests/test_gpu_limits.py)
    assert rf.rf_attention_workspace(2, 8, 8, 16, 16, 2, 128, rf.RF_BF16, 256) > 0
    assert _attn_ws(**kwargs) == status
    assert lib.rf_last_error().decode().startswith("rf_keyframe_attention_ws")


def _proj(lat=A, out=B_, ts=(24.0, 21.0, 23.0), mask=(1, 0, 1, 0, 1), B=1, C=4, T=5, Hl=16,
          Wl=16, dtype=rf.RF_F32):
    t = (ctypes.c_double * 3)(*ts)
    m = (ctypes.c_uint8 * max(1, len(mask)))(*mask)
    return lib.rf_project_latents(lat, out, t, m, B, C, T, Hl, Wl, dtype, None)


@pytest.mark.parametrize("kwargs,status", [
    (dict(lat=0), rf.RF_ERR_INVALID_ARG),
    (dict(out=0), rf.RF_ERR_INVALID_ARG),
    (dict(C=0), rf.RF_ERR_INVALID_ARG),
    (dict(ts=(24.0, math.nan, 23.0)), rf.RF_ERR_INVALID_ARG),
    (dict(ts=(math.inf, 21.0, 23.0)), rf.RF_ERR_INVALID_ARG),
    (dict(T=300, mask=(0,) * 300), rf.RF_ERR_RANGE),
    (dict(dtype=3), rf.RF_ERR_UNSUPPORTED),
    (dict(out=B_ + 4), rf.RF_ERR_UNSUPPORTED),
    (dict(out=A + 16), rf.RF_ERR_INVALID_ARG),           # partial overlap
    (dict(out=A + 4 * 5 * 256 * 4, B=2), rf.RF_ERR_INVALID_ARG),  # slot-1 alias needs B == 1
])
def test_projection_validation(kwargs, status):
    assert _proj(**kwargs) == status
    assert lib.rf_last_error().decode().startswith("rf_project_latents")


def test_projection_null_timesteps():
    m = (ctypes.c_uint8 * 5)()
    assert lib.rf_project_latents(A, B_, None, m, 1, 4, 5, 16, 16, rf.RF_F32, None) == rf.RF_ERR_INVALID_ARG


@pytest.mark.parametrize("fn", ["rf_gather_frames", "rf_scatter_frames"])
@pytest.mark.parametrize("args,status", [
    (dict(src=0), rf.RF_ERR_INVALID_ARG),
    (dict(ids=(1, 0)), rf.RF_ERR_INVALID_ARG),
    (dict(ids=(0, 9)), rf.RF_ERR_RANGE),
    (dict(rows=0), rf.RF_ERR_INVALID_ARG),
    (dict(row_bytes=24), rf.RF_ERR_UNSUPPORTED),
    (dict(dst=B_ + 8), rf.RF_ERR_UNSUPPORTED),
    (dict(dst=A + 16), rf.RF_ERR_INVALID_ARG),
])
def test_frame_copy_validation(fn, args, status):
    a = dict(src=A, dst=B_, ids=(0, 2), T=5, rows=64, row_bytes=256)
    a.update(args)
    ids = (ctypes.c_int32 * len(a["ids"]))(*a["ids"])
    got = getattr(lib, fn)(a["src"], a["dst"], ids, len(a["ids"]), a["T"], a["rows"],
                           a["row_bytes"], None)
    assert got == status


@pytest.mark.parametrize("args,status", [
    (dict(ops=None), rf.RF_ERR_INVALID_ARG),
    (dict(sink=None), rf.RF_ERR_INVALID_ARG),
    (dict(wg=0), rf.RF_ERR_RANGE),
    (dict(wg=(1 << 20) + 1), rf.RF_ERR_RANGE),
    (dict(rounds=0), rf.RF_ERR_RANGE),
    (dict(rounds=(1 << 22) + 1), rf.RF_ERR_RANGE),
    (dict(ops=A + 8), rf.RF_ERR_UNSUPPORTED),
    (dict(sink=B_ + 2), rf.RF_ERR_UNSUPPORTED),
])
def test_mfma_probe_validation(args, status):
    a = dict(ops=A, wg=4, rounds=8, sink=B_)
    a.update(args)
    assert lib.rf_probe_mfma_bf16(a["ops"], a["wg"], a["rounds"], a["sink"], None) == status


@pytest.mark.parametrize("args,status", [
    (dict(src=None), rf.RF_ERR_INVALID_ARG),
    (dict(sink=None), rf.RF_ERR_INVALID_ARG),
    (dict(nbytes=0), rf.RF_ERR_INVALID_ARG),
    (dict(nbytes=24), rf.RF_ERR_INVALID_ARG),
    (dict(nbytes=-16), rf.RF_ERR_INVALID_ARG),
    (dict(wg=0), rf.RF_ERR_RANGE),
    (dict(src=A + 8), rf.RF_ERR_UNSUPPORTED),
    (dict(sink=B_ + 1), rf.RF_ERR_UNSUPPORTED),
])
def test_hbm_probe_validation(args, status):
    a = dict(src=A, nbytes=4096, wg=4, sink=B_)
    a.update(args)
    assert lib.rf_probe_hbm_read(a["src"], a["nbytes"], a["wg"], a["sink"], None) == status


@pytest.mark.parametrize("args,status", [
    (dict(sink=None), rf.RF_ERR_INVALID_ARG),
    (dict(width=4), rf.RF_ERR_INVALID_ARG),
    (dict(width=32), rf.RF_ERR_INVALID_ARG),
    (dict(wg=0), rf.RF_ERR_RANGE),
    (dict(wg=(1 << 20) + 1), rf.RF_ERR_RANGE),
    (dict(rounds=0), rf.RF_ERR_RANGE),
    (dict(rounds=(1 << 22) + 1), rf.RF_ERR_RANGE),
    (dict(sink=B_ + 2), rf.RF_ERR_UNSUPPORTED),
    (dict(ticks=A + 4), rf.RF_ERR_UNSUPPORTED),
])
def test_lds_probe_validation(args, status):
    a = dict(wg=4, rounds=8, width=16, sink=B_, ticks=A)
    a.update(args)
    assert lib.rf_probe_lds_read(a["wg"], a["rounds"], a["width"], a["sink"], a["ticks"], None) == status


def test_sizes_overflowing_byte_counts_are_range_errors():
    """Sizes whose byte counts would pass 64 bits are rejected before any is
    formed in integers (and before any HIP call)."""
    big = 2 ** 31 - 1
    ids = (ctypes.c_int32 * 2)(0, 1)
    assert lib.rf_keyframe_attention(A, B_, A + 4096, B_ + 4096, ids, 2, 4, big, big, 8, 128,
                                     rf.RF_BF16, None) == rf.RF_ERR_RANGE
    n = ctypes.c_int64(0)
    assert lib.rf_attention_workspace(2, 4, 4, big, big, 8, 128, rf.RF_BF16, 256, ctypes.byref(n)) == rf.RF_ERR_RANGE
    m = (ctypes.c_uint8 * 5)(1, 0, 1, 0, 1)
    ts = (ctypes.c_double * 3)(24.0, 21.0, 23.0)
    assert lib.rf_project_latents(A, B_, ts, m, big, 16, 5, big, 16, rf.RF_F32, None) == rf.RF_ERR_RANGE
    for fn in (lib.rf_gather_frames, lib.rf_scatter_frames):
        assert fn(A, B_, ids, 2, 4, 2 ** 40, 2 ** 32, None) == rf.RF_ERR_RANGE
