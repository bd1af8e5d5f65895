"""The Python binding never computes on the host: every call that launches work
rejects host tensors (and non-contiguous ones) with an error before anything
reaches the library, so there is no silent CPU path."""
import numpy as np
import pytest
import torch

rf = pytest.importorskip("paper_2606_06309_amd.binding")

T, H, W, HEADS, D = 3, 4, 4, 2, 64
S = T * H * W


def _qkv(dtype=torch.bfloat16):
    return tuple(torch.zeros((S, HEADS, D), dtype=dtype) for _ in range(3))


CALLS = {
    "keyframe_attention": lambda: rf.rf_keyframe_attention(*_qkv(), [0, 2], T, H, W),
    "keyframe_attention_ws": lambda: rf.rf_keyframe_attention_ws(*_qkv(), [0, 2], T, H, W),
    "frame_attention": lambda: rf.rf_frame_attention(*_qkv(), [0, 2], [0, 1], T, H, W),
    "project_latents": lambda: rf.rf_project_latents(torch.zeros((1, 2, 4, T, 8, 8)), (24.0, 21.0, 23.0),
                                                     np.array([1, 0, 1], dtype=np.uint8)),
    "gather_frames": lambda: rf.rf_gather_frames(torch.zeros((S, HEADS, D), dtype=torch.bfloat16), [0, 2], T, H * W),
    "scatter_frames": lambda: rf.rf_scatter_frames(torch.zeros((2 * H * W, HEADS, D), dtype=torch.bfloat16),
                                                   torch.zeros((S, HEADS, D), dtype=torch.bfloat16), [0, 2], T, H * W),
    "frame_similarity": lambda: rf.rf_frame_similarity(torch.zeros((1, 4, T, 8, 8))),
    "probe_mfma": lambda: rf.rf_probe_mfma_bf16(torch.zeros((12, 64, 8), dtype=torch.bfloat16), 1, 1,
                                                sink=torch.zeros(256)),
    "probe_hbm": lambda: rf.rf_probe_hbm_read(torch.zeros(4096, dtype=torch.uint8), 1,
                                              sink=torch.zeros(256, dtype=torch.int32)),
    "probe_lds": lambda: rf.rf_probe_lds_read(1, 1, 16, device="cpu"),
}


@pytest.mark.parametrize("name", sorted(CALLS))
def test_host_tensors_are_rejected(name):
    with pytest.raises((ValueError, TypeError)) as e:
        CALLS[name]()
    assert "device" in str(e.value)


def test_non_contiguous_is_rejected_before_the_device_check():
    x = torch.zeros((S, HEADS, D), dtype=torch.bfloat16).transpose(1, 2)
    with pytest.raises((ValueError, TypeError)):
        rf._dev(x, "x")
    with pytest.raises(TypeError):
        rf._dev(np.zeros(4), "x")


def test_probe_operand_shape_is_checked():
    with pytest.raises(ValueError, match="12 \\* 64 \\* 8"):
        rf.rf_probe_mfma_bf16(torch.zeros((16, 64, 8), dtype=torch.bfloat16), 1, 1)


# --- the rolling cache's buffers: sizes and dtypes checked before any launch --------

NK = [1, 2]            # cached frames of a T = 3 video, 16 rows of 128 elements each
ROWS, HID = H * W, HEADS * D


def _h(T_=T, dtype=torch.bfloat16, rows=ROWS):
    return torch.zeros((T_ * rows, HID), dtype=dtype)


def _store(n_frames=len(NK), dtype=torch.bfloat16):
    return torch.zeros((2 * n_frames * ROWS, HID), dtype=dtype)


@pytest.mark.parametrize("bad,err,match", [
    (dict(store=_store(1)), ValueError, "store is smaller"),
    (dict(h_full=_h(T_=T - 1)), ValueError, "h_full holds"),
    (dict(h_full=_h(dtype=torch.float32)), TypeError, "dtype"),
    (dict(store=None), ValueError, "needs a store"),
])
def test_cache_init_checks_buffers(bad, err, match):
    args = dict(store=_store(), h_full=_h())
    args.update(bad)
    with pytest.raises(err, match=match):
        rf.rf_cache_init(NK, T, ROWS, HID, torch.bfloat16, 10.0, **args)


def test_cache_init_right_sizes_reach_the_device_check():
    with pytest.raises(ValueError, match="device"):
        rf.rf_cache_init(NK, T, ROWS, HID, torch.bfloat16, 10.0, store=_store(), h_full=_h())


@pytest.mark.parametrize("bad,err,match", [
    (dict(store=_store(1)), ValueError, "store is smaller"),
    (dict(h_full=torch.zeros((T * ROWS + 1, HID), dtype=torch.bfloat16)), ValueError, "h_full holds"),
    (dict(h_full=_h(dtype=torch.float32)), TypeError, "dtype"),
])
def test_cache_shift_store_checks_buffers(bad, err, match):
    cache = rf.rf_cache_init(NK, T, ROWS, HID, torch.bfloat16, 10.0)   # bookkeeping only, no copy
    args = dict(store=_store(), h_full=_h())
    args.update(bad)
    with pytest.raises(err, match=match):
        rf.rf_cache_shift_store(cache, 8.0, **args)
    assert cache.t_after[1] == 10.0   # nothing changed
