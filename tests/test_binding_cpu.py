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
