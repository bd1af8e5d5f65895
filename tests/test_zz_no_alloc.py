"""rf_keyframe_attention_noalloc (the entry point for callers that cannot
allocate) against rf_keyframe_attention_ws, through the C ABI: two calls in a
row, the second with a smaller input (and the other head dimension), each
bit-identical to the workspace entry point on the same inputs (same plan, same
kernels), the smaller one also within the bf16 gates of the fp64 oracle; the
second call changes the device's free memory by nothing; a shape whose
split-key tail needs more than the static scratch is refused before any
launch."""
import pytest
import torch

import oracle
from paper_2606_06309_amd import workloads
from parity import assert_parity, torch_bf16_to_f64

pytestmark = pytest.mark.gpu

rf = pytest.importorskip("paper_2606_06309_amd.binding")


def _plan(w):
    return rf.rf_attention_plan(w.M, w.T, w.T, w.H, w.W, w.heads, w.head_dim, rf.RF_BF16)


def test_two_calls_match_the_workspace_entry_point():
    # the Wan2.1-1.3B shape (21 frames of 45 x 80, 12 heads x 128, 4 keyframes): 684 tiles, 172 split in
    # parts, about 153 MiB of the 160 MiB scratch; then a ragged head-dimension-64 case (18 frames of
    # 10 x 13, 3 heads, 3 keyframes: 6 tiles, every one split in 2)
    big = workloads.WORKLOADS["wan-1.3b"]
    small = workloads.custom(18, 10, 13, 3, 64, (1, 4, 7), dtype="bf16", seed=53)
    cases = []
    for w in (big, small):
        plan = _plan(w)
        print(f"[case] noalloc {w.name} T={w.T} N={w.N} heads={w.heads} d={w.head_dim} plan={plan}", flush=True)
        assert 0 < plan["workspace_bytes"] <= rf.RF_NOALLOC_SCRATCH_BYTES
        q, k, v = workloads.make_qkv(w, device="cuda")
        ref = rf.rf_keyframe_attention_ws(q, k, v, w.keyframes, w.T, w.H, w.W)
        out = torch.full_like(ref, float("nan"))
        cases.append((w, (q, k, v), ref, out))
    torch.cuda.synchronize()
    w, (q, k, v), _, out = cases[0]
    rf.rf_keyframe_attention_noalloc(q, k, v, w.keyframes, w.T, w.H, w.W, out=out)
    torch.cuda.synchronize()
    free_before = torch.cuda.mem_get_info()[0]
    w, (q, k, v), _, out = cases[1]
    rf.rf_keyframe_attention_noalloc(q, k, v, w.keyframes, w.T, w.H, w.W, out=out)
    torch.cuda.synchronize()
    assert torch.cuda.mem_get_info()[0] == free_before
    for w, (q, k, v), ref, out in cases:
        assert torch.equal(out, ref), w.name
    w, (q, k, v), _, out = cases[1]
    want = oracle.keyframe_attention(q.cpu(), k.cpu(), v.cpu(), w.keyframes, w.N)
    assert_parity(torch_bf16_to_f64(out), want, "bf16", "noalloc second call")


def test_more_than_the_static_scratch_is_refused():
    # one head, 14 frames of 64 x 64 all queried: 224 tiles, all past the last full round at 256
    # compute units, 896 key tiles: 8 parts each, 224 * 8 * 256 * 520 bytes = 228 MiB > 160 MiB
    w = workloads.custom(14, 64, 64, 1, 128, tuple(range(14)), dtype="bf16", seed=70)
    if torch.cuda.get_device_properties(0).multi_processor_count != 256:
        pytest.skip("the shape is sized for 256 compute units")
    plan = _plan(w)
    assert plan["workspace_bytes"] > rf.RF_NOALLOC_SCRATCH_BYTES
    q, k, v = workloads.make_qkv(w, device="cuda")
    out = torch.full((w.M * w.N, 1, 128), 3.0, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(rf.RhymeFlowError) as e:
        rf.rf_keyframe_attention_noalloc(q, k, v, w.keyframes, w.T, w.H, w.W, out=out)
    assert e.value.status == rf.RF_ERR_RANGE and "static scratch" in str(e.value)
    torch.cuda.synchronize()
    assert bool((out == 3.0).all())
