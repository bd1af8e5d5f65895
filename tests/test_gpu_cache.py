"""GPU parity of the rolling cache (App. B.2) through the C ABI against the
oracle's RollingCache: the store copies of initialisation and shift-and-store
(bit-exact), the projected keys and values at skipped steps (element-wise
bound below), the keyframe rows left untouched, K = V on the projected frames,
and keyframe-query attention over the assembled keys and values.

Element-wise bound of the projection, from its arithmetic: alpha is rounded
once to float (relative 2^-24), 1 - alpha and the product (1 - alpha) h_before
round once each, the fma once, so the fp32 value is within
4 * 2^-24 * max(|h_before|, |h_after|) = 2^-22 * max of the exact one; a bf16
result then rounds once more (relative 2^-8). The gates:
  fp32: |out - ref| <= 2^-22 * max(|h_before|, |h_after|)
  bf16: |out - ref| <= 2^-8 * |ref| + 2^-21 * max(|h_before|, |h_after|)
"""
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


def _check_projection(out, ref, hb, ha, dtype, what):
    out = np.asarray(out, np.float64)
    scale = np.maximum(np.abs(hb), np.abs(ha))
    if dtype == torch.bfloat16:
        bound = 2.0 ** -8 * np.abs(ref) + 2.0 ** -21 * scale
    else:
        bound = 2.0 ** -22 * scale
    err = np.abs(out - ref)
    bad = err > bound
    assert np.isfinite(out).all(), what
    assert not bad.any(), f"{what}: {int(bad.sum())} elements over the bound, worst {float((err - bound).max())}"


def _nonkeys(w):
    return [f for f in range(w.T) if f not in w.keyframes]


# frame sizes in 16-byte vectors against the kernels' 64-vector (one wave) blocks
SMALL = [
    workloads.WORKLOADS["tiny"],                                          # fp32, 2 x 64: 2048 vectors a frame
    workloads.custom(7, 6, 10, 1, 64, (0, 4), dtype="bf16", seed=31),     # 480 vectors: 7.5 blocks
    workloads.custom(9, 5, 7, 2, 128, (0, 3, 8), dtype="bf16", seed=32),  # N = 35: 1120 vectors, 17.5 blocks
    workloads.WORKLOADS["small"],                                         # 12 x 128: 299,520 vectors a frame
    workloads.custom(4, 1, 1, 1, 64, (0,), dtype="bf16", seed=33),        # one token: 8 vectors, under a block
    workloads.custom(5, 1, 13, 1, 64, (0, 2), dtype="bf16", seed=34),     # 104 vectors: 1.6 blocks
]


def _make_store(w, n, fill=0.0):
    nbytes = rf.rf_cache_store_bytes(n, w.N, w.heads * w.head_dim, w.torch_dtype)
    el = torch.tensor([], dtype=w.torch_dtype).element_size()
    return torch.full((nbytes // el,), fill, dtype=w.torch_dtype, device="cuda")


@pytest.mark.parametrize("w", SMALL, ids=lambda w: w.name + f"_T{w.T}")
def test_store_copies_bit_exact(w):
    print(f"[case] cache store copies {w.name} T={w.T} N={w.N} D={w.heads * w.head_dim}", flush=True)
    nk = _nonkeys(w)
    D = w.heads * w.head_dim
    store = _make_store(w, len(nk), fill=-7.0)
    h0 = workloads.make_hidden(w, 0, device="cuda")
    c = rf.rf_cache_init(nk, w.T, w.N, D, w.torch_dtype, 40.0, store=store, h_full=h0)
    torch.cuda.synchronize()
    st = store.view(2 * len(nk), w.N, D)
    hb = h0.view(w.T, w.N, D)
    for i, f in enumerate(nk):
        assert c.before_slot[f] == c.after_slot[f] == 2 * i
        assert torch.equal(_bits_t(st[2 * i]), _bits_t(hb[f]))
        assert bool((st[2 * i + 1] == -7.0).all())          # the other slot is not written
    h1 = workloads.make_hidden(w, 1, device="cuda")
    rf.rf_cache_shift_store(c, 37.0, store=store, h_full=h1)
    torch.cuda.synchronize()
    h1f = h1.view(w.T, w.N, D)
    for i, f in enumerate(nk):
        assert c.before_slot[f] == 2 * i and c.after_slot[f] == 2 * i + 1
        assert torch.equal(_bits_t(st[2 * i]), _bits_t(hb[f]))
        assert torch.equal(_bits_t(st[2 * i + 1]), _bits_t(h1f[f]))
    # a partial shift: only the first cached frame moves on
    h2 = workloads.make_hidden(w, 2, device="cuda")
    rf.rf_cache_shift_store(c, 34.0, store=store, h_full=h2, frames=nk[:1])
    torch.cuda.synchronize()
    assert c.before_slot[nk[0]] == 1 and c.after_slot[nk[0]] == 0
    assert torch.equal(_bits_t(st[0]), _bits_t(h2.view(w.T, w.N, D)[nk[0]]))
    if len(nk) > 1:
        assert torch.equal(_bits_t(st[3]), _bits_t(h1f[nk[1]]))


def _bits_t(t):
    return t.contiguous().view(torch.int16 if t.dtype == torch.bfloat16 else torch.int32)


def _run_sequence(w, t_w, shifts, skips):
    """Drives the GPU cache and the oracle's through one schedule; at every
    skipped step compares k and v of all frames with the oracle's."""
    nk = _nonkeys(w)
    D = w.heads * w.head_dim
    store = _make_store(w, len(nk))
    q, k, v = workloads.make_qkv(w, device="cuda")
    k_in, v_in = k.cpu().clone(), v.cpu().clone()
    k0, v0 = _bits(k), _bits(v)
    ref = oracle.RollingCache()
    h = workloads.make_hidden(w, 0, device="cuda")
    c = rf.rf_cache_init(nk, w.T, w.N, D, w.torch_dtype, t_w, store=store, h_full=h)
    hc = _f64(h).reshape(w.T, w.N, D)
    ref.init(nk, {f: hc[f] for f in nk}, t_w)
    for si, t_d in enumerate([None] + list(shifts)):
        if t_d is not None:
            h = workloads.make_hidden(w, si, device="cuda")
            rf.rf_cache_shift_store(c, t_d, store=store, h_full=h)
            hc = _f64(h).reshape(w.T, w.N, D)
            ref.shift_and_store(nk, {f: hc[f] for f in nk}, t_d)
        for t_s in skips[si]:
            print(f"[case] cache projection {w.name} after store {si} at t={t_s}", flush=True)
            rf.rf_cache_project_kv(c, store, k, v, t_s)
            torch.cuda.synchronize()
            kk, vv = _bits(k), _bits(v)
            for f in w.keyframes:     # keyframe rows keep their keys and values
                sl = slice(f * w.N, (f + 1) * w.N)
                assert np.array_equal(kk[sl], k0[sl]) and np.array_equal(vv[sl], v0[sl])
            kf = _f64(k).reshape(w.T, w.N, D)
            for f in nk:
                sl = slice(f * w.N, (f + 1) * w.N)
                assert np.array_equal(kk[sl], vv[sl])          # K = V on projected frames
                _check_projection(kf[f], ref.project(f, t_s), ref.h_before[f], ref.h_after[f],
                                  w.torch_dtype, f"{w.name} frame {f} t={t_s}")
                assert rf.rf_cache_alpha(c, f, t_s) == oracle.hidden_alpha(ref.t_before[f], ref.t_after[f], t_s)
    return c, store, q, k, v, ref, k_in, v_in


@pytest.mark.parametrize("w", SMALL, ids=lambda w: w.name + f"_T{w.T}")
def test_projection_sequence(w):
    _run_sequence(w, 40.0, [37.0, 34.0, 31.5],
                  [[39.0, 40.0], [38.5, 37.0, 40.0], [36.0, 35.2, 30.0], [33.0, 32.75]])


def test_projection_endpoints_bit_exact():
    """alpha = 0 at t_before and alpha = 1 past t_after (and straight after
    initialisation) return the cached states bit for bit."""
    w = SMALL[1]
    nk = _nonkeys(w)
    D = w.heads * w.head_dim
    store = _make_store(w, len(nk))
    q, k, v = workloads.make_qkv(w, device="cuda")
    h0 = workloads.make_hidden(w, 0, device="cuda")
    h1 = workloads.make_hidden(w, 1, device="cuda")
    c = rf.rf_cache_init(nk, w.T, w.N, D, w.torch_dtype, 40.0, store=store, h_full=h0)
    rf.rf_cache_project_kv(c, store, k, v, 39.0)
    torch.cuda.synchronize()
    for f in nk:
        sl = slice(f * w.N, (f + 1) * w.N)
        assert torch.equal(_bits_t(k[sl]), _bits_t(h0[sl]))
    rf.rf_cache_shift_store(c, 37.0, store=store, h_full=h1)
    for t_s, h in [(40.0, h0), (36.0, h1)]:
        rf.rf_cache_project_kv(c, store, k, v, t_s)
        torch.cuda.synchronize()
        for f in nk:
            sl = slice(f * w.N, (f + 1) * w.N)
            assert torch.equal(_bits_t(k[sl]), _bits_t(h[sl])) and torch.equal(_bits_t(v[sl]), _bits_t(h[sl]))


def test_projection_frame_subset():
    w = SMALL[2]
    nk = _nonkeys(w)
    D = w.heads * w.head_dim
    store = _make_store(w, len(nk))
    q, k, v = workloads.make_qkv(w, device="cuda")
    before = _bits(k)
    c = rf.rf_cache_init(nk, w.T, w.N, D, w.torch_dtype, 40.0, store=store,
                         h_full=workloads.make_hidden(w, 0, device="cuda"))
    rf.rf_cache_shift_store(c, 37.0, store=store, h_full=workloads.make_hidden(w, 1, device="cuda"))
    sub = nk[1::2]
    rf.rf_cache_project_kv(c, store, k, v, 38.0, frames=sub)
    torch.cuda.synchronize()
    kk = _bits(k)
    for f in range(w.T):
        sl = slice(f * w.N, (f + 1) * w.N)
        assert np.array_equal(kk[sl], before[sl]) == (f not in sub), f


@pytest.mark.parametrize("w,kind", [(SMALL[0], "f32"), (SMALL[2], "bf16"),
                                    (workloads.custom(6, 8, 16, 2, 128, (0, 3), dtype="bf16", seed=33), "bf16")],
                         ids=["tiny_f32", "T9_bf16", "T6_bf16"])
def test_attention_over_projected_kv(w, kind):
    """Keyframe-query attention at a skipped step: keyframes keep their K/V,
    non-keyframes contribute the projected hidden state as key and value."""
    c, store, q, k, v, ref, k_in, v_in = _run_sequence(w, 40.0, [37.0], [[], [38.0]])
    out = rf.rf_keyframe_attention(q, k, v, list(w.keyframes), w.T, w.H, w.W)
    torch.cuda.synchronize()
    K, V = oracle.skip_step_kv(k_in, v_in, ref, _nonkeys(w), 38.0, w.N)
    exp = oracle.keyframe_attention(oracle.as_oracle_f64(q.cpu()), K, V, list(w.keyframes), w.N)
    assert_parity(_f64(out), exp, kind, f"{w.name} attention over projected K/V")


def test_long_workload_sampled():
    """33 frames of 45 x 80 tokens, 24 heads x 128 (25 cached frames, 1.1 GB
    store): sampled rows of every cached frame against the oracle."""
    w = workloads.WORKLOADS["long"]
    nk = _nonkeys(w)
    D = w.heads * w.head_dim
    print(f"[case] cache long workload: {len(nk)} cached frames", flush=True)
    store = _make_store(w, len(nk))
    k = torch.zeros((w.S, w.heads, w.head_dim), dtype=w.torch_dtype, device="cuda")
    v = torch.zeros_like(k)
    h0 = workloads.make_hidden(w, 0, device="cuda")
    c = rf.rf_cache_init(nk, w.T, w.N, D, w.torch_dtype, 24.0, store=store, h_full=h0)
    h1 = workloads.make_hidden(w, 1, device="cuda")
    rf.rf_cache_shift_store(c, 21.0, store=store, h_full=h1)
    rf.rf_cache_project_kv(c, store, k, v, 23.0)
    torch.cuda.synchronize()
    rows = np.sort(np.random.default_rng(5).choice(w.N, 64, replace=False))
    rows = np.unique(np.concatenate([rows, [0, w.N - 1]]))
    ref = oracle.RollingCache()
    h0c = h0.view(w.T, w.N, D)
    h1c = h1.view(w.T, w.N, D)
    ridx = torch.as_tensor(rows, device="cuda")
    ref.init(nk, {f: _f64(h0c[f][ridx]) for f in nk}, 24.0)
    ref.shift_and_store(nk, {f: _f64(h1c[f][ridx]) for f in nk}, 21.0)
    kf = k.view(w.T, w.N, D)
    vf = v.view(w.T, w.N, D)
    for f in nk:
        got = kf[f][ridx]
        assert torch.equal(_bits_t(got), _bits_t(vf[f][ridx]))
        _check_projection(_f64(got), ref.project(f, 23.0), ref.h_before[f], ref.h_after[f],
                          w.torch_dtype, f"long frame {f}")
    for f in w.keyframes:
        assert not bool((kf[f] != 0).any()) and not bool((vf[f] != 0).any())   # untouched zeros
