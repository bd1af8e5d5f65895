"""Pins of the oracle's frame-masked attention (the frame-level mask M_Rhyme;
Sec. 4's keyframe-only / "w/o projection" ablations): the unmasked case is
the keyframe-query attention, a dense masked softmax written with an explicit
-inf mask matrix agrees, masked frames cannot influence the result (NaN keys
and values there leave it bit-identical), single-frame cases reduce to torch's
attention, and the key order inside the mask does not matter."""
import numpy as np
import pytest
import torch

import oracle


def _qkv(T, N, heads, d, seed):
    rng = np.random.default_rng(seed)
    return tuple(rng.standard_normal((T * N, heads, d)) for _ in range(3))


def test_unmasked_equals_keyframe_attention():
    q, k, v = _qkv(5, 6, 2, 8, 0)
    a = oracle.frame_attention(q, k, v, [0, 2, 4], list(range(5)), 6)
    b = oracle.keyframe_attention(q, k, v, [0, 2, 4], 6)
    assert np.array_equal(a, b)


def _masked_softmax_reference(q, k, v, q_frames, kv_frames, N):
    """Dense formulation: scores over all keys, -inf where the key's frame is
    masked, softmax, weighted sum (numpy, per head)."""
    S, heads, d = k.shape
    key_frame = np.arange(S) // N
    allowed = np.isin(key_frame, kv_frames)
    qt = oracle.rowmap(q_frames, N)
    out = np.zeros((qt.size, heads, d))
    for h in range(heads):
        s = q[qt, h] @ k[:, h].T / np.sqrt(d)
        s = np.where(allowed[None, :], s, -np.inf)
        s -= s.max(axis=1, keepdims=True)
        p = np.exp(s)
        p /= p.sum(axis=1, keepdims=True)
        out[:, h] = p @ v[:, h]
    return out


@pytest.mark.parametrize("qf,kvf", [([0], [0]), ([1, 3], [0, 4]), ([0, 2, 4], [0, 2, 4]),
                                    ([2], [0, 1, 3]), ([0, 1, 2, 3, 4], [3])])
def test_matches_dense_masked_softmax(qf, kvf):
    q, k, v = _qkv(5, 7, 3, 16, 1)
    got = oracle.frame_attention(q, k, v, qf, kvf, 7)
    exp = _masked_softmax_reference(q, k, v, qf, kvf, 7)
    assert np.abs(got - exp).max() < 1e-12


def test_masked_frames_have_no_influence():
    q, k, v = _qkv(6, 5, 2, 8, 2)
    kvf = [0, 2, 5]
    base = oracle.frame_attention(q, k, v, [0, 5], kvf, 5)
    k2, v2 = k.copy(), v.copy()
    for f in (1, 3, 4):
        k2[f * 5:(f + 1) * 5] = np.nan
        v2[f * 5:(f + 1) * 5] = np.nan
    got = oracle.frame_attention(q, k2, v2, [0, 5], kvf, 5)
    assert np.isfinite(got).all() and np.array_equal(got, base)
    # and the listed frames do matter
    k3 = k.copy()
    k3[2 * 5] += 1.0
    assert not np.array_equal(oracle.frame_attention(q, k3, v, [0, 5], kvf, 5), base)


def test_single_frame_is_plain_attention():
    q, k, v = _qkv(4, 9, 2, 16, 3)
    got = oracle.frame_attention(q, k, v, [1], [3], 9)
    qt = torch.from_numpy(q[9:18]).permute(1, 0, 2)
    kt = torch.from_numpy(k[27:36]).permute(1, 0, 2)
    vt = torch.from_numpy(v[27:36]).permute(1, 0, 2)
    ref = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt).permute(1, 0, 2).numpy()
    assert np.abs(got - ref).max() < 1e-12


def test_key_order_inside_mask_is_irrelevant():
    q, k, v = _qkv(5, 4, 1, 8, 4)
    a = oracle.frame_attention(q, k, v, [0, 1], [0, 2, 4], 4)
    b = oracle.frame_attention(q, k, v, [0, 1], [4, 0, 2], 4)
    assert np.abs(a - b).max() < 1e-14


def test_bf16_bits_accepted():
    q, k, v = (torch.from_numpy(x).to(torch.bfloat16) for x in _qkv(3, 4, 1, 8, 5))
    got = oracle.frame_attention(q, k, v, [0], [0, 2], 4)
    q64, k64, v64 = (oracle.as_oracle_f64(x) for x in (q, k, v))
    assert np.array_equal(got, oracle.frame_attention(q64, k64, v64, [0], [0, 2], 4))
