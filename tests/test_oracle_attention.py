"""Pins for the oracle's fp64 keyframe-query attention.

The oracle is checked against things other than itself:
  * full 3D attention from independent library routines (scipy softmax with a
    BLAS matmul, and torch's CPU scaled_dot_product_attention in float64):
    with every frame a keyframe the method's attention is exactly the dense
    attention of warm-up steps and Rhythmic Points (Sec. 3.2.1, 3.2.3);
  * the row-subset identity: keyframe-query attention is the dense attention's
    rows at the keyframe tokens (App. B.2: keyframes attend over all frames);
  * softmax rows summing to one and nonnegative;
  * closed forms (constant keys, constant values, one dominant logit, S = 1);
  * invariances (joint K/V permutation, affine maps of V, unread query rows);
  * 50-digit mpmath evaluation of the definition on a few rows.
"""
import math

import mpmath
import numpy as np
import pytest
import scipy.special
import torch

import oracle
from paper_2606_06309_amd import workloads
from parity import passes, torch_bf16_to_f64

TINY = workloads.WORKLOADS["tiny"]


def _dense_scipy(q, k, v):
    """softmax(Q K^T / sqrt(d)) V per head with scipy + numpy BLAS, fp64."""
    S, H, d = k.shape
    out = np.zeros((q.shape[0], H, d))
    for h in range(H):
        a = q[:, h, :] @ k[:, h, :].T / math.sqrt(d)
        out[:, h, :] = scipy.special.softmax(a, axis=1) @ v[:, h, :]
    return out


def _tiny_f64():
    q, k, v = workloads.make_qkv(TINY)
    return q.double().numpy(), k.double().numpy(), v.double().numpy()


def test_all_frames_equals_dense_attention_scipy():
    q, k, v = _tiny_f64()
    ref = _dense_scipy(q, k, v)
    out = oracle.keyframe_attention(q, k, v, range(TINY.T), TINY.N)
    assert np.abs(out - ref).max() < 1e-12


def test_all_frames_equals_torch_sdpa_float64():
    q, k, v = (torch.from_numpy(x) for x in _tiny_f64())
    # [S][H][d] -> [H][S][d]
    ref = torch.nn.functional.scaled_dot_product_attention(
        q.transpose(0, 1).contiguous(), k.transpose(0, 1).contiguous(),
        v.transpose(0, 1).contiguous()).transpose(0, 1).numpy()
    out = oracle.keyframe_attention(q, k, v, range(TINY.T), TINY.N)
    assert np.abs(out - ref).max() < 1e-12


def test_keyframe_rows_are_dense_rows():
    q, k, v = _tiny_f64()
    dense = _dense_scipy(q, k, v)
    kf = TINY.keyframes
    tokens = np.arange(TINY.S).reshape(TINY.T, TINY.N)[list(kf)].ravel()
    out = oracle.keyframe_attention(q, k, v, kf, TINY.N)
    assert out.shape == (len(kf) * TINY.N, TINY.heads, TINY.head_dim)
    assert np.abs(out - dense[tokens]).max() < 1e-12


def test_row_and_head_subsets_are_exact():
    q, k, v = _tiny_f64()
    full = oracle.keyframe_attention(q, k, v, TINY.keyframes, TINY.N)
    rows = np.array([0, 5, 63, 64, 127, 191])
    sub = oracle.keyframe_attention(q, k, v, TINY.keyframes, TINY.N, rows=rows, heads=[1])
    assert np.array_equal(sub[:, 0, :], full[rows, 1, :])


def test_softmax_rows_sum_to_one():
    q, k, v = _tiny_f64()
    out, p = oracle.keyframe_attention(q, k, v, TINY.keyframes, TINY.N, return_probs=True)
    assert (p >= 0).all()
    assert np.abs(p.sum(axis=-1) - 1.0).max() < 1e-12
    # and they are the library softmax rows
    kf_tokens = oracle.rowmap(TINY.keyframes, TINY.N)
    for h in range(TINY.heads):
        a = q[kf_tokens, h, :] @ k[:, h, :].T / math.sqrt(TINY.head_dim)
        assert np.abs(p[:, h, :] - scipy.special.softmax(a, axis=1)).max() < 1e-14


def test_bf16_bits_are_widened_exactly():
    w = workloads.custom(3, 4, 4, 2, 64, (0, 2), dtype="bf16", seed=7)
    q, k, v = workloads.make_qkv(w)
    a = oracle.keyframe_attention(q, k, v, w.keyframes, w.N)
    b = oracle.keyframe_attention(torch_bf16_to_f64(q), torch_bf16_to_f64(k),
                                  torch_bf16_to_f64(v), w.keyframes, w.N)
    assert np.array_equal(a, b)


def test_f32_inputs_are_widened_exactly():
    q, k, v = workloads.make_qkv(TINY)
    a = oracle.keyframe_attention(q, k, v, TINY.keyframes, TINY.N)
    b = oracle.keyframe_attention(q.double(), k.double(), v.double(), TINY.keyframes, TINY.N)
    assert np.array_equal(a, b)


# --- closed forms -----------------------------------------------------------------

def test_constant_keys_give_mean_of_values():
    q, k, v = _tiny_f64()
    k[:] = k[0:1]
    out = oracle.keyframe_attention(q, k, v, TINY.keyframes, TINY.N)
    assert np.abs(out - v.mean(axis=0)[None]).max() < 1e-14


def test_constant_values_give_that_value():
    q, k, v = _tiny_f64()
    v[:] = v[3:4]
    out = oracle.keyframe_attention(q, k, v, TINY.keyframes, TINY.N)
    assert np.abs(out - v[3][None]).max() < 1e-14


def test_one_dominant_logit():
    rng = np.random.default_rng(0)
    S, H, d = 97, 1, 64
    q = np.zeros((1, H, d)); q[0, 0, 0] = 2.0
    k = np.zeros((S, H, d)); jstar = 41
    k[jstar, 0, 0] = 50.0 * math.sqrt(d) / 2.0          # logit of jstar = 50, others 0
    v = rng.standard_normal((S, H, d))
    out = oracle.attention_pairs(q, k, v, [0], [0])[0]
    e = math.exp(50.0)
    expect = (e * v[jstar, 0] + (v[:, 0].sum(axis=0) - v[jstar, 0])) / (e + S - 1)
    assert np.abs(out - expect).max() < 1e-14
    assert np.abs(out - v[jstar, 0]).max() < math.exp(-50.0) * S * np.abs(v).max() * 2


def test_single_key_returns_its_value():
    rng = np.random.default_rng(1)
    q = rng.standard_normal((4, 2, 64))
    k = rng.standard_normal((1, 2, 64))
    v = rng.standard_normal((1, 2, 64))
    out = oracle.keyframe_attention(q, k, v, [0], 4)
    assert np.array_equal(out, np.broadcast_to(v, out.shape))


# --- invariances ----------------------------------------------------------------

def test_joint_kv_permutation_invariance():
    q, k, v = _tiny_f64()
    perm = np.random.default_rng(2).permutation(TINY.S)
    a = oracle.keyframe_attention(q, k, v, TINY.keyframes, TINY.N)
    b = oracle.keyframe_attention(q, k[perm], v[perm], TINY.keyframes, TINY.N)
    assert np.abs(a - b).max() < 1e-13


def test_affine_value_map():
    q, k, v = _tiny_f64()
    a = oracle.keyframe_attention(q, k, v, TINY.keyframes, TINY.N)
    b = oracle.keyframe_attention(q, k, 3.0 * v - 0.75, TINY.keyframes, TINY.N)
    assert np.abs(b - (3.0 * a - 0.75)).max() < 1e-12


def test_non_keyframe_queries_are_never_read():
    q, k, v = _tiny_f64()
    a = oracle.keyframe_attention(q, k, v, TINY.keyframes, TINY.N)
    grid = q.reshape(TINY.T, TINY.N, TINY.heads, TINY.head_dim)
    for f in range(TINY.T):
        if f not in TINY.keyframes:
            grid[f] = np.nan
    b = oracle.keyframe_attention(grid.reshape(q.shape), k, v, TINY.keyframes, TINY.N)
    assert np.array_equal(a, b)


# --- high precision ----------------------------------------------------------------

def test_mpmath_50_digits():
    q, k, v = _tiny_f64()
    rows = [0, 1, 63, 64, 100, 127, 128, 150, 191]
    heads = [0, 1]
    out = oracle.keyframe_attention(q, k, v, TINY.keyframes, TINY.N, rows=rows, heads=heads)
    tokens = np.arange(TINY.S).reshape(TINY.T, TINY.N)[list(TINY.keyframes)].ravel()
    mpmath.mp.dps = 50
    d = TINY.head_dim
    inv = 1 / mpmath.sqrt(d)
    worst = 0.0
    for ri, r in enumerate(rows[:6]):
        for hi, h in enumerate(heads):
            i = tokens[r]
            qi = [mpmath.mpf(float(x)) for x in q[i, h]]
            s = []
            for j in range(TINY.S):
                s.append(mpmath.fsum(qi[c] * mpmath.mpf(float(k[j, h, c])) for c in range(d)) * inv)
            m = max(s)
            p = [mpmath.exp(x - m) for x in s]
            l = mpmath.fsum(p)
            for c in range(0, d, 7):
                o = mpmath.fsum(p[j] * mpmath.mpf(float(v[j, h, c])) for j in range(TINY.S)) / l
                worst = max(worst, abs(float(o) - out[ri, hi, c]))
    assert worst < 1e-13


# --- the parity gate catches plausible kernel mistakes -------------------------------

def _small_like_case():
    """A near-uniform-softmax case shaped like the small workload's inputs
    (Q/K/V scaled by 1/sqrt(128)) but tiny: the kind of case where absolute
    bounds alone would accept a zero output."""
    w = workloads.custom(8, 10, 12, 2, 128, (0, 3, 6), dtype="bf16", seed=11,
                         qkv_scale=1.0 / math.sqrt(128.0))
    q, k, v = workloads.make_qkv(w)
    return w, torch_bf16_to_f64(q), torch_bf16_to_f64(k), torch_bf16_to_f64(v)


def test_gate_rejects_planted_mistakes():
    w, q, k, v = _small_like_case()
    ref = oracle.keyframe_attention(q, k, v, w.keyframes, w.N)
    ok, _ = passes(ref, ref, "bf16")
    assert ok
    # bf16 rounding of the exact output passes
    rounded = torch.from_numpy(ref).to(torch.bfloat16).double().numpy()
    ok, st = passes(rounded, ref, "bf16")
    assert ok, st
    # zeros: passes the absolute bounds, fails the relative one
    ok, st = passes(np.zeros_like(ref), ref, "bf16")
    assert st["max_abs"] <= 2e-2 and not ok
    # query rows shifted by one frame
    shifted = oracle.keyframe_attention(q, k, v, [f + 1 for f in w.keyframes], w.N)
    assert not passes(shifted, ref, "bf16")[0]
    # keys/values restricted to keyframes
    kv_tok = oracle.rowmap(w.keyframes, w.N)
    qk = q[kv_tok]
    restricted = oracle.keyframe_attention(qk, k[kv_tok], v[kv_tok], range(len(w.keyframes)), w.N)
    assert not passes(restricted, ref, "bf16")[0]


def test_gate_rejects_planted_mistakes_unit_inputs():
    """Q/K/V ~ N(0,1) (logit std ~ 1): a wrong softmax scale is visible here,
    while on the near-uniform case above it moves the output by < 1 %."""
    w = workloads.custom(8, 10, 12, 2, 128, (0, 3, 6), dtype="bf16", seed=13)
    q, k, v = (torch_bf16_to_f64(x) for x in workloads.make_qkv(w))
    ref = oracle.keyframe_attention(q, k, v, w.keyframes, w.N)
    rounded = torch.from_numpy(ref).to(torch.bfloat16).double().numpy()
    assert passes(rounded, ref, "bf16")[0]
    wrong_scale = oracle.keyframe_attention(q / math.sqrt(w.head_dim), k, v, w.keyframes, w.N)
    assert not passes(wrong_scale, ref, "bf16")[0]
    assert not passes(np.zeros_like(ref), ref, "bf16")[0]
    shifted = oracle.keyframe_attention(q, k, v, [f + 1 for f in w.keyframes], w.N)
    assert not passes(shifted, ref, "bf16")[0]
    kv_tok = oracle.rowmap(w.keyframes, w.N)
    restricted = oracle.keyframe_attention(q[kv_tok], k[kv_tok], v[kv_tok],
                                           range(len(w.keyframes)), w.N)
    assert not passes(restricted, ref, "bf16")[0]


def test_gate_rejects_planted_mistakes_sharp_softmax():
    w = workloads.custom(6, 4, 6, 2, 64, (0, 3), dtype="f32", seed=12)
    q, k, v = (x.double().numpy() for x in workloads.make_qkv(w))
    q = q * 4.0
    ref = oracle.keyframe_attention(q, k, v, w.keyframes, w.N)
    assert passes(ref + 5e-6, ref, "f32")[0]
    # dropped term: the last key left out of the softmax
    dropped = oracle.keyframe_attention(q, k[:-1], v[:-1], w.keyframes, w.N)
    assert not passes(dropped, ref, "f32")[0]
    # transposed operand: keys and values swapped
    swapped = oracle.keyframe_attention(q, v, k, w.keyframes, w.N)
    assert not passes(swapped, ref, "f32")[0]
