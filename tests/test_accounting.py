"""FLOP accounting: the roofline count and the paper's analytic model.

The paper's worked example for Wan2.1-T2V-1.3B (App. B.1) is the fixture
tests/golden/flops_wan21.json, copied as printed. Values the paper's own
formula reproduces are asserted to the printed precision; printed values that
do not follow from the formula are listed there with the relation they do
satisfy, and that relation is asserted instead.
"""
import json
import os

import pytest

from paper_2606_06309_amd import accounting as acc
from paper_2606_06309_amd import workloads

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "flops_wan21.json")


@pytest.fixture(scope="module")
def wan():
    with open(GOLDEN) as f:
        return json.load(f)


def test_paper_dense_figures(wan):
    c, p = wan["config"], wan["printed"]
    assert c["S"] == c["F"] * c["N"] and c["D"] == c["H"] * c["d"]
    layer = acc.paper_layer_flops(c["S"], c["D"])
    assert round(layer / 1e12, 2) == p["dense_layer_tflops"]
    attn = 2 * c["S"] ** 2 * c["D"]
    assert round(100 * attn / layer, 1) == p["attention_share_percent"]
    dense = acc.paper_dense_flops(c["L"], c["T"], c["S"], c["D"])
    assert round(dense / 1e15, 2) == p["dense_total_pflops"]
    # printed per-term products carry small arithmetic slips (< 0.05 %)
    assert abs(4 * c["S"] * c["D"] ** 2 / p["dense_layer_term_4SD2"] - 1) < 5e-4
    assert abs(attn / p["dense_layer_term_2S2D"] - 1) < 5e-4


def test_paper_step_counts(wan):
    c, p = wan["config"], wan["printed"]
    assert acc.paper_step_counts(c["T"], c["T_warmup"], c["n"]) == (
        p["T_rhymeflow"], p["N_skip"], p["N_denoise"])


def test_paper_phase_figures(wan):
    c, p = wan["config"], wan["printed"]
    r = acc.paper_rhymeflow_flops(c["L"], c["T"], c["T_warmup"], c["F"], c["N"],
                                  c["D"], c["M"], c["n"])
    assert round(r["warmup"] / 1e15, 2) == p["warmup_pflops"]
    assert round(r["denoise"] / 1e15, 2) == p["denoise_total_pflops"]
    s_skip = c["M"] * c["N"]
    assert s_skip == p["skip_S"]
    # the printed skip attention term is 4 S^2 D, twice the formula's 2 S^2 D
    assert p["skip_layer_term_attention"] == 2 * (2 * s_skip ** 2 * c["D"])
    assert abs(4 * s_skip * c["D"] ** 2 / p["skip_layer_term_4SD2"] - 1) < 2e-3
    # with the doubled term the printed totals follow
    doubled_layer = 4 * s_skip * c["D"] ** 2 + 4 * s_skip ** 2 * c["D"]
    assert round(doubled_layer / 1e12, 2) == p["skip_layer_tflops"]
    skip_doubled = c["L"] * p["N_skip"] * doubled_layer
    assert round(skip_doubled / 1e15, 2) == p["skip_total_pflops"]
    total_doubled = r["warmup"] + skip_doubled + r["denoise"]
    assert round(total_doubled / 1e15, 2) == p["rhymeflow_total_pflops"]
    dense = acc.paper_dense_flops(c["L"], c["T"], c["S"], c["D"])
    assert round(dense / total_doubled, 2) == round(p["speedup"], 2)
    # the formula as written
    assert round(r["total"] / 1e15, 2) == 17.14
    assert round(dense / r["total"], 3) == 1.599


@pytest.mark.parametrize("name,tflop,all_tflop", [
    ("small", 0.972, 2.527), ("480p", 1.884, 6.594),
    ("720p", 33.44, 117.05), ("long", 42.04, 173.43)])
def test_roofline_flop_count(name, tflop, all_tflop):
    w = workloads.WORKLOADS[name]
    f = acc.attention_flops(w.M * w.N, w.S, w.head_dim, w.heads)
    fa = acc.attention_flops(w.S, w.S, w.head_dim, w.heads)
    assert round(f / 1e12, 3 if tflop < 10 else 2) == tflop
    assert round(fa / 1e12, 3 if all_tflop < 10 else 2) == all_tflop
    assert fa / f == pytest.approx(acc.ideal_speedup(w.T, w.M))


def test_byte_counts():
    w = workloads.WORKLOADS["480p"]
    # 16 x 21 x 60 x 104 fp32 latents, 6 keyframes: 15 planes r/r/w + 6 planes r/w
    b = acc.projection_bytes(1, 16, 21, 60 * 104, 6, 4)
    assert b == 16 * (15 * 3 + 6 * 2) * 6240 * 4
    assert acc.projection_bytes(1, 16, 21, 6240, 6, 4, aliased=True) == 16 * 45 * 6240 * 4
    assert acc.gather_bytes(6, w.N, w.heads * w.head_dim * 2) == 2 * 9360 * 12 * 128 * 2


def test_cache_byte_counts():
    w = workloads.WORKLOADS["long"]
    # 25 cached frames of 3,600 rows x 3,072 bf16: 22,118,400 bytes each
    fb = w.N * w.heads * w.head_dim * 2
    assert fb == 22_118_400
    assert acc.cache_projection_bytes(25, fb) == 2_211_840_000
    assert acc.cache_store_bytes(25, fb) == 1_105_920_000


def test_schedule_ledger():
    # T = 50 steps, T_w = 8, strides 2 / 3 at T_mid = 25: 8 warm-up, 17 Rhythmic Points, 25 skipped
    plan = oracle.async_schedule(50, 8, 25, 2, 3)
    w = workloads.WORKLOADS["long"]
    led = acc.schedule_attention_flops(plan, w.T, w.M, w.N, w.head_dim, w.heads)
    assert led["steps"] == {"warmup": 8, "rhythmic": 17, "skip": 25}
    S = w.S
    full = 4 * S * S * 128 * 24
    kq = 4 * 8 * 3600 * S * 128 * 24
    assert led["full_step_flop"] == full and led["skip_step_flop"] == kq
    assert led["flop"] == 25 * full + 25 * kq and led["dense_flop"] == 50 * full
    # 50 / (25 + 25 * 8/33) = 1.6097...
    assert abs(led["ratio"] - 50.0 / (25.0 + 25.0 * 8.0 / 33.0)) < 1e-12
