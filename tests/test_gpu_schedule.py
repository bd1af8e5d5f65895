"""A whole progressive asynchronous schedule (Eq. 2, Alg. 2) driven through the
kernels step by step, against the oracle driving the same plan on a state of its
own (fp64, never fed from the GPU):

  warm-up steps and Rhythmic Points run attention with every frame's queries;
  skipped steps run keyframe-query attention and scatter its rows into the
  step's output, the non-keyframe rows keeping the last full step's values.
  Two forms of the skipped step:
    latent: the non-keyframe latents are projected (Eq. 3) over the plan's
      interval at the plan's time; attention takes the step's seeded Q/K/V;
    cache:  the non-keyframes' keys and values come from the per-layer rolling
      cache (App. B.2): initialised from the last warm-up step's output,
      shift-and-store at each Rhythmic Point, projected into K and V before the
      keyframe-query attention. Each stored state is labelled with the step it
      was computed at, so every later skipped step lies below the newest label
      and the appendix's weight clamps to 1 (the cache returns h_after).
    cache_interp: as cache, but each stored state is labelled with the time its
      update leads the non-keyframes to (the plan's target time): the skipped
      steps then lie strictly inside (t_after, t_before) and are interpolated
      with 0 < alpha < 1, which the test asserts at every skipped step.

Every step's whole output is compared with the oracle's under the attention
gates. In the cache form a step's output feeds later steps through the cache;
the GPU caches its rounded outputs, the oracle its exact ones, and the carried
difference (relative 2^-9 in bf16 per stored state) moves the scores by far less
than the gates allow, so the same gates hold at every step."""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_06309_amd import workloads
from parity import assert_parity, torch_bf16_to_f64

pytestmark = pytest.mark.gpu

rf = pytest.importorskip("paper_2606_06309_amd.binding")

# 12 steps: two warm-up steps, stride 2 above t = 6 and 3 below (Eq. 2), so the
# plan holds Rhythmic Points at 10, 8, 6 and 3 and skipped steps between them
# (alpha 1/2, 1/3 and 2/3).
PLAN = (12, 2, 6, 2, 3)

CASES = [
    (workloads.WORKLOADS["tiny"], "f32"),                                          # 5 frames of 64, d = 64
    (workloads.custom(6, 5, 7, 2, 64, (0, 3), dtype="bf16", seed=41), "bf16"),    # N = 35: one partial tile a frame
    (workloads.custom(5, 9, 15, 2, 128, (0, 2), dtype="bf16", seed=42), "bf16"),  # N = 135: ragged over three tiles
]


def _f64(t):
    return torch_bf16_to_f64(t) if t.dtype == torch.bfloat16 else t.detach().cpu().double().numpy()


def _bits(t):
    t = t.detach().cpu().contiguous()
    return t.view(torch.int16 if t.dtype == torch.bfloat16 else torch.int32).numpy()


def test_plan_matches_the_oracle_plan():
    plan = rf.rf_async_schedule(*PLAN)
    ref = oracle.async_schedule(*PLAN)
    assert [p["phase"] for p in plan] == [p["phase"] for p in ref]
    assert [p["phase"] for p in plan].count("skip") == 6
    for p, r in zip(plan, ref):
        assert p["t"] == r["t"] and p["n_skip"] == r["n_skip"]
        if r["phase"] == "skip":
            assert (p["t_start"], p["t_end"]) == (r["t_start"], r["t_end"])
            assert p["alpha"] == pytest.approx(r["alpha"], abs=1e-15)


@pytest.mark.parametrize("mode", ["latent", "cache", "cache_interp"])
@pytest.mark.parametrize("w,kind", CASES, ids=lambda x: getattr(x, "name", None) and f"{x.name}_N{x.N}_d{x.head_dim}")
def test_schedule_step_by_step(w, kind, mode):
    print(f"[case] schedule {PLAN} {mode} {w.name} T={w.T} N={w.N} d={w.head_dim} {kind}", flush=True)
    plan = rf.rf_async_schedule(*PLAN)
    ids, mask = rf.rf_select_keyframes(w.keyframes, w.T)
    ids = ids.tolist()
    nonkey = [f for f in range(w.T) if f not in set(ids)]
    D = w.heads * w.head_dim
    sets = [workloads.make_qkv(w, device="cuda", seed=900 + i) for i in range(2)]
    sets_ref = [tuple(oracle.as_oracle_f64(x.cpu()) for x in s) for s in sets]
    lat = workloads.make_latents(w, B=1, device="cuda")
    lat_cpu = lat.cpu()
    Hl, Wl = w.latent_hw
    full_out = torch.zeros((w.S, w.heads, w.head_dim), dtype=w.torch_dtype, device="cuda")
    full_ref = np.zeros((w.S, w.heads, w.head_dim))
    kq_out = torch.empty((w.M * w.N, w.heads, w.head_dim), dtype=w.torch_dtype, device="cuda")
    el = torch.tensor([], dtype=w.torch_dtype).element_size()
    store = torch.zeros(rf.rf_cache_store_bytes(len(nonkey), w.N, D, w.torch_dtype) // el,
                        dtype=w.torch_dtype, device="cuda")
    cache = cache_ref = None
    nonkey_rows = np.concatenate([np.arange(f * w.N, (f + 1) * w.N) for f in nonkey])
    projections = 0
    alphas = []
    for i, step in enumerate(plan):
        q, k, v = sets[i % 2]
        qr, kr, vr = sets_ref[i % 2]
        what = f"{mode} {w.name} step t={step['t']} ({step['phase']})"
        if step["phase"] != "skip":
            rf.rf_keyframe_attention(q, k, v, list(range(w.T)), w.T, w.H, w.W, out=full_out)
            full_ref = oracle.keyframe_attention(qr, kr, vr, list(range(w.T)), w.N)
            if mode != "latent":
                last_warmup = step["phase"] == "warmup" and (i + 1 == len(plan) or plan[i + 1]["phase"] != "warmup")
                h_ref = full_ref.reshape(w.T, w.N, D)
                label = float(step["nonkey_to"] if mode == "cache_interp" else step["t"])
                if last_warmup:
                    cache = rf.rf_cache_init(nonkey, w.T, w.N, D, w.torch_dtype, label, store=store,
                                             h_full=full_out)
                    cache_ref = oracle.RollingCache()
                    cache_ref.init(nonkey, {f: h_ref[f] for f in nonkey}, label)
                elif step["phase"] == "rhythmic":
                    rf.rf_cache_shift_store(cache, label, store=store, h_full=full_out)
                    cache_ref.shift_and_store(nonkey, {f: h_ref[f] for f in nonkey}, label)
        else:
            before = _bits(full_out)
            if mode != "latent":
                for f in nonkey:
                    a = rf.rf_cache_alpha(cache, f, float(step["t"]))
                    a_ref = oracle.hidden_alpha(cache_ref.t_before[f], cache_ref.t_after[f], float(step["t"]))
                    assert a == pytest.approx(a_ref, abs=1e-15), what
                    if mode == "cache_interp":
                        assert 0.0 < a < 1.0, f"{what}: alpha {a} of frame {f} is not interior"
                        alphas.append(a)
                    else:
                        assert a == 1.0, what
                k, v = k.clone(), v.clone()
                rf.rf_cache_project_kv(cache, store, k, v, float(step["t"]))
                kr, vr = oracle.skip_step_kv(kr, vr, cache_ref, nonkey, float(step["t"]), w.N)
            else:
                ts = (step["t_start"], step["t_end"], step["t"])
                proj = rf.rf_project_latents(lat, ts, mask)
                torch.cuda.synchronize()
                proj_ref = oracle.project_latents(lat_cpu, 1, w.latent_c, w.T, Hl, Wl, ts, mask)
                assert_parity(_f64(proj), proj_ref, "f32", what + " projection")
                projections += 1
            rf.rf_keyframe_attention(q, k, v, ids, w.T, w.H, w.W, out=kq_out)
            rf.rf_scatter_frames(kq_out, full_out, ids, w.T, w.N)
            kq_ref = oracle.keyframe_attention(qr, kr, vr, ids, w.N)
            full_ref = full_ref.copy()
            full_ref[oracle.rowmap(ids, w.N)] = kq_ref
            torch.cuda.synchronize()
            # the non-keyframe rows keep the last full step's output bit for bit
            assert np.array_equal(_bits(full_out)[nonkey_rows], before[nonkey_rows]), what
        torch.cuda.synchronize()
        assert_parity(_f64(full_out), full_ref, kind, what)
    assert cache is not None or mode == "latent"
    assert projections == (6 if mode == "latent" else 0)
    if mode == "cache_interp":
        # the plan's skipped steps: 9 and 7 (alpha 1/2), 5, 4, 2, 1 (alpha 1/3, 2/3)
        assert len(alphas) == 6 * len(nonkey)
        assert sorted(set(round(a, 6) for a in alphas)) == [round(1 / 3, 6), 0.5, round(2 / 3, 6)]
