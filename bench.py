#!/usr/bin/env python3
"""Benchmark of the keyframe-query attention path on one MI355X.

One step is one pass of the hot path at a skip step over one batch of
synthetic input already resident in HBM:
  1. keyframe set normalisation and mask (host, C ABI),
  2. latent trajectory projection of the non-keyframes (Eq. 3),
  3. keyframe-query attention with the fused query gather,
  4. scatter of the keyframe rows into the full-sequence output.
The all-frame comparator (the same kernel with every frame a keyframe, i.e.
the dense attention of warm-up steps and Rhythmic Points) is timed beside it
for the speedup.

Prints ONE JSON line. `value` is keyframe-query attention TFLOP per second of
whole-step time; `roofline` describes the attention kernel alone, timed with
HIP events around each launch on the stream it runs on, with the shader clock
sampled under that load. Side sections time the bandwidth kernels
(projection, gather, scatter), content-aware selection (frame similarity, one
video and an HBM-sized batch, and Alg. 1's scan), the rolling cache of App. B.2
(projection of cached states into K and V, shift-and-store), keyframe-only
attention (a frame-level key/value mask), a whole denoising schedule of Alg. 2
(attention path only; latent projection, rolling cache with clamped and with
interpolating labels) against its dense counterpart, the other workloads
(keyframe-query and all-frame attention at the paper's two model shapes and
the smaller configurations), and the oracle per configuration beside the
headline CPU baseline.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "keyframe-query 3D attention TFLOP/s + % bf16 MFMA peak; speedup vs all-frame"
PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 matrix peak
PEAK_HBM_GBS = 8000.0         # MI355X HBM3E


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=10,
                    help="untimed steps first (the clock takes a few hundred ms to settle under load)")
    ap.add_argument("--workload", default="long",
                    help="long (default), 720p, 480p, small, tiny; the model shapes wan-1.3b, cogvideox")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-comparator", action="store_true")
    ap.add_argument("--no-bandwidth", action="store_true")
    ap.add_argument("--no-selection", action="store_true")
    ap.add_argument("--no-cache", action="store_true")
    ap.add_argument("--no-schedule", action="store_true")
    ap.add_argument("--no-frame-mask", action="store_true")
    ap.add_argument("--no-shard", action="store_true")
    ap.add_argument("--no-peaks", action="store_true")
    ap.add_argument("--no-configs", action="store_true")
    ap.add_argument("--no-clock", action="store_true")
    ap.add_argument("--schedule", default="50,8,25,2,3",
                    help="T,T_w,T_mid,n_small,n_large of the multi-step schedule loop")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="target CPU work of the oracle baseline sample")
    return ap.parse_args()


def _side(name, fn, *args):
    """Runs a side measurement; an exception in it is reported (stderr and the
    JSON line) instead of costing the line itself. The timed step is not run
    through this."""
    try:
        return fn(*args)
    except Exception as e:   # noqa: BLE001 - any failure of a side section is reported, not raised
        print(f"[bench] {name} failed: {e!r}", file=sys.stderr, flush=True)
        return {"error": repr(e)[:300]}


def _events(n):
    import torch
    return [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
            for _ in range(n)]


def _avg_ms(pairs):
    return sum(a.elapsed_time(b) for a, b in pairs) / len(pairs)


def cpu_baseline(w, q, k, v, target_s):
    """The oracle as it stands, on a bounded sample of query rows."""
    import numpy as np
    import oracle
    from paper_2606_06309_amd import accounting

    qh, kh, vh = q.cpu(), k.cpu(), v.cpu()
    rowmap = oracle.rowmap(w.keyframes, w.N)
    rng = np.random.default_rng(2026)
    cores = oracle.num_threads()

    def run(n):
        rows = rng.choice(rowmap.size, n, replace=True)
        heads = rng.integers(0, w.heads, n)
        t0 = time.perf_counter()
        oracle.attention_pairs(qh, kh, vh, rowmap[rows], heads)
        return time.perf_counter() - t0

    n0 = max(2, cores)
    t_cal = run(n0)
    n = int(max(n0, min(200000, n0 * target_s / max(t_cal, 1e-3))))
    t = run(n)
    flop = n * accounting.attention_flops(1, w.S, w.head_dim, 1)
    # the same oracle on one thread, a short sample (about a fifth of the budget)
    oracle.set_num_threads(1)
    n1 = max(1, int(n / max(1, cores) * 0.2))
    t1 = run(n1)
    oracle.set_num_threads(cores)
    flop1 = n1 * accounting.attention_flops(1, w.S, w.head_dim, 1)
    cpu = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    cpu = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"value": flop / t / 1e12, "unit": "TFLOP/s", "cores": cores, "kind": "oracle", "cpu": cpu,
            "one_thread": {"value": flop1 / t1 / 1e12, "sample": f"{n1} pairs, {t1:.1f} s"},
            "sample": f"{n} random (keyframe row, head) pairs of the {w.name} workload, each over "
                      f"all S={w.S} keys, fp64; {t:.1f} s"}


def source_digest(path):
    """sha256 of a source file's code: comments removed and whitespace
    collapsed, so that edits of comments alone keep the digest."""
    import hashlib
    import re
    text = open(path, encoding="utf-8").read()
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    text = " ".join(text.split())
    return hashlib.sha256(text.encode()).hexdigest()


def profiled_traffic(workload):
    """HBM bytes per attention launch from the committed rocprofv3 counter
    summary, or None when there is none or the attention code has changed
    since the counters were taken."""
    path = os.path.join(ROOT, "profiles", f"attn_bf16_{workload}_traffic.txt")
    src = os.path.join(ROOT, "paper_2606_06309_amd", "csrc", "rf_attention.hip")
    if not os.path.exists(path):
        return None
    sha = source_digest(src)
    fields = {}
    for line in open(path):
        if ":" in line:
            key, _, val = line.partition(":")
            fields[key.strip()] = val.strip()
    if fields.get("attention code sha256") != sha:
        return None
    try:
        return int(fields["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}, WORLD_SIZE={world}): "
              "the keyframe-query attention path is provided for a single GPU; across GPUs it "
              "would shard by head, with no exchange between GPUs.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    from paper_2606_06309_amd import accounting, binding as rf, workloads

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    w = workloads.WORKLOADS[args.workload]
    dev = "cuda"
    torch.cuda.set_device(0)
    print(f"[bench] workload {w.name}: T={w.T} H={w.H} W={w.W} heads={w.heads} d={w.head_dim} "
          f"M={w.M} keyframes={list(w.keyframes)}", file=sys.stderr, flush=True)

    q, k, v = workloads.make_qkv(w, device=dev)
    lat = workloads.make_latents(w, B=1, device=dev)
    Hl, Wl = w.latent_hw
    proj_out = torch.empty((1, w.latent_c, w.T, Hl, Wl), dtype=lat.dtype, device=dev)
    Mq = w.M * w.N
    attn_out = torch.empty((Mq, w.heads, w.head_dim), dtype=q.dtype, device=dev)
    full_out = torch.zeros((w.S, w.heads, w.head_dim), dtype=q.dtype, device=dev)
    # split-key tail workspace, sized for the largest launch (the all-frame comparator or this step)
    ws = torch.empty(max(16, rf.rf_attention_workspace(w.M, w.T, w.T, w.H, w.W, w.heads, w.head_dim, q.dtype),
                         rf.rf_attention_workspace(w.T, w.T, w.T, w.H, w.W, w.heads, w.head_dim, q.dtype)),
                     dtype=torch.uint8, device=dev)
    torch.cuda.synchronize()

    def step(ev=None):
        ids, mask = rf.rf_select_keyframes(w.keyframes, w.T)
        rf.rf_project_latents(lat, w.timesteps, mask, out=proj_out)
        if ev is not None:
            ev[0].record()
        rf.rf_keyframe_attention_ws(q, k, v, ids, w.T, w.H, w.W, out=attn_out, workspace=ws)
        if ev is not None:
            ev[1].record()
        rf.rf_scatter_frames(attn_out, full_out, ids, w.T, w.N)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    ev = _events(args.steps)
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0.record()
    for i in range(args.steps):
        step(ev[i])
    t1.record()
    torch.cuda.synchronize()
    total_ms = t0.elapsed_time(t1)
    ms_step = total_ms / args.steps
    attn_ms = _avg_ms(ev)
    flop = accounting.attention_flops(Mq, w.S, w.head_dim, w.heads)
    value = flop / (ms_step * 1e-3) / 1e12
    attn_tflops = flop / (attn_ms * 1e-3) / 1e12
    print(f"[bench] step {ms_step:.3f} ms, attention {attn_ms:.3f} ms = {attn_tflops:.1f} TFLOP/s",
          file=sys.stderr, flush=True)

    result = {
        "metric": METRIC, "value": round(value, 3), "unit": "TFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded normal Q/K/V and latents; no model weights)",
        "config": {"workload": w.name, "T": w.T, "H": w.H, "W": w.W, "tokens": w.S,
                   "heads": w.heads, "head_dim": w.head_dim, "keyframes": list(w.keyframes),
                   "query_rows": Mq, "latents": [1, w.latent_c, w.T, Hl, Wl],
                   "latent_dtype": "f32", "parallelism": "none (1 GPU)"},
        "attention": {"avg_ms": round(attn_ms, 4), "tflops": round(attn_tflops, 2),
                      "frac_bf16_peak": round(attn_tflops / PEAK_BF16_TFLOPS, 4),
                      "flop_per_launch": flop},
        "roofline": {"bound": "mfma", "achieved": round(attn_tflops, 2),
                     "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(attn_tflops / PEAK_BF16_TFLOPS, 4),
                     "traffic": profiled_traffic(w.name)},
    }

    if not args.no_comparator:
        all_out = torch.empty((w.S, w.heads, w.head_dim), dtype=q.dtype, device=dev)
        all_ids = list(range(w.T))
        rf.rf_keyframe_attention_ws(q, k, v, all_ids, w.T, w.H, w.W, out=all_out, workspace=ws)
        torch.cuda.synchronize()
        n_all = max(1, min(args.steps, 5))
        ev_all = _events(n_all)
        for i in range(n_all):
            ev_all[i][0].record()
            rf.rf_keyframe_attention_ws(q, k, v, all_ids, w.T, w.H, w.W, out=all_out, workspace=ws)
            ev_all[i][1].record()
        torch.cuda.synchronize()
        all_ms = _avg_ms(ev_all)
        all_flop = accounting.attention_flops(w.S, w.S, w.head_dim, w.heads)
        result["all_frame"] = {"avg_ms": round(all_ms, 4),
                               "tflops": round(all_flop / (all_ms * 1e-3) / 1e12, 2),
                               "launches": n_all}
        result["speedup_vs_all_frame"] = round(all_ms / attn_ms, 4)
        result["ideal_speedup"] = round(accounting.ideal_speedup(w.T, w.M), 4)
        del all_out
        print(f"[bench] all-frame {all_ms:.3f} ms, speedup {all_ms / attn_ms:.3f} "
              f"(ideal {w.T / w.M:.3f})", file=sys.stderr, flush=True)

    if not args.no_bandwidth:
        result["bandwidth"] = _side("bandwidth", bandwidth, w, q, attn_out, full_out, args)

    if not args.no_selection:
        result["selection"] = _side("selection", selection, w, args)

    if not args.no_cache:
        result["rolling_cache"] = _side("rolling_cache", rolling_cache, w, args)

    if not args.no_frame_mask:
        result["frame_mask"] = _side("frame_mask", frame_mask, w, q, k, v, ws, args)

    if not args.no_schedule:
        result["schedule"] = _side("schedule", schedule_loop, w, ws, args)

    if not args.no_shard:
        result["head_shard"] = _side("head_shard", head_shard, w, args)

    if not args.no_clock:
        result["clock"] = _side("clock", clock_sample, lambda: rf.rf_keyframe_attention_ws(
            q, k, v, w.keyframes, w.T, w.H, w.W, out=attn_out, workspace=ws))
        if isinstance(result["clock"], dict) and "sclk_mhz" in result["clock"]:
            # the clock this attention load holds (the 2.5 PFLOP/s peak assumes 2.4 GHz)
            result["roofline"]["sclk_mhz"] = result["clock"]["sclk_mhz"]

    if not args.no_configs:
        result["configs"] = _side("configs", other_configs, w.name, args)

    if not args.no_peaks:
        result["measured_peaks"] = _side("measured_peaks", measured_peaks, attn_tflops)

    if not args.no_cpu_baseline:
        print("[bench] oracle CPU baseline ...", file=sys.stderr, flush=True)
        result["cpu_baseline"] = _side("cpu_baseline", cpu_baseline, w, q, k, v, args.cpu_seconds)
        if isinstance(result["cpu_baseline"], dict) and "error" not in result["cpu_baseline"]:
            gpu = {name: c.get("keyframe_query", {}).get("tflops") for name, c in
                   (result.get("configs") or {}).items() if isinstance(c, dict)}
            gpu[w.name] = attn_tflops
            result["cpu_baseline"]["per_config"] = _side("cpu_per_config", cpu_per_config, gpu)

    print(json.dumps(result), flush=True)


def clock_sample(launch, seconds=1.2):
    """The shader clock while the timed launch runs back to back: one
    `rocm-smi --showclocks` sample taken in a thread ~0.4 s into a loop of
    launches that lasts `seconds` (the power-limited clock of this load)."""
    import re
    import subprocess
    import threading
    import torch

    found = {}

    def sample():
        time.sleep(0.4)
        try:
            out = subprocess.run(["rocm-smi", "--showclocks"], capture_output=True, text=True,
                                 timeout=20).stdout
        except (OSError, subprocess.SubprocessError) as e:
            found["error"] = repr(e)[:200]
            return
        for line in out.splitlines():
            m = re.search(r"\b(sclk|mclk)\b.*?\((\d+)\s*Mhz\)", line, re.I)
            if m:
                found.setdefault(m.group(1).lower() + "_mhz", int(m.group(2)))

    th = threading.Thread(target=sample)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    th.start()
    n = 0
    while time.perf_counter() - t0 < seconds or th.is_alive():
        launch()
        n += 1
        if n % 4 == 0:
            torch.cuda.synchronize()
    torch.cuda.synchronize()
    th.join()
    found["launches"] = n
    found["source"] = "rocm-smi --showclocks, sampled during back-to-back launches of the timed attention call"
    if "sclk_mhz" in found:
        print(f"[bench] clock under the attention load: sclk {found['sclk_mhz']} MHz", file=sys.stderr, flush=True)
    return found


OTHER_CONFIGS = ["small", "480p", "720p", "wan-1.3b", "cogvideox"]


def other_configs(headline, args):
    """Keyframe-query attention (with the split-key tail) and the all-frame
    comparator at the other workloads: the paper's model shapes and the
    smaller configurations, each warmed for >= 0.3 s before timing."""
    import torch
    from paper_2606_06309_amd import accounting, binding as rf, workloads

    res = {}
    for name in OTHER_CONFIGS:
        if name == headline:
            continue
        w = workloads.WORKLOADS[name]
        q, k, v = workloads.make_qkv(w, device="cuda")
        ws = torch.empty(max(16, rf.rf_attention_workspace(w.M, w.T, w.T, w.H, w.W, w.heads, w.head_dim, q.dtype),
                             rf.rf_attention_workspace(w.T, w.T, w.T, w.H, w.W, w.heads, w.head_dim, q.dtype)),
                         dtype=torch.uint8, device="cuda")
        row = {"shape": [w.T, w.H, w.W], "heads": w.heads, "head_dim": w.head_dim, "keyframes": list(w.keyframes)}
        for what, ids in (("keyframe_query", list(w.keyframes)), ("all_frame", list(range(w.T)))):
            out = torch.empty((len(ids) * w.N, w.heads, w.head_dim), dtype=q.dtype, device="cuda")

            def call():
                rf.rf_keyframe_attention_ws(q, k, v, ids, w.T, w.H, w.W, out=out, workspace=ws)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            while time.perf_counter() - t0 < 0.3:
                call()
                torch.cuda.synchronize()
            n = max(3, min(20, int(0.4 / max(1e-4, (time.perf_counter() - t0) / 10))))
            ev = _events(n)
            for a, b in ev:
                a.record()
                call()
                b.record()
            torch.cuda.synchronize()
            ms = _avg_ms(ev)
            flop = accounting.attention_flops(len(ids) * w.N, w.S, w.head_dim, w.heads)
            tf = flop / (ms * 1e-3) / 1e12
            row[what] = {"avg_ms": round(ms, 4), "tflops": round(tf, 2), "frac_bf16_peak": round(tf / PEAK_BF16_TFLOPS, 4),
                         "launches": n, "flop_per_launch": flop}
            del out
        row["speedup_vs_all_frame"] = round(row["all_frame"]["avg_ms"] / row["keyframe_query"]["avg_ms"], 4)
        row["ideal_speedup"] = round(accounting.ideal_speedup(w.T, w.M), 4)
        print(f"[bench] {name}: keyframe-query {row['keyframe_query']['avg_ms']:.3f} ms = "
              f"{row['keyframe_query']['tflops']:.1f} TFLOP/s, all-frame {row['all_frame']['avg_ms']:.3f} ms, speedup "
              f"{row['speedup_vs_all_frame']:.3f} (ideal {row['ideal_speedup']:.3f})", file=sys.stderr, flush=True)
        res[name] = row
        del q, k, v, ws
        torch.cuda.empty_cache()
    return res


def _gpu_rows(w, q, k, v, pair_rows, pair_heads):
    """The GPU's keyframe-query attention output (the timed call, split-key
    tail included) on the oracle's own inputs q, k, v (host tensors, copied
    to the device bit for bit) at the listed (compact row, head) pairs, as
    exact float64."""
    import numpy as np
    import torch
    from paper_2606_06309_amd import binding as rf

    q, k, v = (x.cuda() for x in (q, k, v))
    out = rf.rf_keyframe_attention_ws(q, k, v, list(w.keyframes), w.T, w.H, w.W)
    torch.cuda.synchronize()
    sel = out[torch.as_tensor(pair_rows, device="cuda"), torch.as_tensor(pair_heads, device="cuda")]
    if sel.dtype == torch.bfloat16:
        bits = sel.cpu().contiguous().view(torch.int16).numpy().view(np.uint16)
        return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return sel.cpu().double().numpy()


def cpu_per_config(gpu_tflops):
    """The oracle per configuration, as the CPU baseline plan states it: the tiny
    workload in full; the small workload one head in full (all 7,800 rows over
    20,280 keys) extrapolated to its 12 heads; the larger ones on seeded row
    samples extrapolated to every (row, head) pair (each costs exactly 4*S*d
    FLOP); the projection oracle on the 480p latents and the selection oracle
    (frame cosine on the long workload's latent grid plus Alg. 1's scan) in full.
    The oracle rows computed for the timing also give each configuration's
    error statistics: the GPU's output at the same (row, head) pairs against
    them (max and mean absolute error, relative Frobenius error)."""
    import numpy as np
    import oracle
    from paper_2606_06309_amd import accounting, workloads

    out = {}
    rng = np.random.default_rng(2027)
    plan = {"tiny": None, "small": "one head", "480p": 64, "720p": 64, "long": 64, "wan-1.3b": 32, "cogvideox": 16}
    for name, how in plan.items():
        w = workloads.WORKLOADS[name]
        q, k, v = workloads.make_qkv(w)
        rowmap = oracle.rowmap(w.keyframes, w.N)
        if how is None:
            rows, heads = np.repeat(np.arange(rowmap.size), w.heads), np.tile(np.arange(w.heads), rowmap.size)
            label = "in full"
        elif how == "one head":
            rows, heads = np.arange(rowmap.size), np.zeros(rowmap.size, dtype=np.int64)
            label = f"head 0 in full ({rowmap.size} rows), extrapolated to {w.heads} heads"
        else:
            rows = np.concatenate([rng.choice(rowmap.size, how, replace=False) for _ in range(w.heads)])
            heads = np.repeat(np.arange(w.heads), how)
            label = f"{how} random rows per head ({rows.size} pairs), extrapolated to {rowmap.size * w.heads} pairs"
        toks = rowmap[rows]
        t0 = time.perf_counter()
        ref = oracle.attention_pairs(q, k, v, toks, heads)
        dt = time.perf_counter() - t0
        pairs_total = rowmap.size * w.heads
        sec = dt * pairs_total / toks.size
        flop = accounting.attention_flops(w.M * w.N, w.S, w.head_dim, w.heads)
        tf = flop / sec / 1e12
        row = {"seconds": round(sec, 3), "tflops": round(tf, 6), "measured_s": round(dt, 2), "sample": label,
               "extrapolated": how is not None}
        g = gpu_tflops.get(name)
        if g:
            row["gpu_over_cpu"] = round(g / tf, 1)
        got = _gpu_rows(w, q, k, v, rows, heads)
        err = np.abs(got - ref)
        row["gpu_error"] = {"max_abs": float(err.max()), "mean_abs": float(err.mean()),
                            "rel_fro": float(np.linalg.norm(got - ref) / np.linalg.norm(ref)),
                            "pairs": int(rows.size)}
        out[name] = row
        print(f"[bench] oracle {name}: {sec:.2f} s per launch ({label})", file=sys.stderr, flush=True)
    w = workloads.WORKLOADS["480p"]
    Hl, Wl = w.latent_hw
    lat = workloads.make_latents(w, B=1)
    mask = oracle.keyframe_mask(w.keyframes, w.T)
    t0 = time.perf_counter()
    oracle.project_latents(lat, 1, w.latent_c, w.T, Hl, Wl, w.timesteps, mask)
    dt = time.perf_counter() - t0
    nb = accounting.projection_bytes(1, w.latent_c, w.T, Hl * Wl, w.M, 4)
    out["projection_480p"] = {"seconds": round(dt, 4), "gbs": round(nb / dt / 1e9, 3), "bytes": nb, "sample": "in full"}
    w = workloads.WORKLOADS["long"]
    Hl, Wl = w.latent_hw
    x = workloads.make_scene_latents(1, w.latent_c, w.T, Hl, Wl, tuple(range(5, w.T, 6)), noise=0.5)
    t0 = time.perf_counter()
    sim = oracle.frame_cosine(x, 1, w.latent_c, w.T, Hl, Wl)
    oracle.select_keyframes_adaptive(sim[0], 0.5, w.M, 0.05, 2.0, 2.0)
    dt = time.perf_counter() - t0
    out["selection_long"] = {"seconds": round(dt, 4), "gbs": round(x.numel() * 4 / dt / 1e9, 3),
                             "sample": "in full (frame cosine of f32 proxies + Alg. 1's scan)"}
    return out


def selection(w, args):
    """Content-aware keyframe selection (Sec. 3.1, Alg. 1) on synthetic
    clean-latent proxies of the workload's latent grid with scene cuts: the
    frame cosine similarity on the GPU (bytes = the proxies read once) and
    Alg. 1's scan on the host."""
    import torch
    from paper_2606_06309_amd import binding as rf, workloads

    Hl, Wl = w.latent_hw
    cuts = tuple(range(5, w.T, 6))
    x = workloads.make_scene_latents(1, w.latent_c, w.T, Hl, Wl, cuts, noise=0.5, device="cuda")
    ws = torch.empty(rf.rf_frame_similarity_workspace(1, w.latent_c, w.T, Hl, Wl),
                     dtype=torch.uint8, device="cuda")
    sim = torch.empty((1, w.T, w.T), dtype=torch.float64, device="cuda")
    for _ in range(3):
        rf.rf_frame_similarity(x, out=sim, workspace=ws)
    torch.cuda.synchronize()
    n = max(5, args.steps)
    ev = _events(n)
    for a, b in ev:
        a.record()
        rf.rf_frame_similarity(x, out=sim, workspace=ws)
        b.record()
    torch.cuda.synchronize()
    ms = _avg_ms(ev)
    host = sim[0].cpu().numpy()
    t0 = time.perf_counter()
    ids, _ = rf.rf_select_keyframes_adaptive(host, 0.5, w.M, 0.05, 2.0, 2.0)
    scan_us = (time.perf_counter() - t0) * 1e6
    nbytes = x.numel() * x.element_size()
    gbs = nbytes / (ms * 1e-3) / 1e9
    # the HBM rate: a batch of videos of >= 1 GiB per launch, rotating through 3 such
    # batches so that no launch finds its input in the 256 MB Infinity Cache
    per = nbytes
    B = max(1, -(-(1 << 30) // per))
    batches = [workloads.make_scene_latents(B, w.latent_c, w.T, Hl, Wl, cuts, noise=0.5, seed=60 + i, device="cuda")
               for i in range(3)]
    wsb = torch.empty(rf.rf_frame_similarity_workspace(B, w.latent_c, w.T, Hl, Wl), dtype=torch.uint8, device="cuda")
    simb = torch.empty((B, w.T, w.T), dtype=torch.float64, device="cuda")
    for xb in batches:
        rf.rf_frame_similarity(xb, out=simb, workspace=wsb)
    torch.cuda.synchronize()
    evb = _events(6)
    for i, (a, b) in enumerate(evb):
        a.record()
        rf.rf_frame_similarity(batches[i % 3], out=simb, workspace=wsb)
        b.record()
    torch.cuda.synchronize()
    msb = _avg_ms(evb)
    gbs_b = per * B / (msb * 1e-3) / 1e9
    del batches, wsb, simb
    print(f"[bench] selection: similarity {ms * 1e3:.1f} us for one video (cache-resident, {gbs:.0f} GB/s); "
          f"batched {B} videos {msb * 1e3:.0f} us = {gbs_b:.0f} GB/s from HBM; scan {scan_us:.0f} us, "
          f"keyframes {ids.tolist()}", file=sys.stderr, flush=True)
    return {"similarity_single": {"avg_us": round(ms * 1e3, 2), "bytes": nbytes, "gbs": round(gbs, 1),
                                  "note": "one video re-read each launch: resident in the 256 MB Infinity Cache, "
                                          "a latency figure, not an HBM rate"},
            "similarity_batched": {"avg_us": round(msb * 1e3, 2), "bytes": per * B, "batch": B, "rotation_sets": 3,
                                   "gbs": round(gbs_b, 1), "frac_hbm": round(gbs_b / PEAK_HBM_GBS, 4)},
            "scan_us": round(scan_us, 1),
            "keyframes": ids.tolist(), "proxies": f"f32 [1][{w.latent_c}][{w.T}][{Hl}][{Wl}], scene cuts {list(cuts)}"}


def frame_mask(w, q, k, v, ws, args):
    """Keyframe-only attention (a frame-level key/value mask; Sec. 4's
    ablations): the keyframes' queries over the keyframes' keys only, timed
    like the main attention launch."""
    import torch
    from paper_2606_06309_amd import accounting, binding as rf

    out = torch.empty((w.M * w.N, w.heads, w.head_dim), dtype=q.dtype, device="cuda")
    need = rf.rf_attention_workspace(w.M, w.M, w.T, w.H, w.W, w.heads, w.head_dim, q.dtype)
    wsm = ws if ws.numel() >= need else torch.empty(need, dtype=torch.uint8, device="cuda")
    rf.rf_frame_attention(q, k, v, w.keyframes, w.keyframes, w.T, w.H, w.W, out=out, workspace=wsm)
    torch.cuda.synchronize()
    n = max(3, args.steps)
    ev = _events(n)
    for a, b in ev:
        a.record()
        rf.rf_frame_attention(q, k, v, w.keyframes, w.keyframes, w.T, w.H, w.W, out=out, workspace=wsm)
        b.record()
    torch.cuda.synchronize()
    ms = _avg_ms(ev)
    flop = accounting.attention_flops(w.M * w.N, w.M * w.N, w.head_dim, w.heads)
    tf = flop / (ms * 1e-3) / 1e12
    print(f"[bench] keyframe-only attention: {ms:.3f} ms = {tf:.1f} TFLOP/s", file=sys.stderr, flush=True)
    del out
    return {"kv_frames": list(w.keyframes), "avg_ms": round(ms, 4), "tflops": round(tf, 2),
            "frac_bf16_peak": round(tf / PEAK_BF16_TFLOPS, 4), "flop_per_launch": flop}


def measured_peaks(attn_tflops):
    """What this device sustains under a pure load of one kind, beside the
    published peaks: the dense bf16 matrix cores (probe kernel of independent
    32x32x16 MFMA chains over random normal operands that change from one
    instruction to the next, 4 workgroups of 4 waves per compute unit, launches
    back to back, the second half averaged; the clock it implies at 4096 FLOP
    per CU and cycle; the same on zero operands, which do not toggle), the
    vendor library's 8192^3 bf16 product as a reference point, HBM reads
    (2 GiB, far beyond the 256 MB Infinity Cache, best of three run lengths),
    and LDS reads (16-byte and transposing 8-byte, at 8 waves per CU)."""
    import torch
    from paper_2606_06309_amd import binding as rf

    wg, rounds, n = 1024, 5000, 10

    def probe(ops):
        sink = rf.rf_probe_mfma_bf16(ops, wg, 2)
        torch.cuda.synchronize()
        ev = _events(n)
        for a, b in ev:
            a.record()
            rf.rf_probe_mfma_bf16(ops, wg, rounds, sink=sink)
            b.record()
        torch.cuda.synchronize()
        return wg * rounds * 2.0 ** 22 / (_avg_ms(ev[n // 2:]) * 1e-3) / 1e12

    g = torch.Generator(device="cpu").manual_seed(7)
    mfma_tf = probe(torch.randn((12, 64, 8), generator=g).to(torch.bfloat16).cuda())
    mfma_zero_tf = probe(torch.zeros((12, 64, 8), dtype=torch.bfloat16, device="cuda"))
    clock = mfma_tf * 1e12 / (256 * 4096) / 1e9

    # the vendor library's large product on the same kind of data (a reference point only)
    ga = torch.randn((8192, 8192), generator=g).to(torch.bfloat16).cuda()
    gb = torch.randn((8192, 8192), generator=g).to(torch.bfloat16).cuda()
    gc = torch.matmul(ga, gb)
    torch.cuda.synchronize()
    ev = _events(n)
    for a, b in ev:
        a.record()
        torch.matmul(ga, gb, out=gc)
        b.record()
    torch.cuda.synchronize()
    gemm_tf = 2.0 * 8192 ** 3 / (_avg_ms(ev[n // 2:]) * 1e-3) / 1e12
    del ga, gb, gc

    nbytes = 2 << 30
    src = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    best = (0.0, 0)
    # contiguous runs of 16 KB, 64 KB and 2 MB per workgroup of 1024 threads
    for wgr in (nbytes // 16384, nbytes // 65536, 1024):
        sink = rf.rf_probe_hbm_read(src, wgr)
        torch.cuda.synchronize()
        ev = _events(5)
        for a, b in ev:
            a.record()
            rf.rf_probe_hbm_read(src, wgr, sink=sink)
            b.record()
        torch.cuda.synchronize()
        gbs = nbytes / (_avg_ms(ev) * 1e-3) / 1e9
        best = max(best, (gbs, wgr))
        del sink
    del src

    # LDS reads: two workgroups of 4 waves per CU (the attention kernel's 8 waves), each
    # wave reading its workgroup's 64 KB per round. The longest workgroup's shader-clock
    # ticks span (nearly) the whole launch: the clock is those ticks over the event time,
    # and bytes per clock per CU the launch's bytes over CUs x those ticks.
    lds = {}
    lwg, lrounds = 512, 4000
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    for width in (16, 8):
        sink, ticks = rf.rf_probe_lds_read(lwg, 2, width)
        torch.cuda.synchronize()
        ev = _events(6)
        for a, b in ev:
            a.record()
            rf.rf_probe_lds_read(lwg, lrounds, width, sink=sink, ticks=ticks)
            b.record()
        torch.cuda.synchronize()
        ms = _avg_ms(ev[3:])
        tk = ticks.double()
        tmax, tmin = float(tk.max().item()), float(tk.min().item())
        nbytes_l = lwg * 4 * lrounds * 65536
        lds[f"width_{width}"] = {
            "tbs": round(nbytes_l / (ms * 1e-3) / 1e12, 2),
            "bytes_per_clk_per_cu": round(nbytes_l / (cus * tmax), 1),
            "clock_ghz_from_ticks": round(tmax / (ms * 1e-3) / 1e9, 3),
            "workgroup_ticks_min_over_max": round(tmin / tmax, 3),
            "read": "16-byte" if width == 16 else "transposing 8-byte"}
        del sink, ticks
    print(f"[bench] measured peaks: bf16 MFMA {mfma_tf:.0f} TFLOP/s on random operands (clock {clock:.2f} GHz), "
          f"{mfma_zero_tf:.0f} on zero operands; library GEMM {gemm_tf:.0f}; HBM read {best[0]:.0f} GB/s; "
          f"LDS {lds['width_16']['bytes_per_clk_per_cu']} B/clk/CU (16-byte), "
          f"{lds['width_8']['bytes_per_clk_per_cu']} (transposing 8-byte)", file=sys.stderr, flush=True)
    return {"mfma_bf16": {"tflops": round(mfma_tf, 1), "spec_tflops": PEAK_BF16_TFLOPS,
                          "frac_spec": round(mfma_tf / PEAK_BF16_TFLOPS, 4), "clock_ghz": round(clock, 3),
                          "workgroups": wg, "rounds": rounds, "operands": "random normal bf16",
                          "launches_averaged": n - n // 2, "zero_operands_tflops": round(mfma_zero_tf, 1)},
            "library_gemm_bf16": {"tflops": round(gemm_tf, 1), "shape": [8192, 8192, 8192],
                                  "call": "torch.matmul, random normal bf16"},
            "hbm_read": {"gbs": round(best[0], 1), "spec_gbs": PEAK_HBM_GBS,
                         "frac_spec": round(best[0] / PEAK_HBM_GBS, 4), "bytes": nbytes, "workgroups": best[1],
                         "run_bytes": nbytes // best[1]},
            "lds_read": dict(lds, workgroups=lwg, rounds=lrounds, compute_units=cus),
            "attention_frac_of_measured_mfma": round(attn_tflops / mfma_tf, 4)}


def head_shard(w, args):
    """One GPU's share if the path were sharded by head over 8 GPUs: the same
    frames and keyframes with heads / 8 heads (no exchange between GPUs is
    needed, each holds its heads' full-length Q, K, V)."""
    import torch
    from paper_2606_06309_amd import accounting, binding as rf, workloads

    heads = max(1, w.heads // 8)
    ws_ = workloads.custom(w.T, w.H, w.W, heads, w.head_dim, w.keyframes, dtype=w.dtype, seed=950)
    q, k, v = workloads.make_qkv(ws_, device="cuda")
    out = torch.empty((ws_.M * ws_.N, heads, ws_.head_dim), dtype=q.dtype, device="cuda")
    wsp = torch.empty(max(16, rf.rf_attention_workspace(ws_.M, ws_.T, ws_.T, ws_.H, ws_.W, heads, ws_.head_dim,
                                                        q.dtype)), dtype=torch.uint8, device="cuda")
    rf.rf_keyframe_attention_ws(q, k, v, ws_.keyframes, ws_.T, ws_.H, ws_.W, out=out, workspace=wsp)
    torch.cuda.synchronize()
    n = max(3, args.steps)
    ev = _events(n)
    for a, b in ev:
        a.record()
        rf.rf_keyframe_attention_ws(q, k, v, ws_.keyframes, ws_.T, ws_.H, ws_.W, out=out, workspace=wsp)
        b.record()
    torch.cuda.synchronize()
    ms = _avg_ms(ev)
    flop = accounting.attention_flops(ws_.M * ws_.N, ws_.S, ws_.head_dim, heads)
    tf = flop / (ms * 1e-3) / 1e12
    print(f"[bench] one GPU's head share ({heads} of {w.heads} heads): {ms:.3f} ms = {tf:.1f} TFLOP/s",
          file=sys.stderr, flush=True)
    del q, k, v, out, wsp
    return {"heads": heads, "of_heads": w.heads, "gpus": 8, "avg_ms": round(ms, 4), "tflops": round(tf, 2),
            "frac_bf16_peak": round(tf / PEAK_BF16_TFLOPS, 4)}


def schedule_loop(w, ws, args):
    """A whole denoising schedule (Eq. 2, Alg. 2) at the workload's shape,
    attention path only, three ways on the same plan:
      latent: warm-up steps and Rhythmic Points run attention with every
        frame's queries; skipped steps project the non-keyframe latents
        (Eq. 3, the plan's interval and time) and run keyframe-query
        attention plus the scatter;
      cache: as latent, but the skipped steps take the non-keyframes' keys
        and values from the per-layer rolling cache (App. B.2): initialised
        from the last warm-up step's output, shift-and-store at each Rhythmic
        Point, projection into K and V before each keyframe-query attention;
        each stored state is labelled with its own step, so the skipped steps
        that follow clamp the weight to 1;
      cache_interp: as cache, with each stored state labelled with the time its
        update leads the non-keyframes to, so the skipped steps interpolate
        (0 < alpha < 1) between the two cached states;
      dense: every step all-frame attention (the reference).
    Q/K/V alternate between two seeded sets. `ideal_flop_ratio` is the FLOP
    ratio of the plan."""
    import torch
    from paper_2606_06309_amd import accounting, binding as rf, workloads

    T_steps, T_w, T_mid, n_s, n_l = (int(x) for x in args.schedule.split(","))
    plan = rf.rf_async_schedule(T_steps, T_w, T_mid, n_s, n_l)
    ids, mask = rf.rf_select_keyframes(w.keyframes, w.T)
    all_ids = list(range(w.T))
    nonkey = [f for f in all_ids if f not in set(ids.tolist())]
    sets = [workloads.make_qkv(w, device="cuda", seed=900 + i) for i in range(2)]
    lat = workloads.make_latents(w, B=1, device="cuda")
    Hl, Wl = w.latent_hw
    proj = torch.empty((1, w.latent_c, w.T, Hl, Wl), dtype=lat.dtype, device="cuda")
    dt = sets[0][0].dtype
    kq_out = torch.empty((w.M * w.N, w.heads, w.head_dim), dtype=dt, device="cuda")
    full_out = torch.empty((w.S, w.heads, w.head_dim), dtype=dt, device="cuda")
    D = w.heads * w.head_dim
    el = torch.tensor([], dtype=dt).element_size()
    store = torch.empty(rf.rf_cache_store_bytes(len(nonkey), w.N, D, dt) // el, dtype=dt, device="cuda") \
        if nonkey else None

    def run(mode):
        cache = None
        for i, step in enumerate(plan):
            q, k, v = sets[i % 2]
            if mode == "dense" or step["phase"] != "skip":
                rf.rf_keyframe_attention_ws(q, k, v, all_ids, w.T, w.H, w.W, out=full_out, workspace=ws)
                if mode.startswith("cache") and nonkey:
                    label = float(step["nonkey_to"] if mode == "cache_interp" else step["t"])
                    if cache is None:
                        if step["phase"] == "warmup" and i + 1 < len(plan) and plan[i + 1]["phase"] == "warmup":
                            continue
                        cache = rf.rf_cache_init(nonkey, w.T, w.N, D, dt, label, store=store, h_full=full_out)
                    elif step["phase"] == "rhythmic":
                        rf.rf_cache_shift_store(cache, label, store=store, h_full=full_out)
            else:
                if mode.startswith("cache") and cache is not None:
                    if mode == "cache_interp":
                        alphas.append(rf.rf_cache_alpha(cache, nonkey[0], float(step["t"])))
                    rf.rf_cache_project_kv(cache, store, k, v, float(step["t"]))
                else:
                    rf.rf_project_latents(lat, (step["t_start"], step["t_end"], step["t"]), mask, out=proj)
                rf.rf_keyframe_attention_ws(q, k, v, ids, w.T, w.H, w.W, out=kq_out, workspace=ws)
                rf.rf_scatter_frames(kq_out, full_out, ids, w.T, w.N)

    times = {}
    alphas = []
    for mode in ("latent", "cache", "cache_interp", "dense"):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record()
        run(mode)
        b.record()
        torch.cuda.synchronize()
        times[mode] = a.elapsed_time(b)
        print(f"[bench] schedule loop ({mode}): {times[mode]:.1f} ms", file=sys.stderr, flush=True)
    led = accounting.schedule_attention_flops(plan, w.T, w.M, w.N, w.head_dim, w.heads)
    del sets, lat, proj, kq_out, full_out, store
    return {"T_steps": T_steps, "T_w": T_w, "T_mid": T_mid, "n_small": n_s, "n_large": n_l,
            "steps": led["steps"], "async_ms": round(times["latent"], 2),
            "async_cache_ms": round(times["cache"], 2), "async_cache_interp_ms": round(times["cache_interp"], 2),
            "cache_interp_alpha_range": [round(min(alphas), 4), round(max(alphas), 4)] if alphas else None,
            "dense_ms": round(times["dense"], 2),
            "speedup": round(times["dense"] / times["latent"], 4),
            "speedup_cache": round(times["dense"] / times["cache"], 4),
            "speedup_cache_interp": round(times["dense"] / times["cache_interp"], 4),
            "ideal_flop_ratio": round(led["ratio"], 4),
            "tflops_async": round(led["flop"] / (times["latent"] * 1e-3) / 1e12, 1)}


def rolling_cache(w, args):
    """Rolling cache of App. B.2 at the workload's shape: every non-keyframe
    cached (bf16 [N][heads*head_dim] states). Times the projection of the
    cached frames into K and V at a skipped step and the shift-and-store copy
    of a denoising step; both move well over the 256 MB Infinity Cache."""
    import torch
    from paper_2606_06309_amd import accounting, binding as rf, workloads

    nk = [f for f in range(w.T) if f not in w.keyframes]
    D = w.heads * w.head_dim
    el = torch.tensor([], dtype=w.torch_dtype).element_size()
    store = torch.empty(rf.rf_cache_store_bytes(len(nk), w.N, D, w.torch_dtype) // el,
                        dtype=w.torch_dtype, device="cuda")
    h0 = workloads.make_hidden(w, 0, device="cuda")
    h1 = workloads.make_hidden(w, 1, device="cuda")
    k = torch.empty((w.S, w.heads, w.head_dim), dtype=w.torch_dtype, device="cuda")
    v = torch.empty_like(k)
    c = rf.rf_cache_init(nk, w.T, w.N, D, w.torch_dtype, 1000.0, store=store, h_full=h0)
    t = 1000.0
    n = max(5, args.steps)
    evs = _events(n)
    for i in range(n):
        t -= 3.0
        evs[i][0].record()
        rf.rf_cache_shift_store(c, t, store=store, h_full=h1 if i % 2 == 0 else h0)
        evs[i][1].record()
    for _ in range(2):
        rf.rf_cache_project_kv(c, store, k, v, t + 1.0)
    torch.cuda.synchronize()
    evp = _events(n)
    for i in range(n):
        evp[i][0].record()
        rf.rf_cache_project_kv(c, store, k, v, t + 1.0)
        evp[i][1].record()
    torch.cuda.synchronize()
    p_ms, s_ms = _avg_ms(evp), _avg_ms(evs)
    fb = w.N * D * el
    pb = accounting.cache_projection_bytes(len(nk), fb)
    sb = accounting.cache_store_bytes(len(nk), fb)
    p_gbs = pb / (p_ms * 1e-3) / 1e9
    s_gbs = sb / (s_ms * 1e-3) / 1e9
    print(f"[bench] rolling cache: projection {p_ms * 1e3:.1f} us ({p_gbs:.0f} GB/s), "
          f"shift-and-store {s_ms * 1e3:.1f} us ({s_gbs:.0f} GB/s), {len(nk)} frames",
          file=sys.stderr, flush=True)

    # a whole skipped step, unfused (projection into K and V, then attention) against
    # the fused form (projected tiles formed inside the attention kernel), same inputs
    q, kq, vq = workloads.make_qkv(w, device="cuda")
    ids = list(w.keyframes)
    out = torch.empty((w.M * w.N, w.heads, w.head_dim), dtype=q.dtype, device="cuda")
    wsa = torch.empty(max(16, rf.rf_attention_workspace(w.M, w.T, w.T, w.H, w.W, w.heads, w.head_dim, q.dtype)),
                      dtype=torch.uint8, device="cuda")
    t_skip = t + 1.0

    def unfused():
        rf.rf_cache_project_kv(c, store, kq, vq, t_skip)
        rf.rf_keyframe_attention_ws(q, kq, vq, ids, w.T, w.H, w.W, out=out, workspace=wsa)

    def fused():
        rf.rf_keyframe_attention_cached(q, kq, vq, ids, w.T, w.H, w.W, c, store, t_skip, out=out, workspace=wsa)

    step = {}
    for name, fn in (("unfused", unfused), ("fused", fused)) * 2:    # interleaved twice, best kept
        fn()
        torch.cuda.synchronize()
        n_s = max(3, min(args.steps, 6))
        ev = _events(n_s)
        for a, b in ev:
            a.record()
            fn()
            b.record()
        torch.cuda.synchronize()
        step[name] = min(step.get(name, 1e30), _avg_ms(ev))
    flop = accounting.attention_flops(w.M * w.N, w.S, w.head_dim, w.heads)
    print(f"[bench] skipped step with the rolling cache: unfused {step['unfused']:.3f} ms, "
          f"fused {step['fused']:.3f} ms", file=sys.stderr, flush=True)
    del store, h0, h1, k, v, q, kq, vq, out, wsa
    return {"cached_frames": len(nk), "frame_bytes": fb,
            "skip_step": {"unfused_ms": round(step["unfused"], 4), "fused_ms": round(step["fused"], 4),
                          "unfused_tflops": round(flop / (step["unfused"] * 1e-3) / 1e12, 2),
                          "fused_tflops": round(flop / (step["fused"] * 1e-3) / 1e12, 2),
                          "fused_over_unfused": round(step["unfused"] / step["fused"], 4)},
            "projection": {"bytes": pb, "avg_us": round(p_ms * 1e3, 2), "gbs": round(p_gbs, 1),
                           "frac_hbm": round(p_gbs / PEAK_HBM_GBS, 4)},
            "shift_store": {"bytes": sb, "avg_us": round(s_ms * 1e3, 2), "gbs": round(s_gbs, 1),
                            "frac_hbm": round(s_gbs / PEAK_HBM_GBS, 4)}}


def bandwidth(w, q, attn_out, full_out, args):
    """Projection and gather/scatter bandwidth. A single projection at the
    workload's latent size fits in the 256 MB Infinity Cache, so the HBM rate
    is taken on a batch of >= 1 GB per launch, rotating through 3 buffer sets
    (each set larger than the cache); the single-launch latency is reported
    beside it. Gather and scatter at this size already exceed the cache."""
    import torch
    from paper_2606_06309_amd import accounting, binding as rf, workloads

    dev = "cuda"
    n = max(3, args.steps)
    ids, mask = rf.rf_select_keyframes(w.keyframes, w.T)
    Hl, Wl = w.latent_hw
    plane = Hl * Wl
    per_b = accounting.projection_bytes(1, w.latent_c, w.T, plane, w.M, 4)
    B = max(1, -(-(1 << 30) // per_b))
    sets = []
    for s in range(3):
        lat = workloads.make_latents(w, B=B, device=dev, seed=500 + s)
        sets.append((lat, torch.empty((B, w.latent_c, w.T, Hl, Wl), dtype=lat.dtype, device=dev)))
    for lat, out in sets:
        rf.rf_project_latents(lat, w.timesteps, mask, out=out)
    torch.cuda.synchronize()
    ev = _events(n)
    for i in range(n):
        lat, out = sets[i % 3]
        ev[i][0].record()
        rf.rf_project_latents(lat, w.timesteps, mask, out=out)
        ev[i][1].record()
    torch.cuda.synchronize()
    proj_ms = _avg_ms(ev)
    proj_bytes = per_b * B
    del sets

    lat1 = workloads.make_latents(w, B=1, device=dev)
    out1 = torch.empty((1, w.latent_c, w.T, Hl, Wl), dtype=lat1.dtype, device=dev)
    rf.rf_project_latents(lat1, w.timesteps, mask, out=out1)
    ev1 = _events(n)
    for i in range(n):
        ev1[i][0].record()
        rf.rf_project_latents(lat1, w.timesteps, mask, out=out1)
        ev1[i][1].record()
    torch.cuda.synchronize()
    single_ms = _avg_ms(ev1)

    row_bytes = w.heads * w.head_dim * q.element_size()
    g_bytes = accounting.gather_bytes(w.M, w.N, row_bytes)
    dsts = [attn_out, torch.empty_like(attn_out)]
    rf.rf_gather_frames(q, ids, w.T, w.N, out=dsts[0])
    torch.cuda.synchronize()
    evg = _events(n)
    for i in range(n):
        evg[i][0].record()
        rf.rf_gather_frames(q, ids, w.T, w.N, out=dsts[i % 2])
        evg[i][1].record()
    evs = _events(n)
    for i in range(n):
        evs[i][0].record()
        rf.rf_scatter_frames(dsts[i % 2], full_out, ids, w.T, w.N)
        evs[i][1].record()
    torch.cuda.synchronize()
    g_ms, s_ms = _avg_ms(evg), _avg_ms(evs)

    def rate(b, ms):
        gbs = b / (ms * 1e-3) / 1e9
        return {"bytes": b, "avg_us": round(ms * 1e3, 2), "gbs": round(gbs, 1),
                "frac_hbm": round(gbs / PEAK_HBM_GBS, 4)}

    res = {"projection_batched": dict(rate(proj_bytes, proj_ms), batch=B, dtype="f32",
                                      rotation_sets=3),
           "projection_single": dict(rate(per_b, single_ms), batch=1, dtype="f32"),
           "gather": rate(g_bytes, g_ms), "scatter": rate(g_bytes, s_ms)}
    print(f"[bench] projection {res['projection_batched']['gbs']} GB/s (B={B}), single "
          f"{res['projection_single']['avg_us']} us; gather {res['gather']['gbs']} GB/s, "
          f"scatter {res['scatter']['gbs']} GB/s", file=sys.stderr, flush=True)
    return res


if __name__ == "__main__":
    main()
