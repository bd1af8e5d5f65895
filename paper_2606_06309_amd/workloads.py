"""Seeded synthetic workloads shaped like the paper's video-DiT attention.

This module only draws inputs: shapes, seeds and random tensors. It holds none
of the method's arithmetic and imports neither the HIP library nor the oracle,
so both sides of every parity check can take their inputs from it.

The paper measured Wan2.1-T2V-1.3B (21 latent frames x 3,600 tokens, 12 heads,
head_dim 128), CogVideoX-v1.5 and HunyuanVideo on a prompt benchmark (Sec. 4).
No weights or prompts are available here, so Q/K/V and latents are i.i.d.
normal draws with the shapes of those workloads:

  tiny     T=5  x 8x8   (320 tokens),     2 heads, d=64,  fp32, keyframes {0,2,4}
  small    T=13 x 30x52 (20,280 tokens), 12 heads, d=128, bf16, Q/K/V scaled by
           1/sqrt(128), keyframes every 3rd frame {0,3,6,9,12}
  480p     T=21 x 30x52 (32,760 tokens), 12 heads, d=128, bf16, 6 evenly spaced
           keyframes including first and last {0,4,8,12,16,20}
  720p     T=21 x 45x80 (75,600 tokens, the Wan2.1 720p grid), 40 heads,
           d=128, bf16, first frame + every 4th {0,4,8,12,16,20}
  long     T=33 x 45x80 (118,800 tokens), 24 heads, d=128, bf16, every 6th
           frame {0,6,...,30} plus 2 extra keyframes drawn with
           numpy.random.default_rng(4) from the remaining frames ({22, 31})

Two more named shapes follow the paper's two models at their own sizes, with
the paper's default of 4 keyframes (Sec. 4.1), evenly spaced:

  wan-1.3b  T=21 x 45x80 (75,600 tokens), 12 heads, d=128, bf16 (Wan2.1-1.3B:
            21 latent frames of 3,600 tokens), keyframes {0,7,13,20}
  cogvideox T=11 x 48x85 (44,880 tokens), 48 heads, d=64, bf16 (CogVideoX-v1.5:
            11 latent frames of 4,080 tokens; 48 heads of 64 in that model's
            published configuration), keyframes {0,3,7,10}

Draw order: Q, K, V from one torch generator seeded with the workload's index
(tiny 0 ... long 4, wan-1.3b 5, cogvideox 6), fp32 randn, times the workload's scale, then rounded to
bf16 (round-to-nearest-even, torch's conversion) for the bf16 workloads.
Latents: slot 0 then slot 1, fp32 randn from a generator seeded index + 100.
Latent grids: tiny 4 x 5x16x16; 480p 16 x 21x60x104; the others 16 x T x 2H x 2W.
Projection timesteps (t_start, t_end, tau) = (24, 21, 23), i.e. alpha = 1/3.
Cached hidden states (the rolling cache's attention outputs): one
[S][heads][head_dim] fp32 randn draw per store, generator seeded index + 200 +
the store's number (0 = the warm-up state), rounded to the workload's dtype.
"""
from dataclasses import dataclass, field
from typing import List, Tuple

import numpy as np
import torch


@dataclass(frozen=True)
class Workload:
    name: str
    index: int
    T: int
    H: int
    W: int
    heads: int
    head_dim: int
    dtype: str                      # "f32" or "bf16"
    keyframes: Tuple[int, ...]
    qkv_scale: float
    latent_c: int
    latent_hw: Tuple[int, int]
    timesteps: Tuple[float, float, float] = (24.0, 21.0, 23.0)
    note: str = ""

    @property
    def N(self) -> int:
        return self.H * self.W

    @property
    def S(self) -> int:
        return self.T * self.H * self.W

    @property
    def M(self) -> int:
        return len(self.keyframes)

    @property
    def torch_dtype(self):
        return torch.float32 if self.dtype == "f32" else torch.bfloat16


def _long_video_keyframes() -> Tuple[int, ...]:
    base = list(range(0, 33, 6))
    rest = [f for f in range(33) if f not in base]
    extra = np.random.default_rng(4).choice(rest, 2, replace=False)
    return tuple(sorted(base + [int(x) for x in extra]))


WORKLOADS = {
    "tiny": Workload("tiny", 0, 5, 8, 8, 2, 64, "f32", (0, 2, 4), 1.0, 4, (16, 16)),
    "small": Workload("small", 1, 13, 30, 52, 12, 128, "bf16", (0, 3, 6, 9, 12),
                      1.0 / np.sqrt(128.0), 16, (60, 104)),
    "480p": Workload("480p", 2, 21, 30, 52, 12, 128, "bf16", (0, 4, 8, 12, 16, 20),
                     1.0, 16, (60, 104)),
    "720p": Workload("720p", 3, 21, 45, 80, 40, 128, "bf16", (0, 4, 8, 12, 16, 20),
                     1.0, 16, (90, 160)),
    "long": Workload("long", 4, 33, 45, 80, 24, 128, "bf16", _long_video_keyframes(),
                     1.0, 16, (90, 160)),
    "wan-1.3b": Workload("wan-1.3b", 5, 21, 45, 80, 12, 128, "bf16", (0, 7, 13, 20),
                         1.0, 16, (90, 160)),
    "cogvideox": Workload("cogvideox", 6, 11, 48, 85, 48, 64, "bf16", (0, 3, 7, 10),
                          1.0, 16, (96, 170)),
}
ORDER = ["tiny", "small", "480p", "720p", "long"]
MODEL_SHAPES = ["wan-1.3b", "cogvideox"]


def custom(T, H, W, heads, head_dim, keyframes, dtype="bf16", seed=0,
           qkv_scale=1.0, name="custom") -> Workload:
    """A workload of any shape (parity cases that span several tiles)."""
    return Workload(name, seed, T, H, W, heads, head_dim, dtype, tuple(keyframes),
                    qkv_scale, 4, (2 * H, 2 * W))


def make_qkv(w: Workload, device="cpu", seed=None, scale=None):
    """Q, K, V as [S][heads][head_dim] tensors on `device`."""
    g = torch.Generator(device=device)
    g.manual_seed(w.index if seed is None else seed)
    s = w.qkv_scale if scale is None else scale
    shape = (w.S, w.heads, w.head_dim)
    out = []
    for _ in range(3):
        x = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
        if s != 1.0:
            x.mul_(s)
        out.append(x.to(w.torch_dtype))
    return tuple(out)


def make_latents(w: Workload, B=1, device="cpu", dtype=None, seed=None):
    """Latents [B][2][C][T][Hl][Wl]: slot 0 and slot 1 are independent draws."""
    g = torch.Generator(device=device)
    g.manual_seed((w.index + 100) if seed is None else seed)
    Hl, Wl = w.latent_hw
    shape = (B, 2, w.latent_c, w.T, Hl, Wl)
    x = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    dt = torch.float32 if dtype is None else dtype
    return x.to(dt)


def sample_rows(w: Workload, per_head: int, tile: int = 128, seed: int = 1234):
    """A seeded sample of compact query rows: every keyframe's first and last
    row, rows on both sides of each `tile` boundary, the final row, and
    random rows up to `per_head`."""
    Mq = w.M * w.N
    must = set()
    for m in range(w.M):
        must.add(m * w.N)
        must.add(m * w.N + w.N - 1)
    for b in range(tile, Mq, tile * max(1, (Mq // tile) // 8)):
        must.add(b - 1)
        must.add(b)
    must.add(Mq - 1)
    rng = np.random.default_rng(seed)
    rows = sorted(r for r in must if 0 <= r < Mq)
    extra = max(0, per_head - len(rows))
    if extra:
        pool = np.setdiff1d(np.arange(Mq), np.array(rows))
        rows += rng.choice(pool, min(extra, pool.size), replace=False).tolist()
    return np.array(sorted(rows), dtype=np.int64)


def make_scene_latents(B: int, C: int, T: int, H: int, W: int, cut_frames, noise: float = 0.3,
                       seed: int = 7, device="cpu", dtype=torch.float32):
    """Synthetic clean-latent proxies [B][C][T][H][W] with scene cuts: frames of
    one scene share a random base and differ by independent noise of relative
    size `noise`; a new scene (new base) starts at every listed cut frame."""
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    cuts = sorted(set(int(f) for f in cut_frames) | {0})
    x = torch.empty((B, C, T, H, W), dtype=torch.float32, device=device)
    for si, start in enumerate(cuts):
        end = cuts[si + 1] if si + 1 < len(cuts) else T
        base = torch.randn((B, C, 1, H, W), generator=g, device=device)
        x[:, :, start:end] = base + noise * torch.randn((B, C, end - start, H, W), generator=g, device=device)
    return x.to(dtype)


def make_hidden(w: Workload, store: int, device="cpu", dtype=None):
    """Synthetic post-attention hidden states [S][heads][head_dim] for the
    rolling cache: store 0 is the state cached at the end of warm-up, store
    k >= 1 the k-th shift-and-store."""
    g = torch.Generator(device=device)
    g.manual_seed(w.index + 200 + store)
    x = torch.randn((w.S, w.heads, w.head_dim), generator=g, device=device, dtype=torch.float32)
    return x.to(w.torch_dtype if dtype is None else dtype)
