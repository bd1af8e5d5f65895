"""FLOP and byte accounting for the keyframe-query attention path.

Two counts live here:

* The per-launch counts used for rooflines. Attention performs two matrix
  products per head (scores Q K^T and the weighted sum P V), each of
  Mq x S x d multiply-adds at 2 FLOP per multiply-add, so one launch does
  4 * Mq * S * d * heads FLOP; the softmax is left out, as in App. B.1.
  Algorithmic bytes read or write every operand exactly once.

* The paper's own analytic model (App. B.1), kept as written: per layer
  4 S D^2 + 2 S^2 D (+ 3 S^2 for the softmax), summed over warm-up, skip and
  full denoising steps. It counts one FLOP per multiply-add and models a skip
  step as keyframe-only attention (M*N tokens on both sides); it is context,
  not the count used for rooflines.
"""
import math


def attention_flops(Mq: int, S: int, head_dim: int, heads: int) -> int:
    """FLOP of one keyframe-query attention launch (2 FLOP per multiply-add)."""
    return 4 * Mq * S * head_dim * heads


def attention_bytes(Mq: int, S: int, head_dim: int, heads: int, elem_bytes: int) -> int:
    """Algorithmic bytes of one attention launch: the Mq gathered query rows,
    all S key and value rows, and the Mq output rows, each moved once."""
    row = heads * head_dim * elem_bytes
    return (Mq + 2 * S + Mq) * row


def projection_bytes(B: int, C: int, T: int, plane: int, n_keyframes: int,
                     elem_bytes: int, aliased: bool = False) -> int:
    """Algorithmic bytes of one projection launch over [B][2][C][T][plane]:
    a non-keyframe plane reads both snapshots and writes one; a keyframe plane
    reads the current state and writes it (nothing when out aliases slot 1)."""
    nonkey = T - n_keyframes
    per_bc = nonkey * 3 + (0 if aliased else n_keyframes * 2)
    return B * C * per_bc * plane * elem_bytes


def gather_bytes(M: int, rows_per_frame: int, row_bytes: int) -> int:
    """Bytes of one frame gather or scatter: every moved row read and written."""
    return 2 * M * rows_per_frame * row_bytes


def cache_projection_bytes(n_frames: int, frame_bytes: int) -> int:
    """Bytes of one rolling-cache projection launch (App. B.2): per projected
    frame both cached states are read and the result is written as the key
    and as the value."""
    return 4 * n_frames * frame_bytes


def cache_store_bytes(n_frames: int, frame_bytes: int) -> int:
    """Bytes of one cache store (initialisation or shift-and-store): each
    frame's new state read from the attention output and written to its slot."""
    return 2 * n_frames * frame_bytes


def schedule_attention_flops(plan, T_frames: int, M: int, N: int, head_dim: int, heads: int):
    """Attention FLOP of one layer over a whole step plan (Alg. 2): warm-up
    steps and Rhythmic Points evaluate every frame's queries over all keys,
    skipped steps only the keyframes' queries (still over all keys).
    `plan` is a list of per-step dicts with a "phase" of "warmup", "rhythmic"
    or "skip". Returns the per-phase step counts, FLOP, the dense FLOP (every
    step full) and their ratio."""
    S = T_frames * N
    full = attention_flops(S, S, head_dim, heads)
    kq = attention_flops(M * N, S, head_dim, heads)
    counts = {"warmup": 0, "rhythmic": 0, "skip": 0}
    for step in plan:
        counts[step["phase"]] += 1
    total = (counts["warmup"] + counts["rhythmic"]) * full + counts["skip"] * kq
    dense = len(plan) * full
    return {"steps": counts, "full_step_flop": full, "skip_step_flop": kq, "flop": total,
            "dense_flop": dense, "ratio": dense / total if total else float("nan")}


# ---------------------------------------------------------------------------
# the paper's analytic model, App. B.1 (kept as the paper states it)
# ---------------------------------------------------------------------------

def paper_layer_flops(S: int, D: int, include_softmax: bool = False) -> int:
    """Per-layer FLOP of the dense DiT self-attention block, App. B.1:
    QKV projection 3 S D^2, scores S^2 D, aggregation S^2 D, output projection
    S D^2, and optionally the softmax's 3 S^2."""
    f = 4 * S * D * D + 2 * S * S * D
    if include_softmax:
        f += 3 * S * S
    return f


def paper_dense_flops(L: int, T: int, S: int, D: int) -> int:
    """Dense baseline over L layers and T steps, App. B.1."""
    return L * T * paper_layer_flops(S, D)


def paper_step_counts(T: int, T_warmup: int, n: int):
    """(T_RhymeFlow, N_skip, N_denoise) of App. B.1:
    N_skip = floor(T_RhymeFlow * (n - 1) / n), N_denoise = T_RhymeFlow - N_skip."""
    t_rf = T - T_warmup
    n_skip = (t_rf * (n - 1)) // n
    return t_rf, n_skip, t_rf - n_skip


def paper_rhymeflow_flops(L: int, T: int, T_warmup: int, F: int, N: int, D: int,
                          M: int, n: int):
    """Warm-up, skip and denoise FLOP of App. B.1, as the paper models them
    (skip steps as attention over the M*N keyframe tokens only)."""
    _, n_skip, n_den = paper_step_counts(T, T_warmup, n)
    S = F * N
    warm = L * T_warmup * paper_layer_flops(S, D)
    skip = L * n_skip * paper_layer_flops(M * N, D)
    den = L * n_den * paper_layer_flops(S, D)
    return {"warmup": warm, "skip": skip, "denoise": den, "total": warm + skip + den}


def ideal_speedup(T: int, M: int) -> float:
    """Ratio of all-frame to keyframe-query attention FLOP at one shape: T / M."""
    return T / M if M else math.inf
