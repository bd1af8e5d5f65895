"""Plain, slow CPU oracle for the RhymeFlow keyframe-query attention path.

TEST INFRASTRUCTURE ONLY. Only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this package. It shares no code with
the HIP library and never imports it; nothing in the product path may call it.

Contents, each written from the paper (RhymeFlow, arXiv 2606.06309):

* keyframe-set handling (integer, pure Python): normalisation of an explicit
  frame list with the first frame forced (Sec. 3.1; Alg. 1 starts the set with
  the first frame), the stride and evenly-spaced ("Uniform", Sec. 4 selection
  ablation) policies, the keyframe mask, and the query row map that lists the
  tokens of every keyframe in order (App. B.1: a sequence is F frames of N
  tokens each, S = F x N);
* keyframe-query attention in fp64 (C, ``oracle.c``): keyframe queries attend
  over all frames' keys and values (Sec. 3.2.3-3.2.4; App. B.2);
* latent trajectory projection in fp64 (C), Eq. (3);
* frame gather / scatter on raw bit patterns (numpy fancy indexing);
* content-aware keyframe selection: the cosine similarity between latent
  frames in fp64 (C; Eq. 1's psi_sim) and the sequential scan of Alg. 1 with
  its dynamic threshold (pure Python);
* the per-layer rolling cache of App. B.2 (pure Python/numpy, fp64): two cached
  post-attention hidden states per non-keyframe with their timesteps,
  initialisation at the end of warm-up, shift-and-store at denoising steps,
  the projection with the epsilon form of alpha at skipped steps, and the
  key/value sequence in which the projected state is both key and value;
* the progressive asynchronous schedule (pure Python): Eq. 2's stride and
  Alg. 2's loop over the denoising steps (warm-up, Rhythmic Points, skipped
  steps with Eq. 3's interval and weight);
* attention under a frame-level key/value mask (the keys of listed frames
  only), through the same C attention routine on the selected keys.
"""
import ctypes
import math
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

F64, F32, BF16 = 0, 1, 2


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            from ._build import build_oracle
            build_oracle()
        lib = ctypes.CDLL(_LIB_PATH)
        i64p = ctypes.POINTER(ctypes.c_int64)
        dp = ctypes.POINTER(ctypes.c_double)
        lib.orc_attention_pairs.argtypes = [
            ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int,
            ctypes.c_int64, ctypes.c_int64, ctypes.c_int64,
            i64p, i64p, ctypes.c_int64, dp, dp]
        lib.orc_attention_pairs.restype = ctypes.c_int
        lib.orc_projection_alpha.argtypes = [ctypes.c_double] * 3
        lib.orc_projection_alpha.restype = ctypes.c_double
        lib.orc_project_latents.argtypes = [
            ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_int64,
            ctypes.c_int64, ctypes.c_int64, ctypes.POINTER(ctypes.c_uint8),
            ctypes.c_double, ctypes.c_double, ctypes.c_double, dp]
        lib.orc_project_latents.restype = ctypes.c_int
        lib.orc_frame_cosine.argtypes = [
            ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_int64,
            ctypes.c_int64, ctypes.c_int64, dp]
        lib.orc_frame_cosine.restype = ctypes.c_int
        lib.orc_num_threads.argtypes = []
        lib.orc_num_threads.restype = ctypes.c_int
        lib.orc_set_num_threads.argtypes = [ctypes.c_int]
        lib.orc_set_num_threads.restype = None
        _lib = lib
    return _lib


def num_threads() -> int:
    """Threads the C oracle's OpenMP loops use."""
    return int(_load().orc_num_threads())


def set_num_threads(n: int) -> None:
    """Threads for the C oracle's later OpenMP loops (for timing it)."""
    _load().orc_set_num_threads(int(n))


# ---------------------------------------------------------------------------
# input marshalling (exact bits; no arithmetic)
# ---------------------------------------------------------------------------

def as_oracle_array(x):
    """Return (contiguous numpy array, dtype code) holding the exact bits of x.

    Accepts numpy float64 / float32 / uint16 (bf16 bit patterns) arrays and CPU
    torch tensors of float64 / float32 / bfloat16.
    """
    if not isinstance(x, np.ndarray):
        import torch
        t = x.detach().cpu().contiguous()
        if t.dtype == torch.bfloat16:
            return t.view(torch.int16).numpy().view(np.uint16), BF16
        if t.dtype == torch.float32:
            return t.numpy(), F32
        if t.dtype == torch.float64:
            return t.numpy(), F64
        raise TypeError(f"unsupported tensor dtype {t.dtype}")
    a = np.ascontiguousarray(x)
    if a.dtype == np.float64:
        return a, F64
    if a.dtype == np.float32:
        return a, F32
    if a.dtype == np.uint16:
        return a, BF16
    raise TypeError(f"unsupported array dtype {a.dtype}")


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns (uint16) to float64."""
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


# ---------------------------------------------------------------------------
# keyframe sets (integer)
# ---------------------------------------------------------------------------

def select_keyframes(frame_ids, T: int, force_first: bool = True) -> np.ndarray:
    """Normalise an explicit frame list into the keyframe set K.

    K is a set of frame indices; the first frame always belongs to it (Sec. 3.1:
    the initial frame anchors the video; Alg. 1 initialises K with frame 1,
    index 0 here). Duplicates collapse, the result is sorted ascending, and any
    index outside [0, T) is an error.
    """
    if T <= 0:
        raise ValueError("T must be positive")
    chosen = set()
    for f in frame_ids:
        f = int(f)
        if f < 0 or f >= T:
            raise ValueError(f"frame id {f} outside [0, {T})")
        chosen.add(f)
    if force_first:
        chosen.add(0)
    if not chosen:
        raise ValueError("empty keyframe set")
    return np.array(sorted(chosen), dtype=np.int32)


def keyframe_mask(keyframe_ids, T: int) -> np.ndarray:
    """mask[f] = 1 exactly when frame f is a keyframe; non-keyframes are the
    complement of K (Alg. 1 returns N = {all frames} minus K)."""
    mask = np.zeros(T, dtype=np.uint8)
    for f in keyframe_ids:
        mask[int(f)] = 1
    return mask


def stride_keyframes(T: int, k: int) -> np.ndarray:
    """Frames 0, k, 2k, ... below T (a fixed-interval policy)."""
    if T <= 0 or k <= 0:
        raise ValueError("T and k must be positive")
    out = []
    f = 0
    while f < T:
        out.append(f)
        f += k
    return np.array(out, dtype=np.int32)


def uniform_keyframes(T: int, M: int) -> np.ndarray:
    """M evenly spaced frames from the first to the last ("Uniform" policy of
    the selection ablation, Sec. 4): frame i*(T-1)/(M-1) rounded half up,
    i = 0..M-1. M = 1 gives the first frame alone."""
    if T <= 0 or M <= 0 or M > T:
        raise ValueError("need 0 < M <= T")
    if M == 1:
        return np.array([0], dtype=np.int32)
    out = []
    for i in range(M):
        num = i * (T - 1)
        den = M - 1
        q, r = divmod(num, den)
        out.append(q + (1 if 2 * r >= den else 0))
    return np.array(out, dtype=np.int32)


def rowmap(keyframe_ids, N: int) -> np.ndarray:
    """Token index of each query row: the tokens of every keyframe, frame after
    frame in keyframe order, N tokens per frame (a sequence of F frames holds
    S = F x N tokens, App. B.1)."""
    rows = []
    for f in keyframe_ids:
        for n in range(N):
            rows.append(int(f) * N + n)
    return np.array(rows, dtype=np.int64)


# ---------------------------------------------------------------------------
# attention
# ---------------------------------------------------------------------------

def attention_pairs(q, k, v, tokens, heads_of_pair, return_probs=False):
    """fp64 attention of the listed (query token, head) pairs over all of k/v.

    q, k, v: [S][heads][d] (numpy or torch, exact bits). Returns [n][d]
    float64, and the [n][S] softmax rows when asked.
    """
    qa, dt = as_oracle_array(q)
    ka, dk = as_oracle_array(k)
    va, dv = as_oracle_array(v)
    if not (dt == dk == dv):
        raise TypeError("q, k, v must share a dtype")
    if qa.ndim != 3 or ka.shape != va.shape or ka.ndim != 3:
        raise ValueError("q, k, v must be [S][heads][d]")
    if qa.shape[1:] != ka.shape[1:]:
        raise ValueError("q and k differ in heads or head_dim")
    S, heads, d = ka.shape
    tok = np.ascontiguousarray(np.asarray(tokens, dtype=np.int64))
    hd = np.ascontiguousarray(np.asarray(heads_of_pair, dtype=np.int64))
    if tok.shape != hd.shape or tok.ndim != 1:
        raise ValueError("tokens and heads must be 1-D and equal length")
    if tok.size and (tok.min() < 0 or tok.max() >= qa.shape[0]):
        raise ValueError("query token out of range")
    n = tok.size
    out = np.zeros((n, d), dtype=np.float64)
    probs = np.zeros((n, S), dtype=np.float64) if return_probs else None
    lib = _load()
    dp = ctypes.POINTER(ctypes.c_double)
    i64p = ctypes.POINTER(ctypes.c_int64)
    rc = lib.orc_attention_pairs(
        qa.ctypes.data, ka.ctypes.data, va.ctypes.data, dt, S, heads, d,
        tok.ctypes.data_as(i64p), hd.ctypes.data_as(i64p), n,
        out.ctypes.data_as(dp),
        probs.ctypes.data_as(dp) if probs is not None else None)
    if rc != 0:
        raise RuntimeError("oracle attention failed")
    return (out, probs) if return_probs else out


def keyframe_attention(q, k, v, keyframe_ids, N: int, rows=None, heads=None,
                       return_probs=False):
    """Keyframe-query attention (Sec. 3.2.3-3.2.4; App. B.2).

    Query rows are the tokens of the keyframes (``rowmap``); keys and values
    are every token of every frame. Returns an array [len(rows)][len(heads)][d]
    holding output row r (compact keyframe order) for each head, in fp64.
    ``rows`` defaults to all M*N rows and ``heads`` to all heads; rows are
    independent, so any subset is exact for the rows it lists.
    """
    qa, _ = as_oracle_array(q)
    n_heads = qa.shape[1]
    rm = rowmap(keyframe_ids, N)
    rows = np.arange(rm.size) if rows is None else np.asarray(rows, np.int64)
    heads = np.arange(n_heads) if heads is None else np.asarray(heads, np.int64)
    tok = np.repeat(rm[rows], heads.size)
    hd = np.tile(heads, rows.size)
    res = attention_pairs(q, k, v, tok, hd, return_probs=return_probs)
    if return_probs:
        out, probs = res
        d = out.shape[1]
        return (out.reshape(rows.size, heads.size, d),
                probs.reshape(rows.size, heads.size, -1))
    d = res.shape[1]
    return res.reshape(rows.size, heads.size, d)


# ---------------------------------------------------------------------------
# projection
# ---------------------------------------------------------------------------

def projection_alpha(t_start: float, t_end: float, tau: float) -> float:
    """alpha of Eq. (3), clamped to [0, 1]; t_start == t_end gives 1."""
    for t in (t_start, t_end, tau):
        if not math.isfinite(t):
            raise ValueError("timesteps must be finite")
    return float(_load().orc_projection_alpha(t_start, t_end, tau))


def project_latents(latents, B, C, T, Hl, Wl, timesteps, keyframe_mask_):
    """Eq. (3) over latents [B][2][C][T][Hl][Wl]; returns [B][C][T][Hl][Wl]
    float64. Keyframe planes take slot 1 (the current state) unchanged."""
    la, dt = as_oracle_array(latents)
    P = Hl * Wl
    if la.size != B * 2 * C * T * P:
        raise ValueError("latents size does not match B*2*C*T*Hl*Wl")
    t_start, t_end, tau = (float(x) for x in timesteps)
    for t in (t_start, t_end, tau):
        if not math.isfinite(t):
            raise ValueError("timesteps must be finite")
    mask = np.ascontiguousarray(np.asarray(keyframe_mask_, dtype=np.uint8))
    if mask.size != T:
        raise ValueError("keyframe mask must have T entries")
    out = np.zeros((B, C, T, Hl, Wl), dtype=np.float64)
    rc = _load().orc_project_latents(
        la.ctypes.data, dt, B, C, T, P,
        mask.ctypes.data_as(ctypes.POINTER(ctypes.c_uint8)),
        t_start, t_end, tau,
        out.ctypes.data_as(ctypes.POINTER(ctypes.c_double)))
    if rc != 0:
        raise RuntimeError("oracle projection failed")
    return out


# ---------------------------------------------------------------------------
# gather / scatter (bit patterns)
# ---------------------------------------------------------------------------

def gather_frames(src_full: np.ndarray, frame_ids, rows_per_frame: int) -> np.ndarray:
    """Rows of the listed frames, frame after frame: dst[r] = src[rowmap[r]].
    src_full is [T*rows_per_frame][...] raw bits (any integer dtype)."""
    return src_full[rowmap(frame_ids, rows_per_frame)].copy()


def scatter_frames(src_compact: np.ndarray, dst_full: np.ndarray, frame_ids,
                   rows_per_frame: int) -> np.ndarray:
    """Inverse of gather_frames into a copy of dst_full; rows of frames not
    listed keep their old contents."""
    out = dst_full.copy()
    out[rowmap(frame_ids, rows_per_frame)] = src_compact
    return out


# ---------------------------------------------------------------------------
# content-aware keyframe selection (Sec. 3.1, Eq. 1; App. A, Alg. 1)
# ---------------------------------------------------------------------------

def frame_cosine(latents, B: int, C: int, T: int, Hl: int, Wl: int) -> np.ndarray:
    """Cosine similarity between the frames of latents [B][C][T][Hl][Wl]
    (each frame flattened over C*Hl*Wl, norms clamped to >= 1e-8); returns
    [B][T][T] float64."""
    la, dt = as_oracle_array(latents)
    P = Hl * Wl
    if la.size != B * C * T * P:
        raise ValueError("latents size does not match B*C*T*Hl*Wl")
    out = np.zeros((B, T, T), dtype=np.float64)
    rc = _load().orc_frame_cosine(la.ctypes.data, dt, B, C, T, P,
                                  out.ctypes.data_as(ctypes.POINTER(ctypes.c_double)))
    if rc != 0:
        raise RuntimeError("oracle frame cosine failed")
    return out


def select_keyframes_adaptive(sim, tau: float, M: int, dtau: float, delta_up: float,
                              delta_down: float, intent_sign: bool = False) -> np.ndarray:
    """Dynamic sequential keyframe selection (Alg. 1) on a [T][T] frame
    similarity matrix.

    The first frame seeds the set and is the first reference. Frames are
    visited in order while fewer than M are selected; frame i joins when its
    similarity to the most recent keyframe is strictly below the current
    threshold (Eq. 1). On each selection the gap to the previous keyframe is
    compared with the expected interval L_avg = T / M (real division): a gap
    of at least L_avg + delta_up lowers the threshold by dtau, a gap of at most
    L_avg - delta_down raises it. ``intent_sign`` swaps the two adjustments
    (the prose describes the large-gap change as encouraging selection, which
    under the rule S < tau is a raise)."""
    sim = np.asarray(sim, dtype=np.float64)
    T = sim.shape[0]
    if sim.shape != (T, T) or T <= 0:
        raise ValueError("sim must be a square [T][T] matrix")
    if M <= 0:
        raise ValueError("M must be positive")
    keys = [0]
    last = 0
    l_avg = T / M
    for i in range(1, T):
        if len(keys) >= M:
            break
        s = sim[i, last]
        if s < tau:
            gap = i - last
            if gap >= l_avg + delta_up:
                tau = tau + dtau if intent_sign else tau - dtau
            elif gap <= l_avg - delta_down:
                tau = tau - dtau if intent_sign else tau + dtau
            keys.append(i)
            last = i
    return np.asarray(keys, dtype=np.int32)


# ---------------------------------------------------------------------------
# rolling cache of post-attention hidden states (App. B.2)
# ---------------------------------------------------------------------------

HIDDEN_EPS = 1e-8


def hidden_alpha(t_before: float, t_after: float, t_skip: float) -> float:
    """alpha = (t_before - t_skip) / (t_before - t_after + eps), eps = 1e-8,
    kept in [0, 1] (right after initialisation t_before = t_after, which makes
    the quotient huge; clamped it selects the cached state, which both slots
    hold then)."""
    for t in (t_before, t_after, t_skip):
        if not math.isfinite(t):
            raise ValueError("timesteps must be finite")
    a = (t_before - t_skip) / (t_before - t_after + HIDDEN_EPS)
    return min(1.0, max(0.0, a))


class RollingCache:
    """The per-layer, per-frame cache of App. B.2 for one layer, written as the
    appendix states it: each frame holds h_before and h_after (arrays of the
    frame's hidden states) and the timesteps t_before >= t_after."""

    def __init__(self):
        self.h_before, self.h_after = {}, {}
        self.t_before, self.t_after = {}, {}

    def init(self, frames, h, t_w: float):
        """End of warm-up: h_before = h_after = the attention output at t_w."""
        for f in frames:
            self.h_before[f] = np.array(h[f], dtype=np.float64)
            self.h_after[f] = np.array(h[f], dtype=np.float64)
            self.t_before[f] = self.t_after[f] = float(t_w)

    def shift_and_store(self, frames, h_new, t_denoise: float):
        """At a denoising (Rhythmic Point) step: h_before <- h_after,
        t_before <- t_after, h_after <- the new attention output, t_after <- t."""
        for f in frames:
            self.h_before[f] = self.h_after[f]
            self.t_before[f] = self.t_after[f]
            self.h_after[f] = np.array(h_new[f], dtype=np.float64)
            self.t_after[f] = float(t_denoise)

    def project(self, f, t_skip: float) -> np.ndarray:
        """h at a skipped step: (1 - alpha) h_before + alpha h_after."""
        a = hidden_alpha(self.t_before[f], self.t_after[f], t_skip)
        return (1.0 - a) * self.h_before[f] + a * self.h_after[f]


def skip_step_kv(k, v, cache: RollingCache, nonkey_frames, t_skip: float, N: int):
    """Keys and values over all frames at a skipped step: keyframes keep their
    computed K and V; every listed non-keyframe contributes its projected hidden
    state as both key and value (App. B.2). k, v: [T*N][heads][d] (any exact
    dtype); returns float64 copies."""
    K = as_oracle_f64(k)
    V = as_oracle_f64(v)
    shape = K.shape
    K = K.reshape(-1, N, *shape[1:])
    V = V.reshape(-1, N, *shape[1:])
    for f in nonkey_frames:
        h = cache.project(f, t_skip).reshape(N, *shape[1:])
        K[f] = h
        V[f] = h
    return K.reshape(shape), V.reshape(shape)


def as_oracle_f64(x) -> np.ndarray:
    """float64 copy of a tensor's exact values (bf16 widened exactly)."""
    a, dt = as_oracle_array(x)
    if dt == BF16:
        return bf16_bits_to_f64(a).reshape(a.shape)
    return np.array(a, dtype=np.float64)


# ---------------------------------------------------------------------------
# progressive asynchronous schedule (Eq. 2, Alg. 2)
# ---------------------------------------------------------------------------

def skip_stride(t: int, T: int, T_w: int, T_mid: int, n_small: int, n_large: int) -> int:
    """Eq. 2: n_small while T_mid < t <= T - T_w, n_large once t <= T_mid.
    Defined for the asynchronous phase only (t <= T - T_w)."""
    if t > T - T_w:
        raise ValueError("warm-up steps have no skip stride")
    return n_small if t > T_mid else n_large


def async_schedule(T: int, T_w: int, T_mid: int, n_small: int, n_large: int):
    """Alg. 2's loop over t = T down to 1, as a list of per-step dicts.

    Warm-up (t > T - T_w): every frame takes one full step. Afterwards the
    keyframes take one step at every t; the non-keyframes, all on one shared
    schedule, take a step of n_skip(t) (Eq. 2; stopping at 0) whenever their
    state time equals t (a Rhythmic Point, where every frame is updated), and
    are otherwise skipped, their state at t being projected between the time
    they last left (t_start) and the time they reached (t_end) with Eq. 3's
    weight. Each non-keyframe's state time is followed step by step; when the
    stride never changes between two updates this is Alg. 2's test
    (T - T_w - t) mod n_skip == 0."""
    steps = []
    state = T          # the non-keyframes' state time
    left = None        # the time of their last update (Eq. 3's t_start)
    for t in range(T, 0, -1):
        if t > T - T_w:
            steps.append(dict(t=t, phase="warmup", n_skip=1, nonkey_to=t - 1,
                              t_start=None, t_end=None, alpha=None))
            state = t - 1
            continue
        n = skip_stride(t, T, T_w, T_mid, n_small, n_large)
        if state == t:
            to = max(t - n, 0)
            steps.append(dict(t=t, phase="rhythmic", n_skip=n, nonkey_to=to,
                              t_start=None, t_end=None, alpha=None))
            left, state = t, to
        else:
            steps.append(dict(t=t, phase="skip", n_skip=n, nonkey_to=None, t_start=left,
                              t_end=state, alpha=(left - t) / (left - state)))
    return steps


def alg2_nonkey_active(t: int, T: int, T_w: int, T_mid: int, n_small: int, n_large: int) -> bool:
    """Alg. 2's membership test for non-keyframes at an asynchronous step, as
    printed: (T - T_w - t) mod n_skip(t) == 0."""
    return (T - T_w - t) % skip_stride(t, T, T_w, T_mid, n_small, n_large) == 0


# ---------------------------------------------------------------------------
# frame-level key/value mask (the frame mask M_Rhyme; Sec. 4's ablations)
# ---------------------------------------------------------------------------

def frame_attention(q, k, v, q_frames, kv_frames, N: int, rows=None, heads=None):
    """Attention under a frame-level mask: the query rows are the tokens of
    q_frames (compact order, as keyframe_attention), the keys and values are
    the tokens of kv_frames only; every other key is masked out. This is the
    frame mask M_Rhyme with one key set for all query frames (the Discussions
    on combining it with a token mask), and with kv_frames = the keyframes it
    is the keyframe-only ("w/o projection") attention of Sec. 4's ablations.
    Written as the definition: the masked keys are removed before the fp64
    softmax. Returns [len(rows)][len(heads)][d] float64."""
    ka, dk = as_oracle_array(k)
    va, dv = as_oracle_array(v)
    kv_tok = rowmap(kv_frames, N)
    kc = np.ascontiguousarray(ka[kv_tok])
    vc = np.ascontiguousarray(va[kv_tok])
    qa, _ = as_oracle_array(q)
    n_heads = qa.shape[1]
    rm = rowmap(q_frames, N)
    rows = np.arange(rm.size) if rows is None else np.asarray(rows, np.int64)
    heads = np.arange(n_heads) if heads is None else np.asarray(heads, np.int64)
    tok = np.repeat(rm[rows], heads.size)
    hd = np.tile(heads, rows.size)
    res = attention_pairs(qa, kc, vc, tok, hd)
    return res.reshape(rows.size, heads.size, res.shape[1])
