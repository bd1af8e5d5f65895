"""Thin Python binding over librhymeflow.so (argument marshalling only).

Every function here has the name of the C entry point it calls and does no
arithmetic of the method: it checks that tensors are contiguous device tensors
of the right dtype, passes their device pointers and torch's current HIP
stream, and turns a nonzero status into RhymeFlowError. All compute runs in
the HIP kernels; there is no CPU fallback. Importing this module fails loudly
if the library has not been built.
"""
import ctypes
import os

import numpy as np
import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "librhymeflow.so")

RF_OK = 0
RF_ERR_INVALID_ARG = -1
RF_ERR_UNSUPPORTED = -2
RF_ERR_RANGE = -3
RF_ERR_HIP = -4
RF_BF16 = 0
RF_F32 = 1
RF_SEL_NO_FORCE_FIRST = 1
RF_SEL_INTENT_SIGN = 1
RF_MAX_FRAMES = 256

EXPORTED = [
    "rf_status_string", "rf_last_error", "rf_abi_version",
    "rf_select_keyframes", "rf_keyframes_stride", "rf_keyframes_uniform",
    "rf_project_latents", "rf_keyframe_attention", "rf_keyframe_attention_ws", "rf_attention_workspace",
    "rf_attention_plan", "rf_keyframe_attention_noalloc",
    "rf_frame_attention",
    "rf_gather_frames", "rf_scatter_frames",
    "rf_frame_similarity", "rf_frame_similarity_workspace", "rf_select_keyframes_adaptive",
    "rf_cache_store_bytes", "rf_cache_init", "rf_cache_shift_store", "rf_cache_alpha",
    "rf_cache_project_kv", "rf_keyframe_attention_cached", "rf_async_schedule",
    "rf_probe_mfma_bf16", "rf_probe_hbm_read", "rf_probe_lds_read",
]

RF_STEP_WARMUP = 0
RF_STEP_RHYTHMIC = 1
RF_STEP_SKIP = 2
_PHASE_NAMES = {RF_STEP_WARMUP: "warmup", RF_STEP_RHYTHMIC: "rhythmic", RF_STEP_SKIP: "skip"}


class rf_step_plan(ctypes.Structure):
    """The C struct rf_step_plan (one denoising step of the schedule)."""
    _fields_ = [
        ("t", ctypes.c_int32),
        ("phase", ctypes.c_int32),
        ("n_skip", ctypes.c_int32),
        ("nonkey_to", ctypes.c_int32),
        ("t_start", ctypes.c_int32),
        ("t_end", ctypes.c_int32),
        ("alpha", ctypes.c_double),
    ]


class rf_rolling_cache(ctypes.Structure):
    """The C struct rf_rolling_cache (host bookkeeping of one layer's cache)."""
    _fields_ = [
        ("T", ctypes.c_int32),
        ("n_cached", ctypes.c_int32),
        ("rows_per_frame", ctypes.c_int64),
        ("hidden", ctypes.c_int32),
        ("dtype", ctypes.c_int32),
        ("frame_bytes", ctypes.c_int64),
        ("magic", ctypes.c_uint32),
        ("reserved", ctypes.c_int32),
        ("before_slot", ctypes.c_int16 * RF_MAX_FRAMES),
        ("after_slot", ctypes.c_int16 * RF_MAX_FRAMES),
        ("t_before", ctypes.c_double * RF_MAX_FRAMES),
        ("t_after", ctypes.c_double * RF_MAX_FRAMES),
    ]


class rf_attention_split(ctypes.Structure):
    """The C struct rf_attention_split (how a bf16 attention launch is cut)."""
    _fields_ = [
        ("tiles", ctypes.c_int64),
        ("whole_tiles", ctypes.c_int64),
        ("tail_tiles", ctypes.c_int64),
        ("parts", ctypes.c_int32),
        ("key_tiles_per_part", ctypes.c_int32),
        ("workspace_bytes", ctypes.c_int64),
        ("compute_units", ctypes.c_int32),
        ("reserved", ctypes.c_int32),
    ]


class RhymeFlowError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{message} [{status}]")
        self.status = status


if not os.path.exists(LIB_PATH):
    raise ImportError(
        f"{LIB_PATH} is missing: build the HIP library first "
        "(python -c 'import __graft_entry__ as g; g.build()')")

lib = ctypes.CDLL(LIB_PATH)

_i32 = ctypes.c_int32
_i64 = ctypes.c_int64
_vp = ctypes.c_void_p
_i32p = ctypes.POINTER(ctypes.c_int32)
_u8p = ctypes.POINTER(ctypes.c_uint8)
_dp = ctypes.POINTER(ctypes.c_double)

lib.rf_status_string.argtypes = [ctypes.c_int]
lib.rf_status_string.restype = ctypes.c_char_p
lib.rf_last_error.argtypes = []
lib.rf_last_error.restype = ctypes.c_char_p
lib.rf_abi_version.argtypes = []
lib.rf_abi_version.restype = ctypes.c_int
lib.rf_select_keyframes.argtypes = [_i32p, _i32, _i32, ctypes.c_uint32, _i32p, _i32p, _u8p]
lib.rf_select_keyframes.restype = ctypes.c_int
lib.rf_keyframes_stride.argtypes = [_i32, _i32, _i32p, _i32p]
lib.rf_keyframes_stride.restype = ctypes.c_int
lib.rf_keyframes_uniform.argtypes = [_i32, _i32, _i32p, _i32p]
lib.rf_keyframes_uniform.restype = ctypes.c_int
lib.rf_project_latents.argtypes = [_vp, _vp, _dp, _u8p, _i32, _i32, _i32, _i32, _i32, _i32, _vp]
lib.rf_project_latents.restype = ctypes.c_int
lib.rf_keyframe_attention.argtypes = [_vp, _vp, _vp, _vp, _i32p, _i32, _i32, _i32, _i32,
                                      _i32, _i32, _i32, _vp]
lib.rf_keyframe_attention.restype = ctypes.c_int
lib.rf_frame_attention.argtypes = [_vp, _vp, _vp, _vp, _i32p, _i32, _i32p, _i32, _i32, _i32, _i32,
                                   _i32, _i32, _i32, _vp, _i64, _vp]
lib.rf_keyframe_attention_ws.argtypes = [_vp, _vp, _vp, _vp, _i32p, _i32, _i32, _i32, _i32,
                                         _i32, _i32, _i32, _vp, _i64, _vp]
lib.rf_keyframe_attention_ws.restype = ctypes.c_int
lib.rf_keyframe_attention_noalloc.argtypes = [_vp, _vp, _vp, _vp, _i32p, _i32, _i32, _i32, _i32,
                                              _i32, _i32, _i32, _vp]
lib.rf_keyframe_attention_noalloc.restype = ctypes.c_int
RF_NOALLOC_SCRATCH_BYTES = 160 << 20
lib.rf_attention_workspace.argtypes = [_i32, _i32, _i32, _i32, _i32, _i32, _i32, _i32, _i32, ctypes.POINTER(_i64)]
lib.rf_attention_workspace.restype = ctypes.c_int
lib.rf_attention_plan.argtypes = [_i32, _i32, _i32, _i32, _i32, _i32, _i32, _i32, _i32,
                                  ctypes.POINTER(rf_attention_split)]
lib.rf_attention_plan.restype = ctypes.c_int
lib.rf_frame_attention.restype = ctypes.c_int
lib.rf_gather_frames.argtypes = [_vp, _vp, _i32p, _i32, _i32, _i64, _i64, _vp]
lib.rf_gather_frames.restype = ctypes.c_int
lib.rf_scatter_frames.argtypes = [_vp, _vp, _i32p, _i32, _i32, _i64, _i64, _vp]
lib.rf_scatter_frames.restype = ctypes.c_int
lib.rf_frame_similarity.argtypes = [_vp, _vp, _vp, _i64, _i32, _i32, _i32, _i32, _i32, _i32, _vp]
lib.rf_frame_similarity.restype = ctypes.c_int
lib.rf_frame_similarity_workspace.argtypes = [_i32, _i32, _i32, _i32, _i32, ctypes.POINTER(_i64)]
lib.rf_frame_similarity_workspace.restype = ctypes.c_int
lib.rf_select_keyframes_adaptive.argtypes = [_dp, _i32, ctypes.c_double, _i32, ctypes.c_double,
                                             ctypes.c_double, ctypes.c_double, ctypes.c_uint32,
                                             _i32p, _i32p, _u8p]
lib.rf_select_keyframes_adaptive.restype = ctypes.c_int
_cachep = ctypes.POINTER(rf_rolling_cache)
lib.rf_cache_store_bytes.argtypes = [_i32, _i64, _i32, _i32, ctypes.POINTER(_i64)]
lib.rf_cache_store_bytes.restype = ctypes.c_int
lib.rf_cache_init.argtypes = [_cachep, _vp, _vp, _i32p, _i32, _i32, _i64, _i32, _i32,
                              ctypes.c_double, _vp]
lib.rf_cache_init.restype = ctypes.c_int
lib.rf_cache_shift_store.argtypes = [_cachep, _vp, _vp, _i32p, _i32, ctypes.c_double, _vp]
lib.rf_cache_shift_store.restype = ctypes.c_int
lib.rf_cache_alpha.argtypes = [_cachep, _i32, ctypes.c_double, _dp]
lib.rf_cache_alpha.restype = ctypes.c_int
lib.rf_cache_project_kv.argtypes = [_cachep, _vp, _vp, _vp, _i32p, _i32, ctypes.c_double, _vp]
lib.rf_cache_project_kv.restype = ctypes.c_int
lib.rf_keyframe_attention_cached.argtypes = [_vp, _vp, _vp, _vp, _i32p, _i32, _i32, _i32, _i32, _i32, _i32, _i32,
                                             _cachep, _vp, ctypes.c_double, _vp, _i64, _vp]
lib.rf_keyframe_attention_cached.restype = ctypes.c_int
lib.rf_async_schedule.argtypes = [_i32, _i32, _i32, _i32, _i32, ctypes.POINTER(rf_step_plan), _i32p, _i32p]
lib.rf_async_schedule.restype = ctypes.c_int
lib.rf_probe_mfma_bf16.argtypes = [_vp, _i32, _i32, _vp, _vp]
lib.rf_probe_mfma_bf16.restype = ctypes.c_int
lib.rf_probe_hbm_read.argtypes = [_vp, _i64, _i32, _vp, _vp]
lib.rf_probe_hbm_read.restype = ctypes.c_int
lib.rf_probe_lds_read.argtypes = [_i32, _i32, _i32, _vp, _vp, _vp]
lib.rf_probe_lds_read.restype = ctypes.c_int


def _check(status: int):
    if status != RF_OK:
        msg = lib.rf_last_error().decode(errors="replace")
        raise RhymeFlowError(status, f"{lib.rf_status_string(status).decode()}: {msg}")


def _ids(ids):
    a = np.ascontiguousarray(np.asarray(list(ids), dtype=np.int32))
    return a, a.ctypes.data_as(_i32p)


def _stream(stream):
    if stream is None:
        return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, torch.cuda.Stream):
        return ctypes.c_void_p(stream.cuda_stream)
    return ctypes.c_void_p(int(stream))


def _torch_stream(stream):
    """The torch stream object of a launch stream argument (None: torch's
    current stream, which needs no handling)."""
    if stream is None or isinstance(stream, torch.cuda.Stream):
        return stream
    if int(stream) == 0:
        return torch.cuda.default_stream()
    return torch.cuda.ExternalStream(int(stream))


def _empty(shape, dtype, device, stream):
    """A tensor the call allocates for itself (an output or a workspace),
    allocated while the launch stream is torch's current stream: the caching
    allocator then ties the block to that stream, so once the tensor is dropped
    the block is handed only to later work on the same stream, never to other
    streams while the launch may still be using it."""
    ts = _torch_stream(stream) if torch.device(device).type == "cuda" else None
    if ts is None:
        return torch.empty(shape, dtype=dtype, device=device)
    with torch.cuda.stream(ts):
        return torch.empty(shape, dtype=dtype, device=device)


def _dev(t: torch.Tensor, name: str):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _dtype_code(dt):
    if dt == torch.bfloat16:
        return RF_BF16
    if dt == torch.float32:
        return RF_F32
    raise TypeError(f"unsupported dtype {dt}")


def abi_version() -> int:
    return int(lib.rf_abi_version())


# --- keyframe sets (host) ------------------------------------------------------

def rf_select_keyframes(frame_ids, T: int, force_first: bool = True):
    """Returns (keyframe ids int32 [M], mask uint8 [T])."""
    ids, ids_p = _ids(frame_ids)
    out = np.zeros(max(T, 1), dtype=np.int32)
    mask = np.zeros(max(T, 1), dtype=np.uint8)
    n = ctypes.c_int32(0)
    flags = 0 if force_first else RF_SEL_NO_FORCE_FIRST
    _check(lib.rf_select_keyframes(ids_p if ids.size else None, ids.size, T, flags,
                                   out.ctypes.data_as(_i32p), ctypes.byref(n),
                                   mask.ctypes.data_as(_u8p)))
    return out[:n.value].copy(), mask[:T].copy()


def rf_keyframes_stride(T: int, k: int) -> np.ndarray:
    out = np.zeros(max(T, 1), dtype=np.int32)
    n = ctypes.c_int32(0)
    _check(lib.rf_keyframes_stride(T, k, out.ctypes.data_as(_i32p), ctypes.byref(n)))
    return out[:n.value].copy()


def rf_select_keyframes_adaptive(sim, tau: float, M: int, dtau: float, delta_up: float,
                                 delta_down: float, intent_sign: bool = False):
    """Alg. 1's scan on a host [T][T] similarity matrix (numpy or a tensor,
    copied to host). Returns (keyframe ids int32, mask uint8 [T])."""
    if isinstance(sim, torch.Tensor):
        sim = sim.detach().cpu().numpy()
    a = np.ascontiguousarray(np.asarray(sim, dtype=np.float64))
    if a.ndim != 2 or a.shape[0] != a.shape[1]:
        raise ValueError("sim must be a square [T][T] matrix")
    T = a.shape[0]
    out = np.zeros(max(T, 1), dtype=np.int32)
    mask = np.zeros(max(T, 1), dtype=np.uint8)
    n = ctypes.c_int32(0)
    flags = RF_SEL_INTENT_SIGN if intent_sign else 0
    _check(lib.rf_select_keyframes_adaptive(a.ctypes.data_as(_dp), T, float(tau), M, float(dtau),
                                            float(delta_up), float(delta_down), flags,
                                            out.ctypes.data_as(_i32p), ctypes.byref(n),
                                            mask.ctypes.data_as(_u8p)))
    return out[:n.value].copy(), mask[:T].copy()


def rf_frame_similarity_workspace(B: int, C: int, T: int, H: int, W: int) -> int:
    """Bytes of device workspace rf_frame_similarity needs."""
    n = _i64(0)
    _check(lib.rf_frame_similarity_workspace(B, C, T, H, W, ctypes.byref(n)))
    return int(n.value)


def rf_keyframes_uniform(T: int, M: int) -> np.ndarray:
    out = np.zeros(max(M, 1), dtype=np.int32)
    n = ctypes.c_int32(0)
    _check(lib.rf_keyframes_uniform(T, M, out.ctypes.data_as(_i32p), ctypes.byref(n)))
    return out[:n.value].copy()


# --- device calls ----------------------------------------------------------------

def rf_project_latents(latents: torch.Tensor, timesteps, keyframe_mask, out=None, stream=None):
    """latents [B][2][C][T][Hl][Wl] -> out [B][C][T][Hl][Wl] (same dtype)."""
    if latents.dim() != 6 or latents.shape[1] != 2:
        raise ValueError("latents must be [B][2][C][T][Hl][Wl]")
    B, _, C, T, Hl, Wl = latents.shape
    if out is None:
        out = _empty((B, C, T, Hl, Wl), latents.dtype, latents.device, stream)
    if out.dtype != latents.dtype or out.numel() != B * C * T * Hl * Wl:
        raise ValueError("out must match latents' dtype and [B][C][T][Hl][Wl] size")
    ts = (ctypes.c_double * 3)(*[float(x) for x in timesteps])
    mask = np.ascontiguousarray(np.asarray(keyframe_mask, dtype=np.uint8))
    if mask.size != T:
        raise ValueError("keyframe_mask must have T entries")
    _check(lib.rf_project_latents(_dev(latents, "latents"), _dev(out, "out"), ts,
                                  mask.ctypes.data_as(_u8p), B, C, T, Hl, Wl,
                                  _dtype_code(latents.dtype), _stream(stream)))
    return out


def rf_keyframe_attention(q, k, v, keyframe_ids, T: int, H: int, W: int, out=None, stream=None):
    """q, k, v [T*H*W][heads][head_dim] -> out [M*H*W][heads][head_dim]."""
    if q.dim() != 3 or k.shape != q.shape or v.shape != q.shape:
        raise ValueError("q, k, v must share one [S][heads][head_dim] shape")
    if not (q.dtype == k.dtype == v.dtype):
        raise TypeError("q, k, v must share a dtype")
    S, heads, d = q.shape
    if S != T * H * W:
        raise ValueError(f"S = {S} differs from T*H*W = {T * H * W}")
    ids, ids_p = _ids(keyframe_ids)
    M = ids.size
    if out is None:
        out = _empty((M * H * W, heads, d), q.dtype, q.device, stream)
    if out.dtype != q.dtype or out.numel() != M * H * W * heads * d:
        raise ValueError("out must be [M*H*W][heads][head_dim] of q's dtype")
    _check(lib.rf_keyframe_attention(_dev(q, "q"), _dev(k, "k"), _dev(v, "v"), _dev(out, "out"),
                                     ids_p, M, T, H, W, heads, d, _dtype_code(q.dtype),
                                     _stream(stream)))
    return out


def rf_attention_workspace(M: int, Mkv: int, T: int, H: int, W: int, heads: int, head_dim: int, dtype,
                           compute_units: int = 0) -> int:
    """Bytes of split-tail workspace rf_keyframe_attention_ws (Mkv = T) or
    rf_frame_attention uses (0: nothing is split) on a device of compute_units
    compute units (0: the current device, which the launch uses)."""
    n = _i64(0)
    code = dtype if isinstance(dtype, int) else _dtype_code(dtype)
    _check(lib.rf_attention_workspace(M, Mkv, T, H, W, heads, head_dim, code, compute_units, ctypes.byref(n)))
    return int(n.value)


def rf_attention_plan(M: int, Mkv: int, T: int, H: int, W: int, heads: int, head_dim: int, dtype,
                      compute_units: int = 0) -> dict:
    """The split plan of a bf16 attention launch as a dict of the fields of
    rf_attention_split (compute_units 0: the current device)."""
    p = rf_attention_split()
    code = dtype if isinstance(dtype, int) else _dtype_code(dtype)
    _check(lib.rf_attention_plan(M, Mkv, T, H, W, heads, head_dim, code, compute_units, ctypes.byref(p)))
    return {name: int(getattr(p, name)) for name, _ in rf_attention_split._fields_ if name != "reserved"}


def _workspace(workspace, nbytes, device, stream):
    if workspace is None:
        workspace = _empty(max(nbytes, 16), torch.uint8, device, stream)
    return workspace, workspace.numel() * workspace.element_size()


def rf_keyframe_attention_ws(q, k, v, keyframe_ids, T: int, H: int, W: int, out=None, workspace=None,
                             stream=None):
    """rf_keyframe_attention with the split-key tail; the workspace (a device
    tensor) is allocated here if not given."""
    if q.dim() != 3 or k.shape != q.shape or v.shape != q.shape:
        raise ValueError("q, k, v must share one [S][heads][head_dim] shape")
    if not (q.dtype == k.dtype == v.dtype):
        raise TypeError("q, k, v must share a dtype")
    S, heads, d = q.shape
    if S != T * H * W:
        raise ValueError(f"S = {S} differs from T*H*W = {T * H * W}")
    ids, ids_p = _ids(keyframe_ids)
    M = ids.size
    if out is None:
        out = _empty((M * H * W, heads, d), q.dtype, q.device, stream)
    if out.dtype != q.dtype or out.numel() != M * H * W * heads * d:
        raise ValueError("out must be [M*H*W][heads][head_dim] of q's dtype")
    ptrs = [_dev(q, "q"), _dev(k, "k"), _dev(v, "v"), _dev(out, "out")]
    need = rf_attention_workspace(M, T, T, H, W, heads, d, q.dtype) if M > 0 and workspace is None else 0
    workspace, wbytes = _workspace(workspace, need, q.device, stream)
    _check(lib.rf_keyframe_attention_ws(*ptrs, ids_p, M, T, H, W, heads, d, _dtype_code(q.dtype),
                                        _dev(workspace, "workspace"), wbytes, _stream(stream)))
    return out


def rf_keyframe_attention_noalloc(q, k, v, keyframe_ids, T: int, H: int, W: int, out=None, stream=None):
    """rf_keyframe_attention with the split-key tail in the library's static
    device scratch (no workspace; the library allocates nothing). Calls that
    overlap in time on one GPU race on that scratch."""
    if q.dim() != 3 or k.shape != q.shape or v.shape != q.shape:
        raise ValueError("q, k, v must share one [S][heads][head_dim] shape")
    if not (q.dtype == k.dtype == v.dtype):
        raise TypeError("q, k, v must share a dtype")
    S, heads, d = q.shape
    if S != T * H * W:
        raise ValueError(f"S = {S} differs from T*H*W = {T * H * W}")
    ids, ids_p = _ids(keyframe_ids)
    M = ids.size
    if out is None:
        out = _empty((M * H * W, heads, d), q.dtype, q.device, stream)
    if out.dtype != q.dtype or out.numel() != M * H * W * heads * d:
        raise ValueError("out must be [M*H*W][heads][head_dim] of q's dtype")
    _check(lib.rf_keyframe_attention_noalloc(_dev(q, "q"), _dev(k, "k"), _dev(v, "v"), _dev(out, "out"),
                                             ids_p, M, T, H, W, heads, d, _dtype_code(q.dtype), _stream(stream)))
    return out


def rf_frame_attention(q, k, v, q_frames, kv_frames, T: int, H: int, W: int, out=None, workspace=None,
                       stream=None):
    """Attention of the tokens of q_frames over the keys/values of kv_frames
    only; q, k, v [T*H*W][heads][head_dim] -> out [Mq*H*W][heads][head_dim].
    workspace: a device tensor for the split-key tail, or None (no split)."""
    if q.dim() != 3 or k.shape != q.shape or v.shape != q.shape:
        raise ValueError("q, k, v must share one [S][heads][head_dim] shape")
    if not (q.dtype == k.dtype == v.dtype):
        raise TypeError("q, k, v must share a dtype")
    S, heads, d = q.shape
    if S != T * H * W:
        raise ValueError(f"S = {S} differs from T*H*W = {T * H * W}")
    ids, ids_p = _ids(q_frames)
    kv, kv_p = _ids(kv_frames)
    M = ids.size
    if out is None:
        out = _empty((M * H * W, heads, d), q.dtype, q.device, stream)
    if out.dtype != q.dtype or out.numel() != M * H * W * heads * d:
        raise ValueError("out must be [Mq*H*W][heads][head_dim] of q's dtype")
    ws_p, wbytes = (None, 0) if workspace is None else (_dev(workspace, "workspace"),
                                                        workspace.numel() * workspace.element_size())
    _check(lib.rf_frame_attention(_dev(q, "q"), _dev(k, "k"), _dev(v, "v"), _dev(out, "out"),
                                  ids_p, M, kv_p, kv.size, T, H, W, heads, d, _dtype_code(q.dtype),
                                  ws_p, wbytes, _stream(stream)))
    return out


def rf_frame_similarity(latents: torch.Tensor, out=None, workspace=None, stream=None):
    """latents [B][C][T][H][W] -> cosine similarity [B][T][T] float64 (device).
    The workspace (a device uint8 tensor) is allocated here if not given."""
    if latents.dim() != 5:
        raise ValueError("latents must be [B][C][T][H][W]")
    B, C, T, H, W = latents.shape
    if out is None:
        out = _empty((B, T, T), torch.float64, latents.device, stream)
    if out.dtype != torch.float64 or out.numel() != B * T * T:
        raise ValueError("out must be float64 [B][T][T]")
    need = rf_frame_similarity_workspace(B, C, T, H, W)
    if workspace is None:
        workspace = _empty(max(need, 16), torch.uint8, latents.device, stream)
    _check(lib.rf_frame_similarity(_dev(latents, "latents"), _dev(out, "out"),
                                   _dev(workspace, "workspace"), workspace.numel() * workspace.element_size(),
                                   B, C, T, H, W, _dtype_code(latents.dtype), _stream(stream)))
    return out


def _row_geometry(t: torch.Tensor, rows_per_frame: int):
    if t.dim() < 1 or t.shape[0] % rows_per_frame:
        raise ValueError("leading dimension must be a multiple of rows_per_frame")
    return t.numel() // t.shape[0] * t.element_size()


def rf_gather_frames(src_full: torch.Tensor, frame_ids, T: int, rows_per_frame: int,
                     out=None, stream=None):
    """src_full [T*N][...] -> out [M*N][...] (rows of the listed frames)."""
    row_bytes = _row_geometry(src_full, rows_per_frame)
    if src_full.shape[0] != T * rows_per_frame:
        raise ValueError("src_full must hold T * rows_per_frame rows")
    ids, ids_p = _ids(frame_ids)
    if out is None:
        out = _empty((ids.size * rows_per_frame,) + tuple(src_full.shape[1:]), src_full.dtype,
                     src_full.device, stream)
    if out.numel() * out.element_size() != ids.size * rows_per_frame * row_bytes:
        raise ValueError("out must hold M * rows_per_frame rows")
    _check(lib.rf_gather_frames(_dev(src_full, "src_full"), _dev(out, "out"), ids_p, ids.size, T,
                                rows_per_frame, row_bytes, _stream(stream)))
    return out


def rf_scatter_frames(src_compact: torch.Tensor, dst_full: torch.Tensor, frame_ids, T: int,
                      rows_per_frame: int, stream=None):
    """Writes src_compact's rows into the listed frames of dst_full (in place)."""
    row_bytes = _row_geometry(dst_full, rows_per_frame)
    if dst_full.shape[0] != T * rows_per_frame:
        raise ValueError("dst_full must hold T * rows_per_frame rows")
    ids, ids_p = _ids(frame_ids)
    if src_compact.numel() * src_compact.element_size() != ids.size * rows_per_frame * row_bytes:
        raise ValueError("src_compact must hold M * rows_per_frame rows of dst_full's row size")
    _check(lib.rf_scatter_frames(_dev(src_compact, "src_compact"), _dev(dst_full, "dst_full"),
                                 ids_p, ids.size, T, rows_per_frame, row_bytes, _stream(stream)))
    return dst_full


# --- rolling cache (App. B.2) ------------------------------------------------------

def rf_cache_store_bytes(n_cached: int, rows_per_frame: int, hidden: int, dtype) -> int:
    """Bytes of device store a cache of n_cached frames needs."""
    n = _i64(0)
    code = dtype if isinstance(dtype, int) else _dtype_code(dtype)
    _check(lib.rf_cache_store_bytes(n_cached, rows_per_frame, hidden, code, ctypes.byref(n)))
    return int(n.value)


def _frames_arg(frames):
    if frames is None:
        return None, None, 0
    ids, ids_p = _ids(frames)
    return ids, ids_p, ids.size


def _opt_dev(t, name):
    return None if t is None else _dev(t, name)


def _check_h_full(h_full, code, nbytes):
    """h_full holds all T frames' rows in the cache's dtype: exactly nbytes."""
    if not isinstance(h_full, torch.Tensor):
        raise TypeError("h_full must be a torch.Tensor")
    if _dtype_code(h_full.dtype) != code:
        raise TypeError(f"h_full has dtype {h_full.dtype}, the cache holds {'f32' if code == RF_F32 else 'bf16'}")
    if h_full.numel() * h_full.element_size() != nbytes:
        raise ValueError(f"h_full holds {h_full.numel() * h_full.element_size()} bytes, "
                         f"T * rows_per_frame rows of the cache's row size are {nbytes}")


def _check_store(store, need):
    if not isinstance(store, torch.Tensor):
        raise TypeError("store must be a torch.Tensor")
    if store.numel() * store.element_size() < need:
        raise ValueError(f"store is smaller than the cache needs ({store.numel() * store.element_size()} "
                         f"of {need} bytes)")


def rf_cache_init(frames, T: int, rows_per_frame: int, hidden: int, dtype, t_w: float,
                  store=None, h_full=None, cache=None, stream=None) -> rf_rolling_cache:
    """Sets up (or overwrites) `cache` for the listed frames at t_w and, when
    h_full ([T*N][...] device tensor) is given, copies their rows into the store."""
    cache = rf_rolling_cache() if cache is None else cache
    ids, ids_p = _ids(frames)
    code = dtype if isinstance(dtype, int) else _dtype_code(dtype)
    if h_full is not None:
        # the C ABI cannot see the buffers' sizes: check them here, before any launch
        if store is None:
            raise ValueError("h_full needs a store to copy into")
        esize = 4 if code == RF_F32 else 2
        _check_h_full(h_full, code, T * rows_per_frame * hidden * esize)
        _check_store(store, rf_cache_store_bytes(ids.size, rows_per_frame, hidden, code))
    _check(lib.rf_cache_init(ctypes.byref(cache), _opt_dev(store, "store"), _opt_dev(h_full, "h_full"),
                             ids_p if ids.size else None, ids.size, T, rows_per_frame, hidden, code,
                             float(t_w), _stream(stream) if h_full is not None else None))
    return cache


def rf_cache_shift_store(cache: rf_rolling_cache, t_denoise: float, store=None, h_full=None,
                         frames=None, stream=None) -> rf_rolling_cache:
    """Shift-and-store at t_denoise for `frames` (None: every cached frame)."""
    _, ids_p, n = _frames_arg(frames)
    if h_full is not None:
        if store is None:
            raise ValueError("h_full needs a store to copy into")
        _check_h_full(h_full, cache.dtype, cache.T * cache.frame_bytes)
        _check_store(store, 2 * cache.n_cached * cache.frame_bytes)
    _check(lib.rf_cache_shift_store(ctypes.byref(cache), _opt_dev(store, "store"),
                                    _opt_dev(h_full, "h_full"), ids_p, n, float(t_denoise),
                                    _stream(stream) if h_full is not None else None))
    return cache


def rf_cache_alpha(cache: rf_rolling_cache, frame: int, t_skip: float) -> float:
    a = ctypes.c_double(0.0)
    _check(lib.rf_cache_alpha(ctypes.byref(cache), frame, float(t_skip), ctypes.byref(a)))
    return a.value


def rf_cache_project_kv(cache: rf_rolling_cache, store: torch.Tensor, k: torch.Tensor, v: torch.Tensor,
                        t_skip: float, frames=None, stream=None):
    """Writes the projected hidden state of each listed cached frame (None:
    all) into its rows of k and v, in place ([T*N][heads][head_dim] tensors)."""
    for t, name in ((k, "k"), (v, "v")):
        if t.numel() * t.element_size() != cache.T * cache.frame_bytes:
            raise ValueError(f"{name} must hold T * rows_per_frame rows of the cache's row size")
        if _dtype_code(t.dtype) != cache.dtype:
            raise TypeError(f"{name} must have the cache's dtype")
    if store.numel() * store.element_size() < 2 * cache.n_cached * cache.frame_bytes:
        raise ValueError("store is smaller than the cache needs")
    _, ids_p, n = _frames_arg(frames)
    _check(lib.rf_cache_project_kv(ctypes.byref(cache), _dev(store, "store"), _dev(k, "k"),
                                   _dev(v, "v"), ids_p, n, float(t_skip), _stream(stream)))
    return k, v


def rf_keyframe_attention_cached(q, k, v, keyframe_ids, T: int, H: int, W: int, cache: rf_rolling_cache,
                                 store: torch.Tensor, t_skip: float, out=None, workspace=None, stream=None):
    """Keyframe-query attention at a skipped step whose cached frames take their
    projected hidden states (App. B.2) as keys and values, formed inside the
    kernel; k and v rows of cached frames are not read. The workspace (a device
    tensor) is allocated here if not given."""
    if q.dim() != 3 or k.shape != q.shape or v.shape != q.shape:
        raise ValueError("q, k, v must share one [S][heads][head_dim] shape")
    if not (q.dtype == k.dtype == v.dtype):
        raise TypeError("q, k, v must share a dtype")
    S, heads, d = q.shape
    if S != T * H * W:
        raise ValueError(f"S = {S} differs from T*H*W = {T * H * W}")
    _check_store(store, 2 * cache.n_cached * cache.frame_bytes)
    ids, ids_p = _ids(keyframe_ids)
    M = ids.size
    if out is None:
        out = _empty((M * H * W, heads, d), q.dtype, q.device, stream)
    if out.dtype != q.dtype or out.numel() != M * H * W * heads * d:
        raise ValueError("out must be [M*H*W][heads][head_dim] of q's dtype")
    ptrs = [_dev(q, "q"), _dev(k, "k"), _dev(v, "v"), _dev(out, "out")]
    sp = _dev(store, "store")
    need = rf_attention_workspace(M, T, T, H, W, heads, d, q.dtype) if M > 0 and workspace is None else 0
    workspace, wbytes = _workspace(workspace, need, q.device, stream)
    _check(lib.rf_keyframe_attention_cached(*ptrs, ids_p, M, T, H, W, heads, d, _dtype_code(q.dtype),
                                            ctypes.byref(cache), sp, float(t_skip), _dev(workspace, "workspace"),
                                            wbytes, _stream(stream)))
    return out


# --- asynchronous schedule (Eq. 2, Alg. 2) ----------------------------------------

def rf_async_schedule(T: int, T_w: int, T_mid: int, n_small: int, n_large: int):
    """The step plan for t = T..1 as a list of dicts (phase as "warmup",
    "rhythmic" or "skip"; fields that do not apply to a step are None)."""
    plan = (rf_step_plan * max(T, 1))()
    nr, ns = _i32(0), _i32(0)
    _check(lib.rf_async_schedule(T, T_w, T_mid, n_small, n_large, plan, ctypes.byref(nr), ctypes.byref(ns)))
    out = []
    for p in plan[:T]:
        skip = p.phase == RF_STEP_SKIP
        out.append(dict(t=p.t, phase=_PHASE_NAMES[p.phase], n_skip=p.n_skip,
                        nonkey_to=None if skip else p.nonkey_to,
                        t_start=p.t_start if skip else None, t_end=p.t_end if skip else None,
                        alpha=p.alpha if skip else None))
    return out


# --- device probes (measurement support) ------------------------------------------

PROBE_THREADS = 256


def rf_probe_mfma_bf16(operands: torch.Tensor, workgroups: int, rounds: int, sink=None, stream=None):
    """Enqueues the dense bf16 matrix-core probe (workgroups * rounds * 2^22
    FLOP) on operands, bf16 [12][64][8]; returns the sink, float
    [workgroups * 256] on the operands' device."""
    if operands.dtype != torch.bfloat16 or operands.numel() != 12 * 64 * 8:
        raise ValueError("operands must be bf16 with 12 * 64 * 8 elements")
    if sink is None:
        sink = _empty(workgroups * PROBE_THREADS, torch.float32, operands.device, stream)
    if sink.dtype != torch.float32 or sink.numel() < workgroups * PROBE_THREADS:
        raise ValueError("sink must be float32 with workgroups * 256 elements")
    _check(lib.rf_probe_mfma_bf16(_dev(operands, "operands"), workgroups, rounds, _dev(sink, "sink"),
                                  _stream(stream)))
    return sink


def rf_probe_hbm_read(src: torch.Tensor, workgroups: int, sink=None, stream=None):
    """Enqueues the HBM read probe over src's bytes (workgroup w reads the
    w-th of `workgroups` contiguous runs); returns the sink, int32
    [workgroups] whose XOR is the XOR of src's 32-bit words."""
    if sink is None:
        sink = _empty(workgroups, torch.int32, src.device, stream)
    if sink.element_size() != 4 or sink.numel() < workgroups:
        raise ValueError("sink must have 4-byte elements, workgroups of them")
    _check(lib.rf_probe_hbm_read(_dev(src, "src"), src.numel() * src.element_size(), workgroups,
                                 _dev(sink, "sink"), _stream(stream)))
    return sink


def rf_probe_lds_read(workgroups: int, rounds: int, width: int = 16, sink=None, ticks=None, device="cuda",
                      stream=None):
    """Enqueues the LDS read probe (workgroups * 4 * rounds * 64 KB read from
    LDS, 16-byte reads for width 16, transposing 8-byte reads for width 8);
    returns (sink, ticks): int32 [workgroups * 256] sums and int64
    [workgroups] shader-clock ticks of each workgroup's reads."""
    dev = torch.device(device)
    if sink is None:
        sink = _empty(workgroups * PROBE_THREADS, torch.int32, dev, stream)
    if ticks is None:
        ticks = _empty(workgroups, torch.int64, dev, stream)
    if sink.element_size() != 4 or sink.numel() < workgroups * PROBE_THREADS:
        raise ValueError("sink must have 4-byte elements, workgroups * 256 of them")
    if ticks.element_size() != 8 or ticks.numel() < workgroups:
        raise ValueError("ticks must have 8-byte elements, workgroups of them")
    _check(lib.rf_probe_lds_read(workgroups, rounds, width, _dev(sink, "sink"), _dev(ticks, "ticks"),
                                 _stream(stream)))
    return sink, ticks
