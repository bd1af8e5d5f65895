"""Tolerance gates shared by the parity tests.

Absolute bounds for bf16 outputs: max-abs <= 2e-2 and mean-abs <= 2e-3; the
fp32 path: max-abs <= 1e-4. Several workloads have outputs whose magnitude is
near those bounds (a near-uniform softmax averages many values), so an output
of zeros could pass them; every gate therefore also bounds the relative
Frobenius error: 1e-2 for bf16 (bf16 output rounding alone is ~2e-3 relative)
and 1e-5 for fp32.
"""
import numpy as np

BF16_MAX_ABS = 2e-2
BF16_MEAN_ABS = 2e-3
BF16_REL_FRO = 1e-2
F32_MAX_ABS = 1e-4
F32_REL_FRO = 1e-5


def error_stats(out, ref):
    out = np.asarray(out, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    if out.shape != ref.shape:
        raise ValueError(f"shape mismatch {out.shape} vs {ref.shape}")
    diff = np.abs(out - ref)
    nref = np.linalg.norm(ref.ravel())
    rel = np.linalg.norm((out - ref).ravel()) / nref if nref > 0 else np.linalg.norm(out.ravel())
    return {
        "max_abs": float(diff.max()) if diff.size else 0.0,
        "mean_abs": float(diff.mean()) if diff.size else 0.0,
        "rel_fro": float(rel),
        "finite": bool(np.isfinite(out).all()),
    }


def passes(out, ref, kind: str):
    st = error_stats(out, ref)
    if kind == "bf16":
        ok = (st["finite"] and st["max_abs"] <= BF16_MAX_ABS
              and st["mean_abs"] <= BF16_MEAN_ABS and st["rel_fro"] <= BF16_REL_FRO)
    elif kind == "f32":
        ok = st["finite"] and st["max_abs"] <= F32_MAX_ABS and st["rel_fro"] <= F32_REL_FRO
    else:
        raise ValueError(kind)
    return ok, st


def assert_parity(out, ref, kind: str, what: str = ""):
    ok, st = passes(out, ref, kind)
    assert ok, f"{what} parity failed ({kind}): {st}"
    return st


def torch_bf16_to_f64(t):
    """Exact widening of a bf16 torch tensor to a float64 numpy array."""
    import torch
    bits = t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
