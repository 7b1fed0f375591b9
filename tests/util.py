"""Shared helpers of the GPU parity tests (no operator arithmetic here)."""
from __future__ import annotations

import math
import sys

import numpy as np

import testgen


def rel_err(got, ref):
    """Max over elements of |g - r| / max(|r|, 1e-2 * rms(r)) (the bf16 tolerance metric)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    if ref.size == 0:
        return 0.0
    rms = math.sqrt(float(np.mean(ref * ref)))
    den = np.maximum(np.abs(ref), 1e-2 * rms)
    den = np.where(den > 0, den, 1.0)
    return float(np.max(np.abs(got - ref) / den))


def max_abs(got, ref):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    return float(np.max(np.abs(got - ref))) if ref.size else 0.0


def to_device(a: np.ndarray, io_bf16: bool):
    import torch
    if a.dtype == np.uint16:
        assert io_bf16
        return torch.from_numpy(a.view(np.int16)).cuda().view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def to_host(t) -> np.ndarray:
    import torch
    if t.dtype == torch.bfloat16:
        return testgen.bf16_to_f32(t.view(torch.int16).cpu().numpy().view(np.uint16))
    return t.cpu().numpy()


def io_as_f32(a: np.ndarray) -> np.ndarray:
    return testgen.bf16_to_f32(a) if a.dtype == np.uint16 else a


def shape9(w: testgen.Workload):
    return (w.B, w.T, w.H, w.W, w.heads, w.head_dim, w.kt, w.kh, w.kw)


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def reach_frames(w: testgen.Workload, max_abs_dz: float) -> int:
    """Frames a query's corners can reach away from its own frame."""
    return (w.kt - 1) // 2 + int(math.ceil(max_abs_dz)) + 1
