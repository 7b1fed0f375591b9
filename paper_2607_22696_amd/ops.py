"""Tensor-level calls of the C ABI: allocate outputs with torch, then call the library.

q, k, v (and dout) are [B, T, H, W, heads, head_dim] CUDA tensors in float32 or bfloat16;
offsets are float32 [B, T, H, W, heads, P, 3] with (x, y, z) = (w, h, t) in token units.
"""
from __future__ import annotations

import torch

from ._binding import (dsa3d_backward, dsa3d_backward_timed, dsa3d_backward_workspace_size,
                       dsa3d_forward, make_desc)


def _desc(q, kernel, scale):
    if q.dim() != 6:
        raise ValueError("q must be [B, T, H, W, heads, head_dim]")
    B, T, H, W, heads, D = q.shape
    kt, kh, kw = kernel
    if q.dtype == torch.bfloat16:
        dtype = "bf16"
    elif q.dtype == torch.float32:
        dtype = "f32"
    else:
        raise TypeError(f"unsupported dtype {q.dtype}")
    return make_desc(B, T, H, W, heads, D, kt, kh, kw, dtype, scale)


def _check(name, t, shape, dtype):
    if not t.is_cuda or not t.is_contiguous() or tuple(t.shape) != tuple(shape) or t.dtype != dtype:
        raise ValueError(f"{name}: expected a contiguous CUDA {dtype} tensor of shape {tuple(shape)}")


def forward(q, k, v, offsets, kernel=(3, 3, 3), scale=0.0, need_lse=True, out=None, lse=None):
    """Returns (out, lse); lse is None when need_lse is False."""
    desc = _desc(q, kernel, scale)
    P = kernel[0] * kernel[1] * kernel[2]
    for name, t in (("k", k), ("v", v)):
        _check(name, t, q.shape, q.dtype)
    _check("offsets", offsets, tuple(q.shape[:5]) + (P, 3), torch.float32)
    if out is None:
        out = torch.empty_like(q)
    if need_lse and lse is None:
        lse = torch.empty(q.shape[:5], dtype=torch.float32, device=q.device)
    dsa3d_forward(desc, q, k, v, offsets, out, lse if need_lse else None)
    return out, (lse if need_lse else None)


def backward(q, k, v, offsets, lse, dout, kernel=(3, 3, 3), scale=0.0, grads=None, workspace=None,
             phase_events=None):
    """Returns (dq, dk, dv, d_offsets), all float32.  `workspace` (a uint8 CUDA tensor) is
    allocated here when missing or too small.  `phase_events`: optional list of
    DSA3D_BACKWARD_PHASES + 1 created torch.cuda.Event objects marking the phases (see
    dsa3d_backward_timed)."""
    desc = _desc(q, kernel, scale)
    if grads is None:
        f32 = dict(dtype=torch.float32, device=q.device)
        grads = (torch.empty(q.shape, **f32), torch.empty(q.shape, **f32),
                 torch.empty(q.shape, **f32), torch.empty(offsets.shape, **f32))
    dq, dk, dv, doff = grads
    need = dsa3d_backward_workspace_size(desc)
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=q.device)
    if phase_events is None:
        dsa3d_backward(desc, q, k, v, offsets, lse, dout, dq, dk, dv, doff, workspace, need)
    else:
        dsa3d_backward_timed(desc, q, k, v, offsets, lse, dout, dq, dk, dv, doff, workspace, need,
                             events=phase_events)
    return dq, dk, dv, doff
