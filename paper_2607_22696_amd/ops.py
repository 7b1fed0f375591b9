"""Tensor-level calls of the C ABI: allocate outputs with torch, then call the library.

q, k, v (and dout) are [B, T, H, W, heads, head_dim] CUDA tensors in float32 or bfloat16;
offsets are float32 [B, T, H, W, heads, P, 3] with (x, y, z) = (w, h, t) in token units.
"""
from __future__ import annotations

import torch

from ._binding import (dsa3d_backward, dsa3d_backward_timed, dsa3d_backward_workspace_size,
                       dsa3d_dwconv3d_backward, dsa3d_dwconv3d_backward_workspace_size,
                       dsa3d_dwconv3d_forward, dsa3d_forward, dsa3d_pw_backward,
                       dsa3d_pw_backward_workspace_size, dsa3d_pw_forward, dsa3d_win_backward,
                       dsa3d_win_backward_workspace_size, dsa3d_win_forward, make_conv_desc,
                       make_desc, make_win_desc)


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


def _conv_desc(x, weight):
    if x.dim() != 5:
        raise ValueError("x must be [B, T, H, W, C]")
    B, T, H, W, C = x.shape
    if weight.dim() != 4 or weight.shape[0] != C:
        raise ValueError("weight must be [C, kt, kh, kw]")
    kt, kh, kw = weight.shape[1:]
    return make_conv_desc(B, T, H, W, C, kt, kh, kw,
                          "bf16" if x.dtype == torch.bfloat16 else "f32")


def dwconv3d_forward(x, weight, bias=None, out=None, accumulate=False):
    """Depthwise 3D convolution (the DWConv3D term of Eq. (1)): x [B,T,H,W,C] (bf16 or fp32),
    weight float32 [C,kt,kh,kw], bias float32 [C] or None.  Returns out (x's dtype); with
    accumulate=True the result is added to `out`."""
    desc = _conv_desc(x, weight)
    if out is None:
        if accumulate:
            raise ValueError("accumulate needs an output to add to")
        out = torch.empty_like(x)
    dsa3d_dwconv3d_forward(desc, x, weight, bias, out, accumulate)
    return out


def dwconv3d_backward(x, weight, dy, need_dx=True, need_dweight=True, need_dbias=True,
                      dx=None, accumulate_dx=False, workspace=None):
    """Returns (dx, dweight, dbias) as float32 (None where not requested)."""
    desc = _conv_desc(x, weight)
    f32 = dict(dtype=torch.float32, device=x.device)
    if need_dx and dx is None:
        if accumulate_dx:
            raise ValueError("accumulate_dx needs a dx to add to")
        dx = torch.empty(x.shape, **f32)
    dx = dx if need_dx else None
    dw = torch.empty(weight.shape, **f32) if need_dweight else None
    db = torch.empty(weight.shape[0], **f32) if need_dbias else None
    need = 0
    if dw is not None or db is not None:
        need = dsa3d_dwconv3d_backward_workspace_size(desc)
        if workspace is None or workspace.numel() < need:
            workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=x.device)
    dsa3d_dwconv3d_backward(desc, x, weight, dy, dx, dw, db, workspace, need, accumulate_dx)
    return dx, dw, db


def pw_forward(logits, v, offsets, kernel=(3, 3, 3), need_lse=True, out=None, lse=None):
    """Predicted-weights variant: softmax over the given logits [B,T,H,W,heads,P] (fp32)
    instead of q.k.  Returns (out, lse)."""
    desc = _desc(v, kernel, 0.0)
    if out is None:
        out = torch.empty_like(v)
    if need_lse and lse is None:
        lse = torch.empty(v.shape[:-1], dtype=torch.float32, device=v.device)
    dsa3d_pw_forward(desc, logits, v, offsets, out, lse if need_lse else None)
    return out, lse


def pw_backward(logits, v, offsets, lse, dout, kernel=(3, 3, 3), grads=None, workspace=None,
                phase_events=None):
    """Returns (dlogits, dv, d_offsets), float32.  `phase_events` as for backward()."""
    desc = _desc(v, kernel, 0.0)
    if grads is None:
        f32 = dict(dtype=torch.float32, device=v.device)
        grads = (torch.empty(logits.shape, **f32), torch.empty(v.shape, **f32),
                 torch.empty(offsets.shape, **f32))
    dlog, dv, doff = grads
    need = dsa3d_pw_backward_workspace_size(desc)
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=v.device)
    dsa3d_pw_backward(desc, logits, v, offsets, lse, dout, dlog, dv, doff, workspace, need,
                      events=phase_events)
    return dlog, dv, doff


def _win_desc(q, window, shift, scale):
    if q.dim() != 6 or q.dtype != torch.bfloat16:
        raise ValueError("q must be a bfloat16 [B, T, H, W, heads, head_dim] tensor")
    B, T, H, W, heads, D = q.shape
    return make_win_desc(B, T, H, W, heads, D, window, shift, "bf16", scale)


def win_forward(q, k, v, window=(3, 16, 16), shift=(0, 0, 0), scale=0.0, need_lse=True,
                need_residual=True, out=None, lse=None, out_res=None):
    """Fixed / shifted window attention (bf16).  Returns (out, lse, out_res); out_res, the bf16
    rounding residual of out that the backward uses for an exact Delta, is None when
    need_residual is False (and lse when need_lse is False)."""
    desc = _win_desc(q, window, shift, scale)
    for name, t in (("k", k), ("v", v)):
        _check(name, t, q.shape, q.dtype)
    if out is None:
        out = torch.empty_like(q)
    if need_lse and lse is None:
        lse = torch.empty(q.shape[:5], dtype=torch.float32, device=q.device)
    if need_residual and out_res is None:
        out_res = torch.empty_like(q)
    dsa3d_win_forward(desc, q, k, v, out, out_res if need_residual else None,
                      lse if need_lse else None)
    return out, (lse if need_lse else None), (out_res if need_residual else None)


def win_backward(q, k, v, out, out_res, lse, dout, window=(3, 16, 16), shift=(0, 0, 0),
                 scale=0.0, grads=None, workspace=None, phase_events=None):
    """Returns (dq, dk, dv), float32.  out_res may be None (Delta from the rounded out alone).
    `phase_events`: optional DSA3D_WIN_BACKWARD_PHASES + 1 created torch.cuda.Event objects
    marking the two passes."""
    desc = _win_desc(q, window, shift, scale)
    if grads is None:
        f32 = dict(dtype=torch.float32, device=q.device)
        grads = tuple(torch.empty(q.shape, **f32) for _ in range(3))
    dq, dk, dv = grads
    need = dsa3d_win_backward_workspace_size(desc)
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=q.device)
    dsa3d_win_backward(desc, q, k, v, out, out_res, lse, dout, dq, dk, dv, workspace, need,
                       events=phase_events)
    return dq, dk, dv
