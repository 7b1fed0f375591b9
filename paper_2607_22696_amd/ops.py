"""Tensor-level calls of the C ABI: check and allocate tensors with torch, then call the library.

q, k, v (and dout) are [B, T, H, W, heads, head_dim] CUDA tensors in float32 or bfloat16;
offsets are float32 [B, T, H, W, heads, P, 3] with (x, y, z) = (w, h, t) in token units.

The C ABI sees raw device pointers only and cannot know how large a buffer is, so every
tensor handed to it is checked here first (device, dtype, shape, contiguity): a wrong one
raises ValueError before anything is launched.
"""
from __future__ import annotations

import torch

from ._binding import (dsa3d_backward, dsa3d_backward_timed, dsa3d_backward_workspace_size,
                       dsa3d_dwconv3d_backward, dsa3d_dwconv3d_backward_workspace_size,
                       dsa3d_dwconv3d_forward, dsa3d_forward, dsa3d_pw_backward,
                       dsa3d_pw_backward_workspace_size, dsa3d_pw_forward, dsa3d_win_backward,
                       dsa3d_win_backward_workspace_size, dsa3d_win_forward, make_conv_desc,
                       make_desc, make_win_desc)

_IO_DTYPES = {torch.bfloat16: "bf16", torch.float32: "f32"}


class _Checks:
    """Collects every problem with the arguments of one call, then raises them together."""

    def __init__(self, where):
        self.where = where
        self.problems = []

    def tensor(self, name, t, shape, dtype, device):
        if not isinstance(t, torch.Tensor):
            self.problems.append(f"{name}: expected a tensor, got {type(t).__name__}")
            return
        bad = []
        if t.dtype != dtype:
            bad.append(f"dtype {t.dtype} (expected {dtype})")
        if tuple(t.shape) != tuple(shape):
            bad.append(f"shape {tuple(t.shape)} (expected {tuple(shape)})")
        if not t.is_contiguous():
            bad.append("not contiguous")
        if t.device != device:
            bad.append(f"on {t.device} (expected {device})")
        if bad:
            self.problems.append(f"{name}: " + ", ".join(bad))

    def workspace(self, t, device):
        if t is not None:
            n = t.numel() if isinstance(t, torch.Tensor) else 0
            self.tensor("workspace", t, (n,), torch.uint8, device)

    def optional(self, name, t, shape, dtype, device):
        if t is not None:
            self.tensor(name, t, shape, dtype, device)

    def done(self):
        if self.problems:
            raise ValueError(f"{self.where}: " + "; ".join(self.problems))


def _lead(chk, name, x, ndim, what, dtypes=_IO_DTYPES):
    """The tensor that fixes shape, dtype and device of a call: a CUDA tensor of `ndim` dims in
    one of `dtypes`.  Returns its device; raises at once when the other tensors cannot be
    checked against it (not a tensor, wrong rank, unsupported dtype), else the remaining
    problems are collected with those of the other tensors."""
    if not isinstance(x, torch.Tensor):
        chk.problems.append(f"{name}: expected a tensor, got {type(x).__name__}")
        chk.done()
    if x.dim() != ndim:
        chk.problems.append(f"{name}: expected {what}, got shape {tuple(x.shape)}")
    if x.dtype not in dtypes:
        chk.problems.append(f"{name}: unsupported dtype {x.dtype}")
    chk.done()
    if not x.is_cuda:
        chk.problems.append(f"{name}: not a CUDA tensor ({x.device})")
    if not x.is_contiguous():
        chk.problems.append(f"{name}: not contiguous")
    return x.device


def _kernel(chk, kernel):
    try:
        kt, kh, kw = (int(a) for a in kernel)
    except (TypeError, ValueError):
        chk.problems.append(f"kernel: expected three odd sizes, got {kernel!r}")
        return 1, 1, 1
    return kt, kh, kw


def _desc(q, kernel, scale):
    B, T, H, W, heads, D = q.shape
    kt, kh, kw = kernel
    return make_desc(B, T, H, W, heads, D, kt, kh, kw, _IO_DTYPES[q.dtype], scale)


def forward(q, k, v, offsets, kernel=(3, 3, 3), scale=0.0, need_lse=True, out=None, lse=None):
    """Returns (out, lse); lse is None when need_lse is False."""
    chk = _Checks("forward")
    dev = _lead(chk, "q", q, 6, "[B, T, H, W, heads, head_dim]")
    kern = _kernel(chk, kernel)
    P = kern[0] * kern[1] * kern[2]
    for name, t in (("k", k), ("v", v)):
        chk.tensor(name, t, q.shape, q.dtype, dev)
    chk.tensor("offsets", offsets, tuple(q.shape[:5]) + (P, 3), torch.float32, dev)
    chk.optional("out", out, q.shape, q.dtype, dev)
    if need_lse:
        chk.optional("lse", lse, q.shape[:5], torch.float32, dev)
    chk.done()
    desc = _desc(q, kern, scale)
    if out is None:
        out = torch.empty_like(q)
    if need_lse and lse is None:
        lse = torch.empty(q.shape[:5], dtype=torch.float32, device=dev)
    dsa3d_forward(desc, q, k, v, offsets, out, lse if need_lse else None)
    return out, (lse if need_lse else None)


def backward(q, k, v, offsets, lse, dout, kernel=(3, 3, 3), scale=0.0, grads=None, workspace=None,
             phase_events=None, out=None):
    """Returns (dq, dk, dv, d_offsets), all float32.  `out` (the forward's output) is optional:
    the library forms Delta exactly without it.  `grads` = (dq, dk, dv, d_offsets) to write
    into.  `workspace` (a uint8 CUDA tensor) is allocated here when missing or too small.
    `phase_events`: optional list of DSA3D_BACKWARD_PHASES + 1 created torch.cuda.Event objects
    marking the phases (see dsa3d_backward_timed)."""
    chk = _Checks("backward")
    dev = _lead(chk, "q", q, 6, "[B, T, H, W, heads, head_dim]")
    kern = _kernel(chk, kernel)
    P = kern[0] * kern[1] * kern[2]
    off_shape = tuple(q.shape[:5]) + (P, 3)
    for name, t in (("k", k), ("v", v), ("dout", dout)):
        chk.tensor(name, t, q.shape, q.dtype, dev)
    chk.optional("out", out, q.shape, q.dtype, dev)
    chk.tensor("offsets", offsets, off_shape, torch.float32, dev)
    chk.tensor("lse", lse, q.shape[:5], torch.float32, dev)
    if grads is not None:
        if len(grads) != 4:
            chk.problems.append("grads: expected (dq, dk, dv, d_offsets)")
        else:
            for name, t in zip(("dq", "dk", "dv"), grads[:3]):
                chk.tensor(name, t, q.shape, torch.float32, dev)
            chk.tensor("d_offsets", grads[3], off_shape, torch.float32, dev)
    chk.workspace(workspace, dev)
    chk.done()
    desc = _desc(q, kern, scale)
    if grads is None:
        f32 = dict(dtype=torch.float32, device=dev)
        grads = (torch.empty(q.shape, **f32), torch.empty(q.shape, **f32),
                 torch.empty(q.shape, **f32), torch.empty(off_shape, **f32))
    dq, dk, dv, doff = grads
    need = dsa3d_backward_workspace_size(desc)
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    if phase_events is None:
        dsa3d_backward(desc, q, k, v, offsets, out, lse, dout, dq, dk, dv, doff, workspace, need)
    else:
        dsa3d_backward_timed(desc, q, k, v, offsets, out, lse, dout, dq, dk, dv, doff, workspace,
                             need, events=phase_events)
    return dq, dk, dv, doff


def _conv_desc(chk, x, weight):
    dev = _lead(chk, "x", x, 5, "[B, T, H, W, C]")
    if not isinstance(weight, torch.Tensor) or weight.dim() != 4:
        chk.problems.append("weight: expected a float32 [C, kt, kh, kw] tensor")
        chk.done()
    B, T, H, W, C = x.shape
    kt, kh, kw = weight.shape[1:]
    chk.tensor("weight", weight, (C, kt, kh, kw), torch.float32, dev)
    return dev, make_conv_desc(B, T, H, W, C, kt, kh, kw, _IO_DTYPES[x.dtype])


def dwconv3d_forward(x, weight, bias=None, out=None, accumulate=False):
    """Depthwise 3D convolution (the DWConv3D term of Eq. (1)): x [B,T,H,W,C] (bf16 or fp32),
    weight float32 [C,kt,kh,kw], bias float32 [C] or None.  Returns out (x's dtype); with
    accumulate=True the result is added to `out`."""
    chk = _Checks("dwconv3d_forward")
    dev, desc = _conv_desc(chk, x, weight)
    chk.optional("bias", bias, (x.shape[4],), torch.float32, dev)
    chk.optional("out", out, x.shape, x.dtype, dev)
    if accumulate and out is None:
        chk.problems.append("accumulate needs an output to add to")
    chk.done()
    if out is None:
        out = torch.empty_like(x)
    dsa3d_dwconv3d_forward(desc, x, weight, bias, out, accumulate)
    return out


def dwconv3d_backward(x, weight, dy, need_dx=True, need_dweight=True, need_dbias=True,
                      dx=None, accumulate_dx=False, workspace=None):
    """Returns (dx, dweight, dbias) as float32 (None where not requested)."""
    chk = _Checks("dwconv3d_backward")
    dev, desc = _conv_desc(chk, x, weight)
    chk.tensor("dy", dy, x.shape, x.dtype, dev)
    if need_dx:
        chk.optional("dx", dx, x.shape, torch.float32, dev)
        if accumulate_dx and dx is None:
            chk.problems.append("accumulate_dx needs a dx to add to")
    chk.workspace(workspace, dev)
    chk.done()
    f32 = dict(dtype=torch.float32, device=dev)
    if need_dx and dx is None:
        dx = torch.empty(x.shape, **f32)
    dx = dx if need_dx else None
    dw = torch.empty(weight.shape, **f32) if need_dweight else None
    db = torch.empty(weight.shape[0], **f32) if need_dbias else None
    need = 0
    if dw is not None or db is not None:
        need = dsa3d_dwconv3d_backward_workspace_size(desc)
        if workspace is None or workspace.numel() < need:
            workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    dsa3d_dwconv3d_backward(desc, x, weight, dy, dx, dw, db, workspace, need, accumulate_dx)
    return dx, dw, db


def pw_forward(logits, v, offsets, kernel=(3, 3, 3), need_lse=True, out=None, lse=None):
    """Predicted-weights variant: softmax over the given logits [B,T,H,W,heads,P] (fp32)
    instead of q.k.  Returns (out, lse)."""
    chk = _Checks("pw_forward")
    dev = _lead(chk, "v", v, 6, "[B, T, H, W, heads, head_dim]")
    kern = _kernel(chk, kernel)
    P = kern[0] * kern[1] * kern[2]
    chk.tensor("logits", logits, tuple(v.shape[:5]) + (P,), torch.float32, dev)
    chk.tensor("offsets", offsets, tuple(v.shape[:5]) + (P, 3), torch.float32, dev)
    chk.optional("out", out, v.shape, v.dtype, dev)
    if need_lse:
        chk.optional("lse", lse, v.shape[:5], torch.float32, dev)
    chk.done()
    desc = _desc(v, kern, 0.0)
    if out is None:
        out = torch.empty_like(v)
    if need_lse and lse is None:
        lse = torch.empty(v.shape[:-1], dtype=torch.float32, device=dev)
    dsa3d_pw_forward(desc, logits, v, offsets, out, lse if need_lse else None)
    return out, (lse if need_lse else None)


def pw_backward(logits, v, offsets, lse, dout, kernel=(3, 3, 3), grads=None, workspace=None,
                phase_events=None):
    """Returns (dlogits, dv, d_offsets), float32.  `phase_events` as for backward()."""
    chk = _Checks("pw_backward")
    dev = _lead(chk, "v", v, 6, "[B, T, H, W, heads, head_dim]")
    kern = _kernel(chk, kernel)
    P = kern[0] * kern[1] * kern[2]
    lshape, oshape = tuple(v.shape[:5]) + (P,), tuple(v.shape[:5]) + (P, 3)
    chk.tensor("logits", logits, lshape, torch.float32, dev)
    chk.tensor("offsets", offsets, oshape, torch.float32, dev)
    chk.tensor("lse", lse, v.shape[:5], torch.float32, dev)
    chk.tensor("dout", dout, v.shape, v.dtype, dev)
    if grads is not None:
        if len(grads) != 3:
            chk.problems.append("grads: expected (dlogits, dv, d_offsets)")
        else:
            chk.tensor("dlogits", grads[0], lshape, torch.float32, dev)
            chk.tensor("dv", grads[1], v.shape, torch.float32, dev)
            chk.tensor("d_offsets", grads[2], oshape, torch.float32, dev)
    chk.workspace(workspace, dev)
    chk.done()
    desc = _desc(v, kern, 0.0)
    if grads is None:
        f32 = dict(dtype=torch.float32, device=dev)
        grads = (torch.empty(lshape, **f32), torch.empty(v.shape, **f32),
                 torch.empty(oshape, **f32))
    dlog, dv, doff = grads
    need = dsa3d_pw_backward_workspace_size(desc)
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    dsa3d_pw_backward(desc, logits, v, offsets, lse, dout, dlog, dv, doff, workspace, need,
                      events=phase_events)
    return dlog, dv, doff


def _win_lead(chk, q):
    return _lead(chk, "q", q, 6, "[B, T, H, W, heads, head_dim]", {torch.bfloat16: "bf16"})


def win_forward(q, k, v, window=(3, 16, 16), shift=(0, 0, 0), scale=0.0, need_lse=True,
                need_residual=True, out=None, lse=None, out_res=None):
    """Fixed / shifted window attention (bf16).  Returns (out, lse, out_res); out_res, the bf16
    rounding residual of out that the backward uses for an exact Delta, is None when
    need_residual is False (and lse when need_lse is False)."""
    chk = _Checks("win_forward")
    dev = _win_lead(chk, q)
    for name, t in (("k", k), ("v", v)):
        chk.tensor(name, t, q.shape, q.dtype, dev)
    chk.optional("out", out, q.shape, q.dtype, dev)
    if need_lse:
        chk.optional("lse", lse, q.shape[:5], torch.float32, dev)
    if need_residual:
        chk.optional("out_res", out_res, q.shape, q.dtype, dev)
    chk.done()
    B, T, H, W, heads, D = q.shape
    desc = make_win_desc(B, T, H, W, heads, D, window, shift, "bf16", scale)
    if out is None:
        out = torch.empty_like(q)
    if need_lse and lse is None:
        lse = torch.empty(q.shape[:5], dtype=torch.float32, device=dev)
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
    chk = _Checks("win_backward")
    dev = _win_lead(chk, q)
    for name, t in (("k", k), ("v", v), ("out", out), ("dout", dout)):
        chk.tensor(name, t, q.shape, q.dtype, dev)
    chk.optional("out_res", out_res, q.shape, q.dtype, dev)
    chk.tensor("lse", lse, q.shape[:5], torch.float32, dev)
    if grads is not None:
        if len(grads) != 3:
            chk.problems.append("grads: expected (dq, dk, dv)")
        else:
            for name, t in zip(("dq", "dk", "dv"), grads):
                chk.tensor(name, t, q.shape, torch.float32, dev)
    chk.workspace(workspace, dev)
    chk.done()
    B, T, H, W, heads, D = q.shape
    desc = make_win_desc(B, T, H, W, heads, D, window, shift, "bf16", scale)
    if grads is None:
        f32 = dict(dtype=torch.float32, device=dev)
        grads = tuple(torch.empty(q.shape, **f32) for _ in range(3))
    dq, dk, dv = grads
    need = dsa3d_win_backward_workspace_size(desc)
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    dsa3d_win_backward(desc, q, k, v, out, out_res, lse, dout, dq, dk, dv, workspace, need,
                       events=phase_events)
    return dq, dk, dv
