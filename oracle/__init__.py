"""CPU oracle for 3D Deformable Slide Attention (MegaSlide-DiT, Section 5.2, Eq. (1)).

TEST INFRASTRUCTURE ONLY: only ``tests/``, ``__graft_entry__.smoke()`` and the
bench's CPU-baseline leg may import this package.  It wraps ``dsa3d_oracle.c``
(the attention term and its predicted-weights variant), ``dwconv3d_oracle.c`` (the
depthwise 3D convolution term and the offset network's depthwise convolution) and
``winattn_oracle.c`` (the Swin-DiT baseline's shifted-window attention), plain C with fp64
accumulation and OpenMP, with ctypes, and shares nothing with the GPU library.  The arithmetic and
the readings it follows are described at the top of each C file.
"""
from __future__ import annotations

import ctypes
import math
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRCS = [os.path.join(_HERE, "dsa3d_oracle.c"), os.path.join(_HERE, "dwconv3d_oracle.c"),
         os.path.join(_HERE, "winattn_oracle.c")]
_LIB = os.path.join(_HERE, "liboracle.so")


def build(force: bool = True) -> str:
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-shared", "-fPIC", "-std=c11",
                               *_SRCS, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


class _Problem(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int64), ("T", ctypes.c_int64), ("H", ctypes.c_int64),
                ("W", ctypes.c_int64), ("heads", ctypes.c_int64), ("D", ctypes.c_int64),
                ("kt", ctypes.c_int64), ("kh", ctypes.c_int64), ("kw", ctypes.c_int64),
                ("scale", ctypes.c_double), ("bf16", ctypes.c_int32), ("pad_", ctypes.c_int32)]


class _Conv(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int64), ("T", ctypes.c_int64), ("H", ctypes.c_int64),
                ("W", ctypes.c_int64), ("C", ctypes.c_int64), ("kt", ctypes.c_int64),
                ("kh", ctypes.c_int64), ("kw", ctypes.c_int64), ("bf16", ctypes.c_int32),
                ("pad_", ctypes.c_int32)]


class _Win(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int64) for n in ("B", "T", "H", "W", "heads", "D", "wt", "wh", "ww",
                                              "st", "sh", "sw")] + \
               [("scale", ctypes.c_double), ("bf16", ctypes.c_int32), ("pad_", ctypes.c_int32)]


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        lib = ctypes.CDLL(_LIB)
        vp = ctypes.c_void_p
        lib.orc_forward.argtypes = [ctypes.POINTER(_Problem), vp, vp, vp, vp, vp, ctypes.c_int64, vp, vp]
        lib.orc_forward.restype = ctypes.c_int
        lib.orc_backward.argtypes = [ctypes.POINTER(_Problem), vp, vp, vp, vp, vp, ctypes.c_int64,
                                     ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, vp, vp, vp, vp]
        lib.orc_backward.restype = ctypes.c_int
        lib.orc_backward_rows.argtypes = [ctypes.POINTER(_Problem), vp, vp, vp, vp, vp, vp,
                                          ctypes.c_int64, vp, vp]
        lib.orc_backward_rows.restype = ctypes.c_int
        lib.orc_pw_forward.argtypes = [ctypes.POINTER(_Problem), vp, vp, vp, vp, ctypes.c_int64, vp,
                                       vp]
        lib.orc_pw_forward.restype = ctypes.c_int
        lib.orc_pw_backward.argtypes = [ctypes.POINTER(_Problem), vp, vp, vp, vp, ctypes.c_int64,
                                        ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, vp, vp, vp]
        lib.orc_pw_backward.restype = ctypes.c_int
        W = ctypes.POINTER(_Win)
        lib.orc_win_forward.argtypes = [W, vp, vp, vp, ctypes.c_int64, ctypes.c_int64, vp, vp]
        lib.orc_win_forward.restype = ctypes.c_int
        lib.orc_win_backward.argtypes = [W, vp, vp, vp, vp, ctypes.c_int64, ctypes.c_int64, vp, vp,
                                         vp]
        lib.orc_win_backward.restype = ctypes.c_int
        lib.orc_dwconv_forward.argtypes = [ctypes.POINTER(_Conv), vp, vp, vp, ctypes.c_int64,
                                           ctypes.c_int64, vp]
        lib.orc_dwconv_forward.restype = ctypes.c_int
        lib.orc_dwconv_backward.argtypes = [ctypes.POINTER(_Conv), vp, vp, vp, ctypes.c_int64,
                                            ctypes.c_int64, vp, vp, vp]
        lib.orc_dwconv_backward.restype = ctypes.c_int
        lib.orc_max_threads.argtypes = []
        lib.orc_max_threads.restype = ctypes.c_int
        _lib = lib
    return _lib


def threads() -> int:
    """OpenMP threads the oracle's parallel loops use."""
    return int(_load().orc_max_threads())


def default_scale(head_dim: int) -> float:
    """Logit scale 1/sqrt(head_dim) (per-head reading of the paper's 1/sqrt(d))."""
    return 1.0 / math.sqrt(head_dim)


def _problem(shape, dtype: str, scale):
    B, T, H, W, heads, D, kt, kh, kw = shape
    if scale is None:
        scale = default_scale(D)
    return _Problem(B, T, H, W, heads, D, kt, kh, kw, float(scale), 1 if dtype == "bf16" else 0, 0)


def _check_io(a, dtype):
    want = np.uint16 if dtype == "bf16" else np.float32
    a = np.ascontiguousarray(a)
    if a.dtype != want:
        raise TypeError(f"expected {want} array for dtype {dtype}, got {a.dtype}")
    return a


def forward(shape, dtype, q, k, v, off, rows=None, scale=None):
    """Attention output and LSE for the given flat query rows (all rows if None).

    shape = (B, T, H, W, heads, head_dim, kt, kh, kw); q/k/v are [B,T,H,W,heads,D]
    arrays (float32, or uint16 bf16 bit patterns when dtype == "bf16");
    off is float32 [B,T,H,W,heads,P,3].  Returns (out[nrows, D], lse[nrows]) in fp64.
    """
    pr = _problem(shape, dtype, scale)
    q, k, v = (_check_io(a, dtype) for a in (q, k, v))
    off = np.ascontiguousarray(off, dtype=np.float32)
    B, T, H, W, heads, D = shape[:6]
    if rows is None:
        rows = np.arange(B * T * H * W * heads, dtype=np.int64)
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    out = np.empty((rows.size, D), dtype=np.float64)
    lse = np.empty(rows.size, dtype=np.float64)
    rc = _load().orc_forward(ctypes.byref(pr), q.ctypes.data, k.ctypes.data, v.ctypes.data,
                             off.ctypes.data, rows.ctypes.data, rows.size, out.ctypes.data,
                             lse.ctypes.data)
    if rc != 0:
        raise ValueError("oracle forward: malformed problem")
    return out, lse


def backward_slab(shape, dtype, q, k, v, off, dout, b, m, t0, t1, scale=None, dk=None, dv=None):
    """Gradients from the queries of batch b, head m, frames [t0, t1).

    Returns (dq[(t1-t0),H,W,D], doff[(t1-t0),H,W,P,3], dk[T,H,W,D], dv[T,H,W,D]); dk/dv
    hold only the contributions of those queries (accumulated into the given arrays)."""
    pr = _problem(shape, dtype, scale)
    q, k, v, dout = (_check_io(a, dtype) for a in (q, k, v, dout))
    off = np.ascontiguousarray(off, dtype=np.float32)
    B, T, H, W, heads, D, kt, kh, kw = shape
    P = kt * kh * kw
    dq = np.empty((t1 - t0, H, W, D), dtype=np.float64)
    doff = np.empty((t1 - t0, H, W, P, 3), dtype=np.float64)
    if dk is None:
        dk = np.zeros((T, H, W, D), dtype=np.float64)
    if dv is None:
        dv = np.zeros((T, H, W, D), dtype=np.float64)
    assert dk.flags["C_CONTIGUOUS"] and dv.flags["C_CONTIGUOUS"]
    rc = _load().orc_backward(ctypes.byref(pr), q.ctypes.data, k.ctypes.data, v.ctypes.data,
                              off.ctypes.data, dout.ctypes.data, b, m, t0, t1, dq.ctypes.data,
                              doff.ctypes.data, dk.ctypes.data, dv.ctypes.data)
    if rc != 0:
        raise ValueError("oracle backward: malformed problem")
    return dq, doff, dk, dv


def backward_rows(shape, dtype, q, k, v, off, dout, rows, scale=None):
    """dq[nrows, D] and doff[nrows, P, 3] (fp64) of the given flat query rows."""
    pr = _problem(shape, dtype, scale)
    q, k, v, dout = (_check_io(a, dtype) for a in (q, k, v, dout))
    off = np.ascontiguousarray(off, dtype=np.float32)
    D = shape[5]
    P = shape[6] * shape[7] * shape[8]
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    dq = np.empty((rows.size, D), dtype=np.float64)
    doff = np.empty((rows.size, P, 3), dtype=np.float64)
    rc = _load().orc_backward_rows(ctypes.byref(pr), q.ctypes.data, k.ctypes.data, v.ctypes.data,
                                   off.ctypes.data, dout.ctypes.data, rows.ctypes.data, rows.size,
                                   dq.ctypes.data, doff.ctypes.data)
    if rc != 0:
        raise ValueError("oracle backward: malformed problem")
    return dq, doff


def backward(shape, dtype, q, k, v, off, dout, scale=None):
    """Full gradients (dq, dk, dv as [B,T,H,W,heads,D], doff as [B,T,H,W,heads,P,3]), fp64."""
    B, T, H, W, heads, D, kt, kh, kw = shape
    P = kt * kh * kw
    dq = np.empty((B, T, H, W, heads, D))
    dk = np.empty((B, T, H, W, heads, D))
    dv = np.empty((B, T, H, W, heads, D))
    doff = np.empty((B, T, H, W, heads, P, 3))
    for b in range(B):
        for m in range(heads):
            a, o, kk, vv = backward_slab(shape, dtype, q, k, v, off, dout, b, m, 0, T, scale)
            dq[b, :, :, :, m] = a
            doff[b, :, :, :, m] = o
            dk[b, :, :, :, m] = kk
            dv[b, :, :, :, m] = vv
    return dq, dk, dv, doff


# ----------------------------------------------------------------------------- predicted weights

def pw_forward(shape, dtype, logits, v, off, rows=None):
    """Predicted-weights variant: output and LSE of the given flat rows (all if None), fp64.

    logits float32 [B,T,H,W,heads,P]; v as in forward(); off float32 [..,heads,P,3]."""
    pr = _problem(shape, dtype, 1.0)
    v = _check_io(v, dtype)
    logits = np.ascontiguousarray(logits, dtype=np.float32)
    off = np.ascontiguousarray(off, dtype=np.float32)
    B, T, H, W, heads, D = shape[:6]
    if rows is None:
        rows = np.arange(B * T * H * W * heads, dtype=np.int64)
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    out = np.empty((rows.size, D), dtype=np.float64)
    lse = np.empty(rows.size, dtype=np.float64)
    rc = _load().orc_pw_forward(ctypes.byref(pr), logits.ctypes.data, v.ctypes.data,
                                off.ctypes.data, rows.ctypes.data, rows.size, out.ctypes.data,
                                lse.ctypes.data)
    if rc != 0:
        raise ValueError("oracle pw forward: malformed problem")
    return out, lse


def pw_backward_slab(shape, dtype, logits, v, off, dout, b, m, t0, t1, dv=None):
    """Predicted-weights variant: gradients from the queries of batch b, head m, frames
    [t0, t1).  Returns (dlogits[(t1-t0),H,W,P], doff[(t1-t0),H,W,P,3], dv[T,H,W,D]); dv holds
    only those queries' contributions (accumulated into the given array)."""
    pr = _problem(shape, dtype, 1.0)
    v, dout = _check_io(v, dtype), _check_io(dout, dtype)
    logits = np.ascontiguousarray(logits, dtype=np.float32)
    off = np.ascontiguousarray(off, dtype=np.float32)
    B, T, H, W, heads, D, kt, kh, kw = shape
    P = kt * kh * kw
    dlog = np.empty((t1 - t0, H, W, P), dtype=np.float64)
    doff = np.empty((t1 - t0, H, W, P, 3), dtype=np.float64)
    if dv is None:
        dv = np.zeros((T, H, W, D), dtype=np.float64)
    assert dv.flags["C_CONTIGUOUS"]
    rc = _load().orc_pw_backward(ctypes.byref(pr), logits.ctypes.data, v.ctypes.data,
                                 off.ctypes.data, dout.ctypes.data, b, m, t0, t1,
                                 dlog.ctypes.data, doff.ctypes.data, dv.ctypes.data)
    if rc != 0:
        raise ValueError("oracle pw backward: malformed problem")
    return dlog, doff, dv


def pw_backward(shape, dtype, logits, v, off, dout):
    """Full predicted-weights gradients: dlogits [B,T,H,W,heads,P], dv [B,T,H,W,heads,D],
    doff [B,T,H,W,heads,P,3], fp64."""
    B, T, H, W, heads, D, kt, kh, kw = shape
    P = kt * kh * kw
    dlog = np.empty((B, T, H, W, heads, P))
    dv = np.empty((B, T, H, W, heads, D))
    doff = np.empty((B, T, H, W, heads, P, 3))
    for b in range(B):
        for m in range(heads):
            a, o, vv = pw_backward_slab(shape, dtype, logits, v, off, dout, b, m, 0, T)
            dlog[b, :, :, :, m] = a
            doff[b, :, :, :, m] = o
            dv[b, :, :, :, m] = vv
    return dlog, dv, doff


# ----------------------------------------------------------------------------- depthwise conv

def _conv(shape, dtype):
    B, T, H, W, C, kt, kh, kw = shape
    return _Conv(B, T, H, W, C, kt, kh, kw, 1 if dtype == "bf16" else 0, 0)


def dwconv_forward(shape, dtype, x, w, bias=None, frames=None):
    """Depthwise 3D convolution y = conv(x) + bias of frames [t0, t1) (all if None).

    shape = (B, T, H, W, C, kt, kh, kw); x is [B,T,H,W,C] (float32, or uint16 bf16 bit
    patterns when dtype == "bf16"); w is float32 [C,kt,kh,kw]; bias float32 [C] or None.
    Returns y[B, t1-t0, H, W, C] in fp64."""
    pr = _conv(shape, dtype)
    x = _check_io(x, dtype)
    w = np.ascontiguousarray(w, dtype=np.float32)
    bias = None if bias is None else np.ascontiguousarray(bias, dtype=np.float32)
    B, T, H, W, C = shape[:5]
    t0, t1 = (0, T) if frames is None else frames
    y = np.empty((B, t1 - t0, H, W, C), dtype=np.float64)
    rc = _load().orc_dwconv_forward(ctypes.byref(pr), x.ctypes.data, w.ctypes.data,
                                    None if bias is None else bias.ctypes.data, t0, t1,
                                    y.ctypes.data)
    if rc != 0:
        raise ValueError("oracle dwconv forward: malformed problem")
    return y


def dwconv_backward(shape, dtype, x, w, dy, frames=None, weight_grads=True):
    """(dx[B, t1-t0, H, W, C], dw[C,kt,kh,kw], dbias[C]) in fp64; dx covers frames [t0, t1)
    (all if None); dw and dbias (None unless weight_grads) sum over the whole grid."""
    pr = _conv(shape, dtype)
    x, dy = _check_io(x, dtype), _check_io(dy, dtype)
    w = np.ascontiguousarray(w, dtype=np.float32)
    B, T, H, W, C, kt, kh, kw = shape
    t0, t1 = (0, T) if frames is None else frames
    dx = np.empty((B, t1 - t0, H, W, C), dtype=np.float64)
    dw = np.empty((C, kt, kh, kw), dtype=np.float64) if weight_grads else None
    db = np.empty(C, dtype=np.float64) if weight_grads else None
    rc = _load().orc_dwconv_backward(ctypes.byref(pr), x.ctypes.data, w.ctypes.data,
                                     dy.ctypes.data, t0, t1, dx.ctypes.data,
                                     None if dw is None else dw.ctypes.data,
                                     None if db is None else db.ctypes.data)
    if rc != 0:
        raise ValueError("oracle dwconv backward: malformed problem")
    return dx, dw, db


# ----------------------------------------------------------------------------- window attention

def _win(shape, dtype, scale):
    B, T, H, W, heads, D, wt, wh, ww, st, sh, sw = shape
    if scale is None:
        scale = default_scale(D)
    return _Win(B, T, H, W, heads, D, wt, wh, ww, st, sh, sw, float(scale),
                1 if dtype == "bf16" else 0, 0)


def win_forward(shape, dtype, q, k, v, frames=None, scale=None):
    """Shifted-window attention output [B, t1-t0, H, W, heads, D] and LSE [B, t1-t0, H, W, heads]
    (fp64) for frames [t0, t1) (all if None).  shape = (B, T, H, W, heads, D, wt, wh, ww,
    st, sh, sw)."""
    pr = _win(shape, dtype, scale)
    q, k, v = (_check_io(a, dtype) for a in (q, k, v))
    B, T, H, W, heads, D = shape[:6]
    t0, t1 = (0, T) if frames is None else frames
    out = np.empty((B, t1 - t0, H, W, heads, D), dtype=np.float64)
    lse = np.empty((B, t1 - t0, H, W, heads), dtype=np.float64)
    rc = _load().orc_win_forward(ctypes.byref(pr), q.ctypes.data, k.ctypes.data, v.ctypes.data,
                                 t0, t1, out.ctypes.data, lse.ctypes.data)
    if rc != 0:
        raise ValueError("oracle window forward: malformed problem")
    return out, lse


def win_backward(shape, dtype, q, k, v, dout, scale=None, frames=None):
    """(dq, dk, dv) of the shifted-window attention for the tokens of frames [t0, t1) (all if
    None), [B, t1 - t0, H, W, heads, D] fp64: dq is complete, dk and dv hold the contributions
    of the queries in the range (complete for keys whose window region lies inside it)."""
    pr = _win(shape, dtype, scale)
    q, k, v, dout = (_check_io(a, dtype) for a in (q, k, v, dout))
    t0, t1 = (0, shape[1]) if frames is None else frames
    oshape = (q.shape[0], t1 - t0) + tuple(q.shape[2:])
    dq, dk, dv = (np.empty(oshape, dtype=np.float64) for _ in range(3))
    rc = _load().orc_win_backward(ctypes.byref(pr), q.ctypes.data, k.ctypes.data, v.ctypes.data,
                                  dout.ctypes.data, t0, t1, dq.ctypes.data, dk.ctypes.data,
                                  dv.ctypes.data)
    if rc != 0:
        raise ValueError("oracle window backward: malformed problem")
    return dq, dk, dv

