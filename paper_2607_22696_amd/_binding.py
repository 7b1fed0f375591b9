"""ctypes binding of libdsa3d.so with the same entry-point names as include/dsa3d.h.

Argument marshalling only: descriptors are packed, tensors become device pointers and the
current torch stream becomes the hipStream_t.  Every step of the operator runs in the HIP
kernels of the library; there is no fallback, so a missing library is an error.
"""
from __future__ import annotations

import ctypes
import math
import os

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libdsa3d.so")

DSA3D_OK = 0
DSA3D_ERR_NULL_POINTER = 1
DSA3D_ERR_INVALID_SHAPE = 2
DSA3D_ERR_UNSUPPORTED = 3
DSA3D_ERR_MISALIGNED = 4
DSA3D_ERR_WORKSPACE = 5
DSA3D_ERR_DEVICE = 6
DSA3D_ERR_ALIAS = 7
DSA3D_ERR_SCRATCH = 8

DSA3D_NOALLOC_SCRATCH_BYTES = 128 << 20

DSA3D_F32 = 0
DSA3D_BF16 = 1
DSA3D_MAX_POINTS = 1024

DSA3D_BACKWARD_PHASES = 4

DSA3D_DWCONV_MAX_TAPS = 128

EXPORTED = ("dsa3d_forward", "dsa3d_backward", "dsa3d_backward_timed", "dsa3d_backward_noalloc",
            "dsa3d_backward_workspace_size", "dsa3d_status_string", "dsa3d_abi_version",
            "dsa3d_dwconv3d_forward", "dsa3d_dwconv3d_backward_workspace_size",
            "dsa3d_dwconv3d_backward", "dsa3d_pw_forward", "dsa3d_pw_backward_workspace_size",
            "dsa3d_pw_backward", "dsa3d_win_forward", "dsa3d_win_backward_workspace_size",
            "dsa3d_win_backward")

DSA3D_WIN_MAX_TOKENS = 65536
DSA3D_WIN_BACKWARD_PHASES = 2


class dsa3d_desc(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("frames", ctypes.c_int32), ("height", ctypes.c_int32),
                ("width", ctypes.c_int32), ("heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("kt", ctypes.c_int32), ("kh", ctypes.c_int32), ("kw", ctypes.c_int32),
                ("scale", ctypes.c_float), ("dtype", ctypes.c_int32)]


class dsa3d_dwconv_desc(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("frames", ctypes.c_int32), ("height", ctypes.c_int32),
                ("width", ctypes.c_int32), ("channels", ctypes.c_int32), ("kt", ctypes.c_int32),
                ("kh", ctypes.c_int32), ("kw", ctypes.c_int32), ("dtype", ctypes.c_int32)]


class dsa3d_win_desc(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("frames", ctypes.c_int32), ("height", ctypes.c_int32),
                ("width", ctypes.c_int32), ("heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("wt", ctypes.c_int32), ("wh", ctypes.c_int32), ("ww", ctypes.c_int32),
                ("st", ctypes.c_int32), ("sh", ctypes.c_int32), ("sw", ctypes.c_int32),
                ("scale", ctypes.c_float), ("dtype", ctypes.c_int32)]


class Dsa3dError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {status_string(status)} (status {status})")


_lib = None


def load():
    """Load the built library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with paper_2607_22696_amd/build.py "
                              "(the operator has no non-HIP implementation)")
        lib = ctypes.CDLL(LIB_PATH)
        vp, pd = ctypes.c_void_p, ctypes.POINTER(dsa3d_desc)
        lib.dsa3d_forward.argtypes = [pd, vp, vp, vp, vp, vp, vp, vp]
        lib.dsa3d_forward.restype = ctypes.c_int
        lib.dsa3d_backward.argtypes = [pd, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                       ctypes.c_size_t, vp]
        lib.dsa3d_backward.restype = ctypes.c_int
        lib.dsa3d_backward_timed.argtypes = [pd, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                             ctypes.c_size_t, vp, ctypes.POINTER(vp)]
        lib.dsa3d_backward_timed.restype = ctypes.c_int
        lib.dsa3d_backward_noalloc.argtypes = [pd, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]
        lib.dsa3d_backward_noalloc.restype = ctypes.c_int
        lib.dsa3d_pw_forward.argtypes = [pd, vp, vp, vp, vp, vp, vp]
        lib.dsa3d_pw_forward.restype = ctypes.c_int
        lib.dsa3d_pw_backward_workspace_size.argtypes = [pd]
        lib.dsa3d_pw_backward_workspace_size.restype = ctypes.c_size_t
        lib.dsa3d_pw_backward.argtypes = [pd, vp, vp, vp, vp, vp, vp, vp, vp, vp, ctypes.c_size_t, vp,
                                          ctypes.POINTER(vp)]
        lib.dsa3d_pw_backward.restype = ctypes.c_int
        cd = ctypes.POINTER(dsa3d_dwconv_desc)
        lib.dsa3d_dwconv3d_forward.argtypes = [cd, vp, vp, vp, vp, ctypes.c_int, vp]
        lib.dsa3d_dwconv3d_forward.restype = ctypes.c_int
        lib.dsa3d_dwconv3d_backward_workspace_size.argtypes = [cd]
        lib.dsa3d_dwconv3d_backward_workspace_size.restype = ctypes.c_size_t
        lib.dsa3d_dwconv3d_backward.argtypes = [cd, vp, vp, vp, vp, ctypes.c_int, vp, vp, vp,
                                                ctypes.c_size_t, vp]
        lib.dsa3d_dwconv3d_backward.restype = ctypes.c_int
        wd = ctypes.POINTER(dsa3d_win_desc)
        lib.dsa3d_win_forward.argtypes = [wd, vp, vp, vp, vp, vp, vp, vp]
        lib.dsa3d_win_forward.restype = ctypes.c_int
        lib.dsa3d_win_backward_workspace_size.argtypes = [wd]
        lib.dsa3d_win_backward_workspace_size.restype = ctypes.c_size_t
        lib.dsa3d_win_backward.argtypes = [wd, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                           ctypes.c_size_t, vp, ctypes.POINTER(vp)]
        lib.dsa3d_win_backward.restype = ctypes.c_int
        lib.dsa3d_backward_workspace_size.argtypes = [pd]
        lib.dsa3d_backward_workspace_size.restype = ctypes.c_size_t
        lib.dsa3d_status_string.argtypes = [ctypes.c_int]
        lib.dsa3d_status_string.restype = ctypes.c_char_p
        lib.dsa3d_abi_version.argtypes = []
        lib.dsa3d_abi_version.restype = ctypes.c_int
        _lib = lib
    return _lib


def make_desc(B, T, H, W, heads, head_dim, kt, kh, kw, dtype="bf16", scale=0.0) -> dsa3d_desc:
    return dsa3d_desc(B, T, H, W, heads, head_dim, kt, kh, kw, float(scale),
                      DSA3D_BF16 if dtype == "bf16" else DSA3D_F32)


def _ptr(x):
    """Device pointer of a tensor (or an int address, or None for NULL)."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def status_string(status: int) -> str:
    return load().dsa3d_status_string(status).decode()


def dsa3d_abi_version() -> int:
    return load().dsa3d_abi_version()


def dsa3d_backward_workspace_size(desc: dsa3d_desc) -> int:
    return load().dsa3d_backward_workspace_size(ctypes.byref(desc))


def dsa3d_forward(desc, q, k, v, offsets, out, lse=None, stream=None, check=True) -> int:
    st = load().dsa3d_forward(ctypes.byref(desc) if desc is not None else None, _ptr(q), _ptr(k),
                              _ptr(v), _ptr(offsets), _ptr(out), _ptr(lse), _stream(stream))
    if check and st != DSA3D_OK:
        raise Dsa3dError(st, "dsa3d_forward")
    return st


def dsa3d_backward(desc, q, k, v, offsets, out, lse, dout, dq, dk, dv, d_offsets,
                   workspace=None, workspace_bytes=0, stream=None, check=True) -> int:
    """`out` (the forward's output) may be None: the library does not read it."""
    st = load().dsa3d_backward(ctypes.byref(desc) if desc is not None else None, _ptr(q), _ptr(k),
                               _ptr(v), _ptr(offsets), _ptr(out), _ptr(lse), _ptr(dout),
                               _ptr(dq), _ptr(dk), _ptr(dv), _ptr(d_offsets), _ptr(workspace),
                               workspace_bytes, _stream(stream))
    if check and st != DSA3D_OK:
        raise Dsa3dError(st, "dsa3d_backward")
    return st


def dsa3d_backward_timed(desc, q, k, v, offsets, out, lse, dout, dq, dk, dv, d_offsets,
                         workspace=None, workspace_bytes=0, stream=None, events=None,
                         check=True) -> int:
    """`events`: None or DSA3D_BACKWARD_PHASES + 1 torch.cuda.Event objects (or raw hipEvent_t
    addresses); each must already be created, i.e. recorded once."""
    arr = _event_array(events)
    st = load().dsa3d_backward_timed(ctypes.byref(desc) if desc is not None else None, _ptr(q),
                                     _ptr(k), _ptr(v), _ptr(offsets), _ptr(out), _ptr(lse),
                                     _ptr(dout), _ptr(dq), _ptr(dk), _ptr(dv), _ptr(d_offsets),
                                     _ptr(workspace), workspace_bytes, _stream(stream), arr)
    if check and st != DSA3D_OK:
        raise Dsa3dError(st, "dsa3d_backward_timed")
    return st


def dsa3d_backward_noalloc(desc, q, k, v, offsets, out, lse, dout, dq, dk, dv, d_offsets,
                           stream=None, check=True) -> int:
    """dsa3d_backward in the library's fixed scratch buffer (no workspace, no allocation)."""
    st = load().dsa3d_backward_noalloc(ctypes.byref(desc) if desc is not None else None, _ptr(q),
                                       _ptr(k), _ptr(v), _ptr(offsets), _ptr(out), _ptr(lse),
                                       _ptr(dout), _ptr(dq), _ptr(dk), _ptr(dv), _ptr(d_offsets),
                                       _stream(stream))
    if check and st != DSA3D_OK:
        raise Dsa3dError(st, "dsa3d_backward_noalloc")
    return st


def dsa3d_pw_forward(desc, logits, v, offsets, out, lse=None, stream=None, check=True) -> int:
    st = load().dsa3d_pw_forward(ctypes.byref(desc) if desc is not None else None, _ptr(logits),
                                 _ptr(v), _ptr(offsets), _ptr(out), _ptr(lse), _stream(stream))
    if check and st != DSA3D_OK:
        raise Dsa3dError(st, "dsa3d_pw_forward")
    return st


def dsa3d_pw_backward_workspace_size(desc) -> int:
    return load().dsa3d_pw_backward_workspace_size(ctypes.byref(desc))


def _event_array(events, phases=DSA3D_BACKWARD_PHASES):
    """None, or a ctypes array of phases + 1 created event handles."""
    if events is None:
        return None
    handles = [e if isinstance(e, int) else e.cuda_event for e in events]
    if len(handles) != phases + 1 or not all(handles):
        raise ValueError(f"phase timing needs {phases} + 1 created events")
    return (ctypes.c_void_p * len(handles))(*handles)


def dsa3d_pw_backward(desc, logits, v, offsets, lse, dout, dlogits, dv, d_offsets, workspace=None,
                      workspace_bytes=0, stream=None, events=None, check=True) -> int:
    st = load().dsa3d_pw_backward(ctypes.byref(desc) if desc is not None else None, _ptr(logits),
                                  _ptr(v), _ptr(offsets), _ptr(lse), _ptr(dout), _ptr(dlogits),
                                  _ptr(dv), _ptr(d_offsets), _ptr(workspace), workspace_bytes,
                                  _stream(stream), _event_array(events))
    if check and st != DSA3D_OK:
        raise Dsa3dError(st, "dsa3d_pw_backward")
    return st


def make_conv_desc(B, T, H, W, C, kt, kh, kw, dtype="bf16") -> dsa3d_dwconv_desc:
    return dsa3d_dwconv_desc(B, T, H, W, C, kt, kh, kw,
                             DSA3D_BF16 if dtype == "bf16" else DSA3D_F32)


def dsa3d_dwconv3d_forward(desc, x, weight, bias, y, accumulate=False, stream=None,
                           check=True) -> int:
    st = load().dsa3d_dwconv3d_forward(ctypes.byref(desc) if desc is not None else None, _ptr(x),
                                       _ptr(weight), _ptr(bias), _ptr(y), int(bool(accumulate)),
                                       _stream(stream))
    if check and st != DSA3D_OK:
        raise Dsa3dError(st, "dsa3d_dwconv3d_forward")
    return st


def dsa3d_dwconv3d_backward_workspace_size(desc) -> int:
    return load().dsa3d_dwconv3d_backward_workspace_size(ctypes.byref(desc))


def dsa3d_dwconv3d_backward(desc, x, weight, dy, dx, dweight, dbias, workspace=None,
                            workspace_bytes=0, accumulate_dx=False, stream=None,
                            check=True) -> int:
    st = load().dsa3d_dwconv3d_backward(ctypes.byref(desc) if desc is not None else None, _ptr(x),
                                        _ptr(weight), _ptr(dy), _ptr(dx),
                                        int(bool(accumulate_dx)), _ptr(dweight), _ptr(dbias),
                                        _ptr(workspace), workspace_bytes, _stream(stream))
    if check and st != DSA3D_OK:
        raise Dsa3dError(st, "dsa3d_dwconv3d_backward")
    return st


def make_win_desc(B, T, H, W, heads, head_dim, window, shift=(0, 0, 0), dtype="bf16",
                  scale=0.0) -> dsa3d_win_desc:
    return dsa3d_win_desc(B, T, H, W, heads, head_dim, *window, *shift, float(scale),
                          DSA3D_BF16 if dtype == "bf16" else DSA3D_F32)


def dsa3d_win_forward(desc, q, k, v, out, out_res=None, lse=None, stream=None,
                      check=True) -> int:
    st = load().dsa3d_win_forward(ctypes.byref(desc) if desc is not None else None, _ptr(q),
                                  _ptr(k), _ptr(v), _ptr(out), _ptr(out_res), _ptr(lse),
                                  _stream(stream))
    if check and st != DSA3D_OK:
        raise Dsa3dError(st, "dsa3d_win_forward")
    return st


def dsa3d_win_backward_workspace_size(desc) -> int:
    return load().dsa3d_win_backward_workspace_size(ctypes.byref(desc))


def dsa3d_win_backward(desc, q, k, v, out, out_res, lse, dout, dq, dk, dv, workspace=None,
                       workspace_bytes=0, stream=None, events=None, check=True) -> int:
    st = load().dsa3d_win_backward(ctypes.byref(desc) if desc is not None else None, _ptr(q),
                                   _ptr(k), _ptr(v), _ptr(out), _ptr(out_res), _ptr(lse),
                                   _ptr(dout), _ptr(dq),
                                   _ptr(dk), _ptr(dv), _ptr(workspace), workspace_bytes,
                                   _stream(stream),
                                   _event_array(events, DSA3D_WIN_BACKWARD_PHASES))
    if check and st != DSA3D_OK:
        raise Dsa3dError(st, "dsa3d_win_backward")
    return st


def default_scale(head_dim: int) -> float:
    return 1.0 / math.sqrt(head_dim)
