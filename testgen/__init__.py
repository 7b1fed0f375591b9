"""Seeded synthetic inputs for the 3D-DSA parity tests and the bench.

Test infrastructure shared by the oracle side and the GPU side: it only draws
random numbers (counter-based Philox4x32-10, see ``testgen.c``) and holds none
of the operator's arithmetic.  The workload table below gives the shapes and
value distributions of the synthetic video-token grids used throughout.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "testgen.c")
_LIB = os.path.join(_HERE, "libtestgen.so")

# Tensor ids (part of the counter); fixed so every slab is reproducible.
TID_Q, TID_K, TID_V, TID_OFF, TID_DOUT, TID_LOGITS = 0, 1, 2, 3, 4, 5

NORMAL, UNIFORM = 0, 1


def build(force: bool = True) -> str:
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O3", "-fopenmp", "-shared", "-fPIC", "-std=c11",
                               _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        lib = ctypes.CDLL(_LIB)
        lib.tg_fill.argtypes = [ctypes.c_uint64, ctypes.c_uint32, ctypes.c_uint64, ctypes.c_uint64,
                                ctypes.c_int, ctypes.c_double, ctypes.c_double, ctypes.c_double,
                                ctypes.c_double, ctypes.c_int, ctypes.c_void_p]
        lib.tg_fill.restype = None
        lib.tg_philox4x32_10.argtypes = [ctypes.POINTER(ctypes.c_uint32)] * 3
        lib.tg_philox4x32_10.restype = None
        lib.tg_f32_to_bf16.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_uint64]
        lib.tg_f32_to_bf16.restype = None
        _lib = lib
    return _lib


def philox4x32_10(ctr, key):
    lib = _load()
    c = (ctypes.c_uint32 * 4)(*ctr)
    k = (ctypes.c_uint32 * 2)(*key)
    o = (ctypes.c_uint32 * 4)()
    lib.tg_philox4x32_10(c, k, o)
    return list(o)


@dataclasses.dataclass(frozen=True)
class Dist:
    kind: int          # NORMAL or UNIFORM
    a: float           # mean (normal) or low end (uniform)
    b: float           # std (normal) or high end (uniform)
    lo: float = -np.inf
    hi: float = np.inf


def fill(out: np.ndarray, seed: int, tid: int, start: int, dist: Dist) -> np.ndarray:
    """Write elements [start, start + out.size) of tensor `tid` into `out`.

    `out` must be C-contiguous float32 or uint16 (bf16 bit patterns)."""
    assert out.flags["C_CONTIGUOUS"]
    if out.dtype == np.float32:
        bf16 = 0
    elif out.dtype == np.uint16:
        bf16 = 1
    else:
        raise TypeError("fill: out must be float32 or uint16 (bf16 bits)")
    _load().tg_fill(seed, tid, start, out.size, dist.kind, dist.a, dist.b, dist.lo, dist.hi, bf16,
                    out.ctypes.data)
    return out


def f32_to_bf16(x: np.ndarray) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty(x.shape, dtype=np.uint16)
    _load().tg_f32_to_bf16(x.ctypes.data, out.ctypes.data, x.size)
    return out


def bf16_to_f32(x: np.ndarray) -> np.ndarray:
    return (x.astype(np.uint32) << 16).view(np.float32)


@dataclasses.dataclass(frozen=True)
class Workload:
    """A synthetic 3D-DSA problem: grid, heads, kernel, dtype and distributions."""
    name: str
    B: int
    T: int
    H: int
    W: int
    heads: int
    head_dim: int
    kt: int
    kh: int
    kw: int
    dtype: str                 # "f32" or "bf16" for q, k, v, out, dout
    qkv: Dist
    offsets: Dist
    seed: int
    backward: bool
    dout: Dist = Dist(NORMAL, 0.0, 1.0)

    @property
    def N(self):
        return self.T * self.H * self.W

    @property
    def P(self):
        return self.kt * self.kh * self.kw

    @property
    def queries(self):
        """(token, head) rows."""
        return self.B * self.N * self.heads

    def qkv_shape(self):
        return (self.B, self.T, self.H, self.W, self.heads, self.head_dim)

    def off_shape(self):
        return (self.B, self.T, self.H, self.W, self.heads, self.P, 3)

    def logits_shape(self):
        return (self.B, self.T, self.H, self.W, self.heads, self.P)

    def np_io_dtype(self):
        return np.float32 if self.dtype == "f32" else np.uint16

    def with_grid(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


N01 = Dist(NORMAL, 0.0, 1.0)

WORKLOADS = {
    # 256 query tokens, fp32, zero-padded borders hit by most points.
    "tiny_f32": Workload("tiny_f32", 1, 4, 8, 8, 2, 32, 3, 3, 3, "f32", N01,
                         Dist(NORMAL, 0.0, 0.5), seed=0, backward=False),
    # 16,384 tokens, bf16 q/k/v, offsets uniform in [-2, 2].
    "medium_bf16": Workload("medium_bf16", 1, 16, 32, 32, 8, 64, 3, 3, 3, "bf16", N01,
                            Dist(UNIFORM, -2.0, 2.0), seed=1, backward=False),
    # 256 frames of a 1080p latent at patch 16: 2,088,960 tokens, 24 heads x 128.
    "full_1080p_256f": Workload("full_1080p_256f", 1, 256, 68, 120, 24, 128, 3, 3, 3, "bf16", N01,
                                Dist(NORMAL, 0.0, 1.0, -3.0, 3.0), seed=2, backward=False),
    # forward + backward, 130,560 tokens, 16 heads x 64.
    "fwdbwd_64x34x60": Workload("fwdbwd_64x34x60", 1, 64, 34, 60, 16, 64, 3, 3, 3, "bf16", N01,
                                Dist(UNIFORM, -2.0, 2.0), seed=3, backward=True),
    # forward + backward, 3x5x5 kernel (75 points), offsets uniform in [-8, 8].
    "wide_64x68x120_p75": Workload("wide_64x68x120_p75", 1, 64, 68, 120, 24, 128, 3, 5, 5, "bf16",
                                   N01, Dist(UNIFORM, -8.0, 8.0), seed=4, backward=True),
    # The paper's kernel, 3x7x7 (147 points), forward + backward on the 64-frame 1080p grid.
    "paper_3x7x7_64x68x120": Workload("paper_3x7x7_64x68x120", 1, 64, 68, 120, 24, 128, 3, 7, 7,
                                      "bf16", N01, Dist(NORMAL, 0.0, 1.0, -3.0, 3.0), seed=5,
                                      backward=True),
    # The paper's kernel on 256 frames of 1080p (2,088,960 tokens), forward.
    "paper_3x7x7_1080p_256f": Workload("paper_3x7x7_1080p_256f", 1, 256, 68, 120, 24, 128, 3, 7,
                                       7, "bf16", N01, Dist(NORMAL, 0.0, 1.0, -3.0, 3.0), seed=6,
                                       backward=False),
}


def gen_tensor(w: Workload, tid: int, shape, dist: Dist, io: bool, start: int = 0) -> np.ndarray:
    out = np.empty(shape, dtype=w.np_io_dtype() if io else np.float32)
    return fill(out, w.seed, tid, start, dist)


def gen_inputs(w: Workload, progress=None):
    """Full host copies of q, k, v (io dtype), offsets (fp32) and dout (io dtype).
    `progress`, if given, is called with a short message before each tensor."""
    def one(name, tid, shape, dist, io):
        if progress is not None:
            progress(f"generating {name} {shape} of {w.name}")
        return gen_tensor(w, tid, shape, dist, io)

    q = one("q", TID_Q, w.qkv_shape(), w.qkv, True)
    k = one("k", TID_K, w.qkv_shape(), w.qkv, True)
    v = one("v", TID_V, w.qkv_shape(), w.qkv, True)
    off = one("offsets", TID_OFF, w.off_shape(), w.offsets, False)
    dout = one("dout", TID_DOUT, w.qkv_shape(), w.dout, True) if w.backward else None
    return q, k, v, off, dout


# ----------------------------------------------------------------------------- predicted weights

# Logits of the predicted-weights variant (the output of a linear layer): N(0, 1.5^2), so that
# the softmax over the points is neither flat nor one-hot.
PW_LOGITS = Dist(NORMAL, 0.0, 1.5)


def gen_pw_inputs(w: Workload, progress=None):
    """Host copies for the predicted-weights variant: logits (fp32), v (io dtype), offsets
    (fp32) and dout (io dtype); v, offsets and dout are the tensors gen_inputs draws."""
    def one(name, tid, shape, dist, io):
        if progress is not None:
            progress(f"generating {name} {shape} of {w.name}")
        return gen_tensor(w, tid, shape, dist, io)

    logits = one("logits", TID_LOGITS, w.logits_shape(), PW_LOGITS, False)
    v = one("v", TID_V, w.qkv_shape(), w.qkv, True)
    off = one("offsets", TID_OFF, w.off_shape(), w.offsets, False)
    dout = one("dout", TID_DOUT, w.qkv_shape(), w.dout, True)
    return logits, v, off, dout


PW_WORKLOADS = {
    # forward + backward of the predicted-weights variant on the forward + backward grid
    "pw_64x34x60": Workload("pw_64x34x60", 1, 64, 34, 60, 16, 64, 3, 3, 3, "bf16", N01,
                            Dist(UNIFORM, -2.0, 2.0), seed=7, backward=True),
}


# ----------------------------------------------------------------------------- depthwise conv

TID_CONV_X, TID_CONV_DY, TID_CONV_W, TID_CONV_B = 10, 11, 12, 13


@dataclasses.dataclass(frozen=True)
class ConvWorkload:
    """A synthetic depthwise 3D convolution problem: x and dy ~ N(0, 1) on a T x H x W grid of
    C channels, weights N(0, 1/taps) (the scale of a fan-in initialisation), bias N(0, 0.1)."""
    name: str
    B: int
    T: int
    H: int
    W: int
    C: int
    kt: int
    kh: int
    kw: int
    dtype: str
    seed: int

    @property
    def taps(self):
        return self.kt * self.kh * self.kw

    @property
    def tokens(self):
        return self.B * self.T * self.H * self.W

    def shape8(self):
        return (self.B, self.T, self.H, self.W, self.C, self.kt, self.kh, self.kw)

    def x_shape(self):
        return (self.B, self.T, self.H, self.W, self.C)

    def np_io_dtype(self):
        return np.float32 if self.dtype == "f32" else np.uint16

    def with_grid(self, **kw) -> "ConvWorkload":
        return dataclasses.replace(self, **kw)


def gen_conv_inputs(w: ConvWorkload, progress=None):
    """Host copies of x, dy (io dtype), weight [C,kt,kh,kw] and bias [C] (float32)."""
    def one(name, tid, shape, dist, io):
        if progress is not None:
            progress(f"generating {name} {shape} of {w.name}")
        out = np.empty(shape, dtype=w.np_io_dtype() if io else np.float32)
        return fill(out, w.seed, tid, 0, dist)

    x = one("x", TID_CONV_X, w.x_shape(), N01, True)
    dy = one("dy", TID_CONV_DY, w.x_shape(), N01, True)
    wt = one("weight", TID_CONV_W, (w.C, w.kt, w.kh, w.kw), Dist(NORMAL, 0.0, w.taps ** -0.5),
             False)
    bias = one("bias", TID_CONV_B, (w.C,), Dist(NORMAL, 0.0, 0.1), False)
    return x, dy, wt, bias


CONV_WORKLOADS = {
    # The DWConv3D term on 256 frames of 1080p: 2,088,960 tokens x 3072 channels (24 x 128).
    "dwconv_1080p_256f": ConvWorkload("dwconv_1080p_256f", 1, 256, 68, 120, 3072, 3, 3, 3, "bf16",
                                      seed=20),
    # The same term on the forward + backward grid: 130,560 tokens x 1024 channels (16 x 64).
    "dwconv_64x34x60": ConvWorkload("dwconv_64x34x60", 1, 64, 34, 60, 1024, 3, 3, 3, "bf16",
                                    seed=21),
}


# ----------------------------------------------------------------------------- window attention

TID_WIN_Q, TID_WIN_K, TID_WIN_V, TID_WIN_DOUT = 30, 31, 32, 33


@dataclasses.dataclass(frozen=True)
class WinWorkload:
    """A synthetic fixed / shifted window attention problem: bf16 q, k, v and dout ~ N(0, 1)
    on a T x H x W grid, windows of wt x wh x ww tokens, cyclic shift (st, sh, sw)."""
    name: str
    B: int
    T: int
    H: int
    W: int
    heads: int
    head_dim: int
    window: tuple
    shift: tuple
    seed: int
    dtype: str = "bf16"

    @property
    def N(self):
        return self.T * self.H * self.W

    @property
    def queries(self):
        return self.B * self.N * self.heads

    def shape12(self):
        return (self.B, self.T, self.H, self.W, self.heads, self.head_dim) + tuple(self.window) + \
            tuple(self.shift)

    def qkv_shape(self):
        return (self.B, self.T, self.H, self.W, self.heads, self.head_dim)

    def with_grid(self, **kw) -> "WinWorkload":
        return dataclasses.replace(self, **kw)


def gen_win_inputs(w: WinWorkload, progress=None):
    """Host copies (bf16 bit patterns) of q, k, v and dout."""
    out = []
    for name, tid in (("q", TID_WIN_Q), ("k", TID_WIN_K), ("v", TID_WIN_V), ("dout", TID_WIN_DOUT)):
        if progress is not None:
            progress(f"generating {name} {w.qkv_shape()} of {w.name}")
        out.append(fill(np.empty(w.qkv_shape(), dtype=np.uint16), w.seed, tid, 0, N01))
    return tuple(out)


WIN_WORKLOADS = {
    # Swin-DiT's attention (Section 6.2): shifted 3 x 16 x 16 windows on 256 frames of 1080p,
    # 2,088,960 tokens, 24 heads x 128.
    "swin_1080p_256f": WinWorkload("swin_1080p_256f", 1, 256, 68, 120, 24, 128, (3, 16, 16),
                                   (1, 8, 8), seed=30),
    # The same windows on the forward + backward grid: 130,560 tokens, 16 heads x 64.
    "swin_64x34x60": WinWorkload("swin_64x34x60", 1, 64, 34, 60, 16, 64, (3, 16, 16), (1, 8, 8),
                                 seed=31),
}
