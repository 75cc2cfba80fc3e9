"""Seeded synthetic inputs for the shard halo-convolution workloads.

A thin ctypes wrapper over ``synth.c``. This module draws values only: it has
no halo, geometry or convolution arithmetic, and is the single source of input
data for both the CPU oracle and the GPU path.

Logical tensors follow PyTorch's [N][C][*spatial] order (the paper's
[B, C, H, W, D] data layout, section "Introduction"); the returned buffers are
dense channels-last boxes [n][x0][x1][x2][c], matching the GPU tile layout.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "synth.c")
_LIB_PATH = os.path.join(_HERE, "libsynth.so")

UNIFORM, NORMAL, SMOOTH, INT, SPARSE_INT = 0, 1, 2, 3, 4
OUT_F64, OUT_F32, OUT_BF16 = 0, 1, 2
STREAM_X, STREAM_W, STREAM_DY = 0, 1, 2


class _Spec(ctypes.Structure):
    _fields_ = [
        ("seed", ctypes.c_uint64),
        ("stream", ctypes.c_int32),
        ("dist", ctypes.c_int32),
        ("p0", ctypes.c_double),
        ("p1", ctypes.c_double),
        ("p2", ctypes.c_double),
        ("ndim", ctypes.c_int32),
        ("pad_", ctypes.c_int32),
        ("full", ctypes.c_int64 * 5),
    ]


def build() -> str:
    """Compile the generator with gcc (always recompiles)."""
    cmd = ["gcc", "-O2", "-fopenmp", "-ffp-contract=off", "-fPIC", "-shared",
           _SRC, "-o", _LIB_PATH + ".tmp", "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(_LIB_PATH + ".tmp", _LIB_PATH)
    return _LIB_PATH


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build()
        lib = ctypes.CDLL(_LIB_PATH)
        lib.synth_fill.argtypes = [ctypes.POINTER(_Spec), ctypes.POINTER(ctypes.c_int64),
                                   ctypes.POINTER(ctypes.c_int64), ctypes.c_int, ctypes.c_void_p]
        lib.synth_fill.restype = ctypes.c_int
        lib.synth_round_bf16.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64]
        lib.synth_round_bf16.restype = None
        lib.synth_threads.restype = ctypes.c_int
        _lib = lib
    return _lib


@dataclass(frozen=True)
class Field:
    """One logical full-domain tensor: its shape, distribution and stream.

    ``shape`` is (N, C, *spatial) with 1..3 spatial axes.
    ``params`` are (p0, p1, p2): UNIFORM (lo, hi), NORMAL (mean, std),
    SMOOTH (unused, std, sigma), INT (lo, hi), SPARSE_INT (lo, hi, density).
    """
    shape: tuple
    dist: int
    params: tuple = (0.0, 1.0, 0.0)
    stream: int = STREAM_X
    seed: int = 0

    @property
    def ndim(self) -> int:
        return len(self.shape) - 2

    def _spec(self) -> _Spec:
        nd = self.ndim
        if not 1 <= nd <= 3:
            raise ValueError("1..3 spatial axes supported")
        full = [1, 1, 1, 1, 1]
        full[0], full[1] = self.shape[0], self.shape[1]
        for k, g in enumerate(self.shape[2:]):
            full[2 + (3 - nd) + k] = g
        p = tuple(self.params) + (0.0,) * (3 - len(self.params))
        sp = _Spec()
        sp.seed, sp.stream, sp.dist = self.seed, self.stream, self.dist
        sp.p0, sp.p1, sp.p2 = (float(v) for v in p[:3])
        sp.ndim = nd
        for k in range(5):
            sp.full[k] = int(full[k])
        return sp

    def box(self, lo=None, hi=None, out: int = OUT_F64) -> np.ndarray:
        """Channels-last box [n][x...][c] of this tensor over [lo, hi).

        ``lo``/``hi`` are (n, c, *spatial) coordinates; spatial bounds may lie
        outside the domain, where the values are 0. Returns float64, float32 or
        uint16 (bfloat16 bit patterns) according to ``out``.
        """
        nd = self.ndim
        lo = [0] * (2 + nd) if lo is None else list(lo)
        hi = list(self.shape) if hi is None else list(hi)
        if len(lo) != 2 + nd or len(hi) != 2 + nd:
            raise ValueError("box rank mismatch")
        lo5 = [lo[0], lo[1], 0, 0, 0]
        hi5 = [hi[0], hi[1], 1, 1, 1]
        for k in range(nd):
            lo5[2 + (3 - nd) + k] = lo[2 + k]
            hi5[2 + (3 - nd) + k] = hi[2 + k]
        shape = [hi[0] - lo[0]] + [hi[2 + k] - lo[2 + k] for k in range(nd)] + [hi[1] - lo[1]]
        dt = {OUT_F64: np.float64, OUT_F32: np.float32, OUT_BF16: np.uint16}[out]
        arr = np.empty(shape, dtype=dt)
        L = ctypes.c_int64 * 5
        rc = _load().synth_fill(ctypes.byref(self._spec()), L(*lo5), L(*hi5), out,
                                arr.ctypes.data_as(ctypes.c_void_p))
        if rc != 0:
            raise RuntimeError("synth_fill failed")
        return arr


def round_bf16(values: np.ndarray) -> np.ndarray:
    """binary32 -> bfloat16 bits, round-to-nearest-even (the generator's rule)."""
    v = np.ascontiguousarray(values, dtype=np.float32)
    out = np.empty(v.shape, dtype=np.uint16)
    _load().synth_round_bf16(v.ctypes.data_as(ctypes.c_void_p), out.ctypes.data_as(ctypes.c_void_p), v.size)
    return out


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns -> exact float64 values."""
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def threads() -> int:
    return int(_load().synth_threads())
