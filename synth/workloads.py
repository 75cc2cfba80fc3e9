"""Synthetic shard workloads: shapes, input splits and value distributions.

Input recipes only (no halo, geometry or convolution arithmetic). The five
workloads stand in for the paper's high-resolution fields: 2D data at
4096^2 (the ViT inference benchmark's largest resolution) and 3D volumes of
10^8..10^9 points (its 3D training benchmark), split along their spatial axes
as domain parallelism does below batch size one.
"""
from __future__ import annotations

import itertools
from dataclasses import dataclass

import numpy as np

from . import (INT, NORMAL, OUT_BF16, OUT_F32, SMOOTH, STREAM_DY, STREAM_W, STREAM_X, UNIFORM, Field,
               bf16_to_f64)


def chunk_sizes(G: int, parts: int) -> list:
    """torch.chunk-style split of G rows into `parts` pieces (ceil-sized, last short)."""
    c = -(-G // parts)
    sizes, left = [], G
    while left > 0:
        sizes.append(min(c, left))
        left -= sizes[-1]
    return sizes


def offsets(sizes) -> list:
    out, acc = [], 0
    for s in sizes:
        out.append(acc)
        acc += s
    return out


@dataclass
class Workload:
    name: str
    dtype: str                 # "f32" | "bf16"
    N: int
    cin: int
    cout: int
    G: tuple                   # global spatial extents, outermost first
    parts: tuple               # shards per axis (1 = unsharded)
    K: tuple
    S: tuple
    shard: tuple               # index of the measured shard per axis
    x_dist: tuple = (NORMAL, (0.0, 1.0))
    w_dist: tuple = None       # default N(0, 1 / (prod K * cin))
    dy_dist: tuple = (NORMAL, (0.0, 1.0))
    seed: int = 0

    @property
    def nd(self):
        return len(self.G)

    def w_spec(self):
        if self.w_dist is not None:
            return self.w_dist
        fan_in = int(np.prod(self.K)) * self.cin
        return (NORMAL, (0.0, 1.0 / np.sqrt(fan_in)))

    def splits(self, a):
        sizes = chunk_sizes(self.G[a], self.parts[a])
        return list(zip(offsets(sizes), sizes))

    def shards(self):
        return list(itertools.product(*[range(len(self.splits(a))) for a in range(self.nd)]))

    def interior(self, idx):
        """(offset, extent) per axis of shard idx's interior."""
        off, ext = [], []
        for a in range(self.nd):
            o, L = self.splits(a)[idx[a]]
            off.append(o)
            ext.append(L)
        return off, ext

    def neighbour_exists(self, idx, axis, side) -> bool:
        j = idx[axis] + (1 if side else -1)
        return 0 <= j < len(self.splits(axis))

    def with_(self, **kw):
        d = dict(self.__dict__)
        d.update(kw)
        return Workload(**d)

    # --- fields -----------------------------------------------------------------
    @property
    def out(self):
        return OUT_F32 if self.dtype == "f32" else OUT_BF16

    def x_field(self, dist=None) -> Field:
        d, p = dist or self.x_dist
        return Field((self.N, self.cin) + tuple(self.G), d, p, stream=STREAM_X, seed=self.seed)

    def w_field(self, dist=None) -> Field:
        d, p = dist or self.w_spec()
        return Field((self.cout, self.cin) + tuple(self.K), d, p, stream=STREAM_W, seed=self.seed)

    def dy_field(self, out_ext_full, dist=None) -> Field:
        d, p = dist or self.dy_dist
        return Field((self.N, self.cout) + tuple(out_ext_full), d, p, stream=STREAM_DY, seed=self.seed)

    def x_box(self, lo, hi, dist=None) -> np.ndarray:
        """Channels-last box of the zero-extended input over spatial [lo, hi)."""
        return self.x_field(dist).box((0, 0, *lo), (self.N, self.cin, *hi), out=self.out)

    def weights_host(self, dist=None) -> np.ndarray:
        """Weights in PyTorch layout [co][ci][k...] (bf16 bit patterns or float32)."""
        cl = self.w_field(dist).box(out=self.out)          # [co][k...][ci]
        return np.ascontiguousarray(np.moveaxis(cl, -1, 1))


def as_f64(arr: np.ndarray) -> np.ndarray:
    return bf16_to_f64(arr) if arr.dtype == np.uint16 else arr.astype(np.float64)


C1 = Workload("c1_2d_fp32", "f32", 1, 8, 8, (64, 64), (2, 1), (3, 3), (1, 1), (0, 0),
              x_dist=(UNIFORM, (-1.0, 1.0)), w_dist=(UNIFORM, (-1.0, 1.0)), dy_dist=(UNIFORM, (-1.0, 1.0)))
C2 = Workload("c2_2d_bf16", "bf16", 1, 64, 64, (4096, 4096), (4, 1), (3, 3), (1, 1), (1, 0))
C3 = Workload("c3_3d_bf16", "bf16", 1, 32, 32, (512, 512, 512), (4, 1, 1), (3, 3, 3), (1, 1, 1), (1, 0, 0),
              x_dist=(SMOOTH, (0.0, 1.0, 4.0)))
C4 = Workload("c4_3d_bf16_k5", "bf16", 1, 16, 64, (256, 256, 256), (2, 2, 1), (5, 5, 5), (1, 1, 1), (0, 0, 0))
C5 = Workload("c5_3d_fp32_s2", "f32", 1, 64, 128, (384, 384, 384), (8, 1, 1), (3, 3, 3), (2, 2, 2), (3, 0, 0),
              x_dist=(UNIFORM, (-1.0, 1.0)), w_dist=(UNIFORM, (-1 / np.sqrt(1728), 1 / np.sqrt(1728))),
              dy_dist=(UNIFORM, (-1.0, 1.0)))
WORKLOADS = {w.name: w for w in (C1, C2, C3, C4, C5)}
SHORT = {"c1": C1, "c2": C2, "c3": C3, "c4": C4, "c5": C5}

# Reduced variants: same channels, kernels, strides and split pattern on small
# ragged domains (the oracle finishes in seconds; every shard is checked).
REDUCED = {
    "c2r": C2.with_(name="c2r", G=(70, 77)),
    "c3r": C3.with_(name="c3r", G=(24, 21, 37), x_dist=(SMOOTH, (0.0, 1.0, 2.0))),
    "c4r": C4.with_(name="c4r", G=(18, 17, 35)),
    "c5r": C5.with_(name="c5r", G=(50, 19, 41)),
    "c1": C1,
}
INT_DIST = (INT, (-2.0, 2.0))
