"""Shard workloads for the parity tests: geometry and expected values.

Workload recipes (shapes, splits, distributions) live in ``synth.workloads``;
inputs come from ``synth`` (seeded, counter-based, so any box of the full
domain is produced on its own); geometry and expected values come from
``oracle`` only. The single GPU plays every neighbour: the slabs a neighbour
would send are cut from the same seeded full-domain tensor.
"""
from __future__ import annotations

from dataclasses import dataclass, field as dc_field

import numpy as np

import synth
from synth.workloads import (C1, C2, C3, C4, C5, INT_DIST, REDUCED, WORKLOADS, Workload,  # noqa: F401
                             as_f64 as _as_f64)
from oracle import conv as oconv
from oracle import geometry as ogeo


# kernel family names of the cross-check tests -> shard_kernels_t
KERNELS = {"": 0, "tiled": 1, "generic": 2}


def torch_dtype(w: Workload):
    import torch
    return torch.float32 if w.dtype == "f32" else torch.bfloat16


def out_code(w: Workload):
    return w.out


def as_f64(arr: np.ndarray, w: Workload = None) -> np.ndarray:
    return _as_f64(arr)


def field(w: Workload, which: str, dist=None) -> synth.Field:
    if which == "x":
        return w.x_field(dist)
    if which == "w":
        return w.w_field(dist)
    if which == "dy":
        n_out = tuple(ogeo.out_len(g, k, s) for g, k, s in zip(w.G, w.K, w.S))
        return w.dy_field(n_out, dist)
    raise ValueError(which)


def to_ncdhw(cl: np.ndarray) -> np.ndarray:
    """channels-last [n][x...][c] -> logical [n][c][x...]"""
    return np.moveaxis(cl, -1, 1)


def to_cl(lg: np.ndarray) -> np.ndarray:
    return np.ascontiguousarray(np.moveaxis(lg, 1, -1))


@dataclass
class ShardGeom:
    off: list
    ext: list
    sharded: list
    g: dict
    tile_lo: list = dc_field(default_factory=list)   # global box of the padded tile
    tile_hi: list = dc_field(default_factory=list)


def shard_geom(w: Workload, idx) -> ShardGeom:
    off, ext = w.interior(idx)
    sharded = [p > 1 for p in w.parts]
    g = ogeo.shard_geometry(w.G, off, ext, w.K, w.S, sharded)
    lo = [o - h for o, h in zip(off, g["halo_lo"])]
    hi = [o + L + h for o, L, h in zip(off, ext, g["halo_hi"])]
    return ShardGeom(off, ext, sharded, g, lo, hi)


def neighbour_exists(w: Workload, idx, axis, side) -> bool:
    return w.neighbour_exists(idx, axis, side)


def x_box(w: Workload, lo, hi, out=None, dist=None) -> np.ndarray:
    """Channels-last box of the zero-extended input over spatial [lo, hi)."""
    return w.x_box(lo, hi, dist)


def interior_tile_cl(w: Workload, sg: ShardGeom, out, canary, dist=None) -> np.ndarray:
    """Padded tile with the interior filled and every margin set to ``canary``."""
    shape = [w.N] + [l + e + h for l, e, h in zip(sg.g["halo_lo"], sg.ext, sg.g["halo_hi"])] + [w.cin]
    dt = np.uint16 if out == synth.OUT_BF16 else np.float32
    tile = np.full(shape, canary, dtype=dt)
    inner = w.x_box(sg.off, [o + e for o, e in zip(sg.off, sg.ext)], dist)
    sl = (slice(None),) + tuple(slice(l, l + e) for l, e in zip(sg.g["halo_lo"], sg.ext)) + (slice(None),)
    tile[sl] = inner
    return tile


def owned_box(sg: ShardGeom):
    lo = list(sg.g["out_off"])
    hi = [o + e for o, e in zip(sg.g["out_off"], sg.g["out_ext"])]
    return lo, hi


def expected_fwd(w: Workload, sg: ShardGeom, xw64, origin, w64) -> np.ndarray:
    """Oracle forward output (channels-last, float64) of the shard's owned box."""
    lo, hi = owned_box(sg)
    return to_cl(oconv.conv_forward_window(xw64, origin, w.G, w64, w.S, lo, hi))


def expected_wgrad(w: Workload, sg: ShardGeom, xw64, origin, dy64) -> np.ndarray:
    lo, hi = owned_box(sg)
    return oconv.conv_wgrad_window(xw64, origin, w.G, dy64, w.K, w.S, lo, hi)


def norm_max_err(got: np.ndarray, ref: np.ndarray) -> float:
    """max |g - r| / max |r| (the reading of 'relative' tolerance for whole tensors)."""
    if not np.all(np.isfinite(got)):
        return float("inf")
    scale = float(np.max(np.abs(ref))) if ref.size else 0.0
    err = float(np.max(np.abs(got - ref))) if ref.size else 0.0
    return err / scale if scale > 0 else err


TOL = {"f32": 1e-5, "bf16": 2e-2}


def bf16_rne_of_f64(v: np.ndarray) -> np.ndarray:
    """Exact float64 values -> bfloat16 bits by the oracle's output rounding rule."""
    return oconv.round_bf16(v)
