"""Halo slabs of a padded tile (oracle; test infrastructure only).

The convolution on a shard fetches the adjacent rows from its neighbours
(section "PyTorch Dispatch", the "halo" operation). Reading used here for a
tile sharded along several axes: the axes are exchanged one after another in
ascending order, so the slab sent along axis a spans the *padded* extent on
every earlier axis (whose margins were already filled, which carries the
corner values) and the *interior* extent on every later axis.

Tile layout for these helpers: logical [N][C][*spatial] float64, the spatial
extents being halo_lo + ext + halo_hi per axis.
"""
from __future__ import annotations

import numpy as np


def _span(a, axis, halo_lo, ext, halo_hi):
    if a < axis:
        return 0, halo_lo[a] + ext[a] + halo_hi[a]
    return halo_lo[a], halo_lo[a] + ext[a]


def face_box(axis, rows, halo_lo, ext, halo_hi):
    """Spatial box (tile coordinates) of a face: ``rows`` = (r0, r1) on ``axis``."""
    lo, hi = [], []
    for a in range(len(ext)):
        if a == axis:
            lo.append(rows[0])
            hi.append(rows[1])
        else:
            s0, s1 = _span(a, axis, halo_lo, ext, halo_hi)
            lo.append(s0)
            hi.append(s1)
    return lo, hi


def pack_rows(axis, side, width, halo_lo, ext):
    """Interior rows a shard sends to its neighbour on ``side`` (0 low, 1 high)."""
    if side == 0:
        return halo_lo[axis], halo_lo[axis] + width
    return halo_lo[axis] + ext[axis] - width, halo_lo[axis] + ext[axis]


def margin_rows(axis, side, halo_lo, ext, halo_hi):
    """Margin rows a shard receives on ``side``."""
    if side == 0:
        return 0, halo_lo[axis]
    return halo_lo[axis] + ext[axis], halo_lo[axis] + ext[axis] + halo_hi[axis]


def _cut(tile, lo, hi):
    sl = (slice(None), slice(None)) + tuple(slice(l, h) for l, h in zip(lo, hi))
    return tile[sl]


def pack(tile, axis, side, width, halo_lo, ext, halo_hi) -> np.ndarray:
    """The slab sent along ``axis`` to the neighbour on ``side``."""
    lo, hi = face_box(axis, pack_rows(axis, side, width, halo_lo, ext), halo_lo, ext, halo_hi)
    return np.array(_cut(tile, lo, hi), copy=True)


def unpack(tile, axis, side, slab, halo_lo, ext, halo_hi) -> np.ndarray:
    """Copy of ``tile`` with the margin on (axis, side) set to ``slab`` (None: zeros)."""
    lo, hi = face_box(axis, margin_rows(axis, side, halo_lo, ext, halo_hi), halo_lo, ext, halo_hi)
    out = np.array(tile, copy=True)
    sl = (slice(None), slice(None)) + tuple(slice(l, h) for l, h in zip(lo, hi))
    out[sl] = 0.0 if slab is None else slab
    return out


def received_slab(x, axis, side, shard_off, halo_lo, ext, halo_hi) -> np.ndarray:
    """The slab the neighbour on ``side`` sends along ``axis``, cut from the
    zero-extended full domain x (logical [N][C][*spatial]): the margin box of
    this shard expressed in global coordinates."""
    from .conv import zero_extend
    lo, hi = face_box(axis, margin_rows(axis, side, halo_lo, ext, halo_hi), halo_lo, ext, halo_hi)
    glo = [shard_off[a] - halo_lo[a] + lo[a] for a in range(len(ext))]
    ghi = [shard_off[a] - halo_lo[a] + hi[a] for a in range(len(ext))]
    return zero_extend(x, glo, ghi)


def slab_shape(n, c, axis, width, halo_lo, ext, halo_hi):
    """Logical [N][C][*spatial] shape of a slab of the given width."""
    shp = [n, c]
    for a in range(len(ext)):
        if a == axis:
            shp.append(width)
        else:
            s0, s1 = _span(a, axis, halo_lo, ext, halo_hi)
            shp.append(s1 - s0)
    return shp


# --- the reverse exchange of the backward pass -----------------------------
#
# The halo exchange copies a neighbour's interior rows into a shard's margin;
# its derivative (the reading taken here of how gradients flow back through the
# exchange) adds the gradient that lands on a margin back onto the rows it was
# copied from. With the forward exchange in ascending axis order, the reverse
# runs in descending axis order over the same boxes: a shard sends the gradient
# on its margin (the box ``unpack`` wrote) and the neighbour adds the slab into
# the interior face rows (the box ``pack`` read), which on later axes span the
# padded extent of earlier axes and so carry the corner gradients onward.


def pack_margin(tile, axis, side, halo_lo, ext, halo_hi) -> np.ndarray:
    """Slab holding the gradient on the margin (axis, side), sent to the
    neighbour it came from."""
    lo, hi = face_box(axis, margin_rows(axis, side, halo_lo, ext, halo_hi), halo_lo, ext, halo_hi)
    return np.array(_cut(tile, lo, hi), copy=True)


def accumulate(tile, axis, side, width, slab, halo_lo, ext, halo_hi, rounding=None) -> np.ndarray:
    """Copy of ``tile`` with ``slab`` added to the ``width`` interior face rows on
    (axis, side) - the rows ``pack`` sends. ``rounding`` maps the float64 sum to
    the stored values (None: exact)."""
    lo, hi = face_box(axis, pack_rows(axis, side, width, halo_lo, ext), halo_lo, ext, halo_hi)
    out = np.array(tile, dtype=np.float64, copy=True)
    sl = (slice(None), slice(None)) + tuple(slice(l, h) for l, h in zip(lo, hi))
    s = out[sl] + np.asarray(slab, dtype=np.float64)
    out[sl] = s if rounding is None else rounding(s)
    return out
