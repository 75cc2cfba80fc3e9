"""Full-domain convolution, its weight gradient, and the zero-extended input box
(oracle; test infrastructure only).

Definition (PyTorch cross-correlation, which the paper's programming model
keeps unchanged: section "Benchmarks and Applications", Algorithm 1 step 4;
no bias, dilation 1, groups 1, zero "same" padding P = (K - 1) // 2 per axis):

    y[n, co, j] = sum_{ci, t} w[co, ci, t] * x[n, ci, j*S - P + t]

with x taken as 0 outside the domain. The domain-parallel result on a shard is
this full-domain output restricted to the shard's owned output box (the
concatenated shard outputs equal the unsharded convolution: section
"PyTorch Dispatch", halo for numerical consistency).

The weight gradient of a shard is the same sum restricted to its owned outputs:

    dW[co, ci, t] = sum_{n, j in box} dy[n, co, j] * x[n, ci, j*S - P + t]

(the gradient of a layer's weights needs its saved input, section
"What Causes High GPU Memory Usage?", the Linear-layer gradient equations).

All arrays are float64 in logical [N][C][*spatial] order. The only library
step is ``numpy.tensordot`` over the channel axis (per tap) or over the
batch/spatial axes (weight gradient); there is no other blocking or reordering.
"""
from __future__ import annotations

import itertools

import numpy as np

from .geometry import out_len


def _check(x, w, stride):
    nd = x.ndim - 2
    if w.ndim != nd + 2 or w.shape[1] != x.shape[1] or len(stride) != nd:
        raise ValueError("shape mismatch")
    return nd


def zero_extend(x: np.ndarray, lo, hi) -> np.ndarray:
    """The zero-extended domain x restricted to the spatial box [lo, hi)
    (bounds may lie outside the domain; those entries are 0)."""
    nd = x.ndim - 2
    shape = list(x.shape[:2]) + [h - l for l, h in zip(lo, hi)]
    out = np.zeros(shape, dtype=np.float64)
    src, dst = [slice(None), slice(None)], [slice(None), slice(None)]
    for a in range(nd):
        s0, s1 = max(lo[a], 0), min(hi[a], x.shape[2 + a])
        if s1 <= s0:
            return out
        src.append(slice(s0, s1))
        dst.append(slice(s0 - lo[a], s1 - lo[a]))
    out[tuple(dst)] = x[tuple(src)]
    return out


def _window_taps(xw, origin, kernel, stride, out_lo, out_hi):
    """Yield (tap, strided view of the window holding x[j*S - P + t] for j in box)."""
    nd = len(kernel)
    for tap in itertools.product(*[range(k) for k in kernel]):
        sl = [slice(None), slice(None)]
        for a in range(nd):
            P = (kernel[a] - 1) // 2
            first = out_lo[a] * stride[a] - P + tap[a] - origin[a]
            count = out_hi[a] - out_lo[a]
            last = first + (count - 1) * stride[a] if count > 0 else first
            if count > 0 and (first < 0 or last >= xw.shape[2 + a]):
                raise ValueError("window does not cover the inputs of the output box")
            sl.append(slice(first, first + (count - 1) * stride[a] + 1 if count > 0 else first, stride[a]))
        yield tap, xw[tuple(sl)]


def _in_domain(xw, origin, G):
    """Copy of a window with entries outside the domain [0, G) set to 0 (the definition)."""
    nd = xw.ndim - 2
    lo = list(origin)
    hi = [o + s for o, s in zip(origin, xw.shape[2:])]
    mask_ok = all(l >= 0 for l in lo) and all(h <= g for h, g in zip(hi, G))
    if mask_ok:
        return xw
    out = np.array(xw, dtype=np.float64, copy=True)
    for a in range(nd):
        idx = np.arange(lo[a], hi[a])
        bad = (idx < 0) | (idx >= G[a])
        if bad.any():
            sl = [slice(None)] * xw.ndim
            sl[2 + a] = bad
            out[tuple(sl)] = 0.0
    return out


def conv_forward_window(xw, origin, G, w, stride, out_lo, out_hi) -> np.ndarray:
    """y over the output box [out_lo, out_hi), from a window xw of the zero-extended
    input whose element 0 sits at global spatial coordinates ``origin``."""
    nd = _check(xw, w, stride)
    xw = _in_domain(np.asarray(xw, dtype=np.float64), origin, G)
    kernel = w.shape[2:]
    y = np.zeros([xw.shape[0], w.shape[0]] + [h - l for l, h in zip(out_lo, out_hi)])
    if y.size == 0:
        return y
    for tap, xs in _window_taps(xw, origin, kernel, stride, out_lo, out_hi):
        wt = w[(slice(None), slice(None)) + tap]                     # [Co, Ci]
        y += np.moveaxis(np.tensordot(wt, xs, axes=([1], [1])), 0, 1)  # sum over ci
    return y


def conv_forward(x, w, stride, out_lo=None, out_hi=None) -> np.ndarray:
    """Full-domain convolution of x (the whole domain), restricted to an output box."""
    nd = _check(x, w, stride)
    G = x.shape[2:]
    kernel = w.shape[2:]
    n_out = [out_len(G[a], kernel[a], stride[a]) for a in range(nd)]
    out_lo = [0] * nd if out_lo is None else list(out_lo)
    out_hi = n_out if out_hi is None else list(out_hi)
    P = [(k - 1) // 2 for k in kernel]
    origin = [-p for p in P]
    xw = zero_extend(x, origin, [g + p for g, p in zip(G, P)])
    return conv_forward_window(xw, origin, G, w, stride, out_lo, out_hi)


def conv_wgrad_window(xw, origin, G, dy, kernel, stride, out_lo, out_hi) -> np.ndarray:
    """dW[co, ci, *t] summed over the output box [out_lo, out_hi); dy covers that box."""
    nd = len(kernel)
    xw = _in_domain(np.asarray(xw, dtype=np.float64), origin, G)
    dy = np.asarray(dy, dtype=np.float64)
    want = [h - l for l, h in zip(out_lo, out_hi)]
    if list(dy.shape[2:]) != want or dy.shape[0] != xw.shape[0]:
        raise ValueError("dy does not match the output box")
    dw = np.zeros([dy.shape[1], xw.shape[1]] + list(kernel))
    if dy.size == 0:
        return dw
    red = [0] + list(range(2, 2 + nd))
    for tap, xs in _window_taps(xw, origin, kernel, stride, out_lo, out_hi):
        dw[(slice(None), slice(None)) + tap] = np.tensordot(dy, xs, axes=(red, red))
    return dw


def conv_wgrad(x, dy, kernel, stride, out_lo=None, out_hi=None) -> np.ndarray:
    """Weight gradient over an output box, from the whole-domain input x."""
    nd = x.ndim - 2
    G = x.shape[2:]
    n_out = [out_len(G[a], kernel[a], stride[a]) for a in range(nd)]
    out_lo = [0] * nd if out_lo is None else list(out_lo)
    out_hi = n_out if out_hi is None else list(out_hi)
    P = [(k - 1) // 2 for k in kernel]
    origin = [-p for p in P]
    xw = zero_extend(x, origin, [g + p for g, p in zip(G, P)])
    return conv_wgrad_window(xw, origin, G, dy, kernel, stride, out_lo, out_hi)


def conv_dgrad(dy, w, G, stride) -> np.ndarray:
    """Full-domain input gradient: the derivative of sum(dy * conv_forward(x, w))
    with respect to x over the domain [0, G),

        dx[n, ci, i] = sum over co, t and outputs j with j*S - P + t = i of
                       w[co, ci, t] * dy[n, co, j]

    (the convolution analogue of dL/dx = dL/dz W for a Linear layer, section
    "What Causes High GPU Memory Usage?", subsection "An Example of Memory
    Usage"). dy covers the whole output. Written as a scatter: for every tap the
    outputs' contributions are added to the input rows they were read from;
    rows that fall in the zero padding are dropped."""
    dy = np.asarray(dy, dtype=np.float64)
    nd = len(G)
    kernel = w.shape[2:]
    n_out = [out_len(G[a], kernel[a], stride[a]) for a in range(nd)]
    if list(dy.shape[2:]) != n_out or dy.shape[1] != w.shape[0]:
        raise ValueError("dy does not match the full output")
    P = [(k - 1) // 2 for k in kernel]
    # accumulate into the zero-extended domain [-P, G + P), then cut the domain
    ext = [G[a] + 2 * P[a] for a in range(nd)]
    dxe = np.zeros([dy.shape[0], w.shape[1]] + ext)
    if dy.size == 0:
        return dxe[(slice(None), slice(None)) + tuple(slice(P[a], P[a] + G[a]) for a in range(nd))]
    for tap in itertools.product(*[range(k) for k in kernel]):
        wt = w[(slice(None), slice(None)) + tap]                              # [Co, Ci]
        contrib = np.moveaxis(np.tensordot(wt, dy, axes=([0], [1])), 0, 1)   # [N, Ci, *out]
        sl = [slice(None), slice(None)]
        for a in range(nd):
            # output j reads extended row j*S + t
            sl.append(slice(tap[a], tap[a] + (n_out[a] - 1) * stride[a] + 1, stride[a]))
        dxe[tuple(sl)] += contrib
    return dxe[(slice(None), slice(None)) + tuple(slice(P[a], P[a] + G[a]) for a in range(nd))]


def tile_dgrad(dy, w, stride, pad_lo, tile_ext) -> np.ndarray:
    """Input gradient read back onto a padded tile: the adjoint of ``tile_conv``.
    Output jj, tap t read tile row jj*S + t - pad_lo along each axis; its
    contribution w[co, ci, t] * dy[jj] is added to that row when the row lies in
    [0, tile_ext) and dropped otherwise (zero padding outside the tile). The
    result covers every tile row, margins included: the margin rows hold the
    gradient that belongs to the neighbours' interiors."""
    dy = np.asarray(dy, dtype=np.float64)
    nd = dy.ndim - 2
    kernel = w.shape[2:]
    out_ext = dy.shape[2:]
    dt = np.zeros([dy.shape[0], w.shape[1]] + list(tile_ext))
    if dy.size == 0:
        return dt
    for tap in itertools.product(*[range(k) for k in kernel]):
        wt = w[(slice(None), slice(None)) + tap]
        contrib = np.moveaxis(np.tensordot(wt, dy, axes=([0], [1])), 0, 1)  # [N, Ci, *out]
        src, dst = [slice(None), slice(None)], [slice(None), slice(None)]
        empty = False
        for a in range(nd):
            rows = np.arange(out_ext[a]) * stride[a] + tap[a] - pad_lo[a]
            ok = np.nonzero((rows >= 0) & (rows < tile_ext[a]))[0]
            if ok.size == 0:
                empty = True
                break
            src.append(slice(ok[0], ok[-1] + 1))
            dst.append(slice(rows[ok[0]], rows[ok[-1]] + 1, stride[a]))
        if not empty:
            dt[tuple(dst)] += contrib[tuple(src)]
    return dt


def shard_input_box(geom: dict, shard_off, shard_ext, global_ext) -> tuple:
    """Spatial box of the shard's padded tile: [o - halo_lo, o + L + halo_hi) on
    sharded axes (margins outside the domain are zero padding), the whole axis
    elsewhere (unsharded axes carry no margin)."""
    lo, hi = [], []
    for a in range(len(global_ext)):
        lo.append(shard_off[a] - geom["halo_lo"][a])
        hi.append(shard_off[a] + shard_ext[a] + geom["halo_hi"][a])
    return lo, hi


def padded_tile(x, geom: dict, shard_off, shard_ext) -> np.ndarray:
    """The shard's padded tile: the zero-extended domain over its input box."""
    lo, hi = shard_input_box(geom, shard_off, shard_ext, x.shape[2:])
    return zero_extend(x, lo, hi)


def tile_conv(tile, w, stride, pad_lo, out_ext) -> np.ndarray:
    """Convolution read directly off a padded tile: output jj, tap t reads tile row
    jj*S + t - pad_lo along each axis, zero outside the tile. This is the local
    computation each shard performs; tests check it equals the full-domain
    convolution restricted to the owned box."""
    nd = tile.ndim - 2
    kernel = w.shape[2:]
    y = np.zeros([tile.shape[0], w.shape[0]] + list(out_ext))
    if y.size == 0:
        return y
    for tap in itertools.product(*[range(k) for k in kernel]):
        idx = []
        for a in range(nd):
            rows = np.arange(out_ext[a]) * stride[a] + tap[a] - pad_lo[a]
            idx.append(rows)
        ok = [(r >= 0) & (r < tile.shape[2 + a]) for a, r in enumerate(idx)]
        xs = tile[np.ix_(range(tile.shape[0]), range(tile.shape[1]),
                         *[np.clip(r, 0, tile.shape[2 + a] - 1) for a, r in enumerate(idx)])]
        mask = np.ones(out_ext, dtype=bool)
        for a in range(nd):
            shp = [1] * nd
            shp[a] = -1
            mask = mask & ok[a].reshape(shp)
        xs = xs * mask
        wt = w[(slice(None), slice(None)) + tap]
        y += np.moveaxis(np.tensordot(wt, xs, axes=([1], [1])), 0, 1)
    return y


def round_bf16(v: np.ndarray) -> np.ndarray:
    """Output rounding of a bf16 convolution: the exact value rounded to
    binary32 (nearest even), then to bfloat16 (nearest even on the upper 16
    bits). Returns the bfloat16 bit patterns (uint16)."""
    b = np.ascontiguousarray(v, dtype=np.float64).astype(np.float32).view(np.uint32).astype(np.uint64)
    r = (b + 0x7FFF + ((b >> 16) & 1)) >> 16
    return r.astype(np.uint16)


def bf16_value(bits: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns -> exact float64 values."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)
