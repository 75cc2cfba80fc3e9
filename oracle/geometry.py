"""Shard geometry by enumeration (oracle; test infrastructure only).

Per spatial axis of extent G, odd kernel K, stride S and "same" zero padding
P = (K - 1) // 2, output j reads inputs j*S - P + t for t in [0, K)
(PyTorch's convolution semantics, which the paper's application programming
model keeps: section "Benchmarks and Applications", Algorithm 1 step 4).

A shard of the input owns the contiguous input range [o, o + L) (its sharding
shape along that axis; per-rank sizes are arbitrary, section "ShardTensor",
Table 2). Because a convolution changes the global shape, output chunks are
uneven (section "ShardTensor"); the reading used here is the anchor rule:
output j belongs to the shard whose input range contains j*S. The halo is the
set of input rows outside [o, o + L) that the owned outputs read (section
"PyTorch Dispatch": the convolution fetches adjacent pixels from neighbouring
devices). Everything below is found by listing outputs and taps one by one.
"""
from __future__ import annotations


def out_len(G: int, K: int, S: int) -> int:
    """Number of outputs of a 'same'-padded convolution along one axis."""
    P = (K - 1) // 2
    return (G + 2 * P - K) // S + 1


def owned_outputs(G: int, K: int, S: int, o: int, L: int) -> list:
    """Outputs j whose anchor input j*S lies in [o, o + L), listed one by one."""
    return [j for j in range(out_len(G, K, S)) if o <= j * S < o + L]


def axis_geometry(G: int, K: int, S: int, o: int, L: int, sharded: bool = True) -> dict:
    """Geometry of one axis of one shard, by enumeration.

    Returns out_off/out_ext (owned output range), halo_lo/halo_hi (margin rows
    of the padded tile; rows outside [0, G) are zero padding) and pad_lo (tile
    row of output 0's tap 0 is ``-pad_lo``; negative on a sharded axis means
    leading interior rows are never read).
    """
    if K < 1 or K % 2 == 0 or S < 1 or G < 1:
        raise ValueError("odd K >= 1, S >= 1, G >= 1 required")
    P = (K - 1) // 2
    n_out = out_len(G, K, S)
    if not sharded:
        return dict(out_off=0, out_ext=n_out, halo_lo=0, halo_hi=0, pad_lo=P)
    mine = owned_outputs(G, K, S, o, L)
    if not mine:
        before = len([j for j in range(n_out) if j * S < o])
        return dict(out_off=before, out_ext=0, halo_lo=0, halo_hi=0, pad_lo=0)
    if mine != list(range(mine[0], mine[-1] + 1)):
        raise AssertionError("owned outputs not contiguous")
    needed = [j * S - P + t for j in mine for t in range(K)]
    lo_need, hi_need = min(needed), max(needed)
    r_lo = o - lo_need
    r_hi = hi_need - (o + L - 1)
    return dict(out_off=mine[0], out_ext=len(mine), halo_lo=max(0, r_lo), halo_hi=max(0, r_hi),
                pad_lo=min(0, r_lo))


def shard_geometry(global_ext, shard_off, shard_ext, kernel, stride, sharded) -> dict:
    """Per-axis geometry of one shard; every argument is a per-axis sequence."""
    per_axis = [axis_geometry(G, K, S, o, L, bool(m))
                for G, o, L, K, S, m in zip(global_ext, shard_off, shard_ext, kernel, stride, sharded)]
    return {k: [a[k] for a in per_axis] for k in per_axis[0]}


def chunk_sizes(G: int, parts: int) -> list:
    """Default split: torch.chunk sizing, ceil(G / parts) per chunk, last ones short
    (the even distribution DTensor assumes, section "ShardTensor")."""
    c = -(-G // parts)
    sizes = []
    left = G
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


def interior_outputs(lo: int, ext: int, hi: int, K: int, S: int, pad_lo: int, n_out: int) -> list:
    """Outputs j along one axis of a padded tile (margins lo and hi around ext
    interior rows) that read no margin row: every input row j*S - pad_lo + t,
    t < K, lies in the interior [lo, lo + ext) on each side that has a margin
    (an axis without margins: every output). They depend on no halo, so they can
    be computed while the exchange (section "PyTorch Dispatch") is in flight,
    the communication/computation overlap the paper lists as missing (section
    "Limitations"). Listed one by one."""
    out = []
    for j in range(n_out):
        rows = [j * S - pad_lo + t for t in range(K)]
        if lo > 0 and min(rows) < lo:
            continue
        if hi > 0 and max(rows) >= lo + ext:
            continue
        out.append(j)
    return out
