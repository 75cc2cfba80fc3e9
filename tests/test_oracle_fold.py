"""Oracle pins for the interior / boundary split of a halo-padded convolution:
the outputs that read no margin row (oracle.geometry.interior_outputs).

Pinned by hand-derived ranges of the measured workloads, the degenerate cases,
and independently by the convolution itself: with every margin row set to a
huge value, exactly the interior outputs of tile_conv stay small.
"""
import itertools

import numpy as np
import pytest

from oracle import conv, geometry


@pytest.mark.parametrize("case", [
    # (lo, ext, hi, K, S, pad_lo, n_out) -> expected interior outputs
    # D axis of the 3D 512^3 shard 1 of 4: output j reads padded rows j..j+2
    ((1, 128, 1, 3, 1, 0, 128), list(range(1, 127))),
    # D axis of the strided shard 3 of 8 (lo 1, hi 0): j reads 2j..2j+2 >= 1
    ((1, 48, 0, 3, 2, 0, 24), list(range(1, 24))),
    # D and H of the corner shard of the 5^3 workload: zero-filled lo margin of 2
    ((2, 128, 2, 5, 1, 0, 128), list(range(2, 126))),
    # unsharded axis (pad 1, no margins): every output
    ((0, 64, 0, 3, 1, 1, 64), list(range(64))),
    # interior thinner than the kernel: nothing
    ((1, 1, 1, 3, 1, 0, 1), []),
    # margin on one side only
    ((0, 10, 2, 5, 1, 0, 8), list(range(0, 6))),
])
def test_hand_worked_interiors(case):
    args, want = case
    assert geometry.interior_outputs(*args) == want


def _random_axes(rng, count):
    for _ in range(count):
        G = int(rng.integers(4, 40))
        K = int(rng.choice([1, 3, 5, 7]))
        S = int(rng.integers(1, 4))
        parts = int(rng.integers(1, 5))
        sizes = geometry.chunk_sizes(G, parts)
        s = int(rng.integers(0, len(sizes)))
        o = geometry.offsets(sizes)[s]
        g = geometry.axis_geometry(G, K, S, o, sizes[s], parts > 1)
        yield g, sizes[s], K, S


def test_interior_is_where_no_margin_reaches_the_output():
    """tile_conv on a 1-D tile whose margins hold 1e300 and interior 1: an output
    stays below 1e200 exactly when it reads no margin row."""
    rng = np.random.default_rng(11)
    for g, L, K, S in _random_axes(rng, 300):
        lo, hi, n_out = g["halo_lo"], g["halo_hi"], g["out_ext"]
        tile = np.ones((1, 1, lo + L + hi))
        tile[..., :lo] = 1e300
        tile[..., lo + L:] = 1e300
        y = conv.tile_conv(tile, np.ones((1, 1, K)), (S,), (g["pad_lo"],), (n_out,))[0, 0]
        small = [j for j in range(n_out) if abs(y[j]) < 1e200]
        assert geometry.interior_outputs(lo, L, hi, K, S, g["pad_lo"], n_out) == small, (g, L, K, S)


def test_interior_is_a_contiguous_range():
    rng = np.random.default_rng(12)
    for g, L, K, S in _random_axes(rng, 300):
        got = geometry.interior_outputs(g["halo_lo"], L, g["halo_hi"], K, S, g["pad_lo"], g["out_ext"])
        assert got == list(range(got[0], got[-1] + 1)) if got else True


def test_interior_box_is_the_product_of_axes_in_3d():
    """3-D: the outputs untouched by huge margins are the product of the per-axis
    interior ranges (a corner output is boundary when any axis is)."""
    ext, lo, hi, K = (5, 6, 7), (1, 2, 0), (1, 0, 0), (3, 5, 3)
    tile = np.ones((1, 1) + tuple(l + e + h for l, e, h in zip(lo, ext, hi)))
    for a in range(3):
        idx = [slice(None)] * 5
        idx[2 + a] = slice(0, lo[a])
        tile[tuple(idx)] = 1e300
        idx[2 + a] = slice(lo[a] + ext[a], None)
        tile[tuple(idx)] = 1e300
    pad = (0, 0, 1)
    out = tuple(e + l + h - k + 1 + 2 * p if p else e + l + h - k + 1 for e, l, h, k, p in zip(ext, lo, hi, K, pad))
    y = conv.tile_conv(tile, np.ones((1, 1) + K), (1, 1, 1), pad, out)[0, 0]
    per_axis = [geometry.interior_outputs(lo[a], ext[a], hi[a], K[a], 1, pad[a], out[a]) for a in range(3)]
    want = np.zeros(out, dtype=bool)
    for j in itertools.product(*per_axis):
        want[j] = True
    assert np.array_equal(np.abs(y) < 1e200, want)
