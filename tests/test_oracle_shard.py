"""Pins for the oracle's shard geometry, padded tiles and halo slabs (CPU only).

The central invariant of domain parallelism (section "PyTorch Dispatch": the
halo makes the sharded convolution numerically consistent with the unsharded
one; section "ShardTensor": outputs come in uneven chunks): every shard,
convolving only its own padded tile, produces exactly its slice of the
full-domain output, and the slices tile the full output.
"""
import itertools
import json
import os

import numpy as np
import pytest

from oracle import conv, geometry, halo

GOLDEN = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "worked_examples.json")))


@pytest.mark.parametrize("case", GOLDEN["geometry1d"], ids=lambda c: c["what"][:48])
def test_hand_worked_axis_geometry(case):
    g = geometry.axis_geometry(case["G"], case["K"], case["S"], case["o"], case["L"])
    for k in ("out_off", "out_ext", "halo_lo", "halo_hi", "pad_lo"):
        assert g[k] == case[k], k


@pytest.mark.parametrize("name", [k for k in GOLDEN["workload_geometry"] if not k.startswith("_")])
def test_workload_geometry(name):
    c = GOLDEN["workload_geometry"][name]
    g = geometry.shard_geometry(c["G"], c["o"], c["L"], c["K"], c["S"], c["sharded"])
    for k in ("out_off", "out_ext", "halo_lo", "halo_hi", "pad_lo"):
        assert g[k] == c[k], k


def test_owned_ranges_partition_outputs():
    """Over every split of small domains, owned output ranges are contiguous,
    disjoint, in order, and cover [0, out_len)."""
    rng = np.random.default_rng(1)
    for G in range(1, 26):
        for K in (1, 3, 5, 7):
            for S in (1, 2, 3):
                for parts in range(1, min(G, 6) + 1):
                    sizes = geometry.chunk_sizes(G, parts)
                    if rng.random() < 0.5 and G > parts:
                        cuts = np.sort(rng.choice(np.arange(1, G), size=parts - 1, replace=False))
                        sizes = list(np.diff(np.concatenate([[0], cuts, [G]])).astype(int))
                    offs = geometry.offsets(sizes)
                    nxt = 0
                    for o, L in zip(offs, sizes):
                        g = geometry.axis_geometry(G, K, S, o, L)
                        assert g["out_off"] == nxt
                        nxt += g["out_ext"]
                        assert g["halo_lo"] >= 0 and g["halo_hi"] >= 0 and g["pad_lo"] <= 0
                    assert nxt == geometry.out_len(G, K, S)


def test_halo_is_minimal_and_sufficient():
    """The margins hold exactly the rows the owned outputs read: each margin's
    outermost row is read by some tap, and no read falls outside the tile."""
    for G, K, S in itertools.product((7, 12, 13), (3, 5, 7), (1, 2, 3)):
        for sizes in (geometry.chunk_sizes(G, 3), [2, G - 5, 3]):
            for o, L in zip(geometry.offsets(sizes), sizes):
                g = geometry.axis_geometry(G, K, S, o, L)
                if g["out_ext"] == 0:
                    continue
                rows = [jj * S + t - g["pad_lo"] for jj in range(g["out_ext"]) for t in range(K)]
                size = g["halo_lo"] + L + g["halo_hi"]
                assert min(rows) >= 0 and max(rows) < size
                if g["halo_lo"] > 0:
                    assert min(rows) == 0
                if g["halo_hi"] > 0:
                    assert max(rows) == size - 1


def _splits(G, parts):
    sizes = geometry.chunk_sizes(G, parts)
    return list(zip(geometry.offsets(sizes), sizes))


CASES = [
    # (G, K, S, parts per axis, integer)
    ((16,), (3,), (1,), (3,)),
    ((19,), (5,), (2,), (4,)),
    ((12, 10), (3, 3), (1, 1), (2, 1)),
    ((13, 11), (5, 3), (1, 2), (3, 2)),
    ((10, 9, 8), (3, 3, 3), (1, 1, 1), (2, 2, 1)),
    ((12, 7, 9), (3, 3, 3), (2, 1, 2), (3, 1, 1)),
    ((9, 10, 7), (5, 5, 5), (1, 1, 1), (2, 2, 1)),
    ((11, 8, 6), (3, 5, 1), (3, 1, 1), (4, 1, 2)),
]


@pytest.mark.parametrize("case", CASES)
@pytest.mark.parametrize("integer", [True, False])
def test_shard_outputs_concatenate_to_full(case, integer):
    G, K, S, parts = case
    nd = len(G)
    rng = np.random.default_rng(sum(G) + 7 * nd)
    mk = (lambda s: rng.integers(-2, 3, size=s).astype(np.float64)) if integer else (lambda s: rng.uniform(-1, 1, s))
    x = mk((1, 2) + G)
    w = mk((3, 2) + K)
    full = conv.conv_forward(x, w, S)
    sharded = [p > 1 for p in parts]
    assembled = np.full(full.shape, np.nan)
    for shard in itertools.product(*[_splits(G[a], parts[a]) for a in range(nd)]):
        off = [s[0] for s in shard]
        ext = [s[1] for s in shard]
        g = geometry.shard_geometry(G, off, ext, K, S, sharded)
        tile = conv.padded_tile(x, g, [o if m else 0 for o, m in zip(off, sharded)],
                                [e if m else G[a] for a, (e, m) in enumerate(zip(ext, sharded))])
        y = conv.tile_conv(tile, w, S, g["pad_lo"], g["out_ext"])
        sl = (slice(None), slice(None)) + tuple(slice(o, o + e) for o, e in zip(g["out_off"], g["out_ext"]))
        assert np.all(np.isnan(assembled[sl]))
        assembled[sl] = y
    assert not np.isnan(assembled).any()
    if integer:
        assert np.array_equal(assembled, full)
    else:
        np.testing.assert_allclose(assembled, full, rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("case", CASES)
def test_shard_wgrad_partials_sum_to_full(case):
    G, K, S, parts = case
    nd = len(G)
    rng = np.random.default_rng(3 * sum(G))
    x = rng.integers(-2, 3, size=(2, 2) + G).astype(np.float64)
    n_out = [geometry.out_len(G[a], K[a], S[a]) for a in range(nd)]
    dy = rng.integers(-2, 3, size=(2, 3) + tuple(n_out)).astype(np.float64)
    full = conv.conv_wgrad(x, dy, K, S)
    total = np.zeros_like(full)
    sharded = [p > 1 for p in parts]
    for shard in itertools.product(*[_splits(G[a], parts[a]) for a in range(nd)]):
        g = geometry.shard_geometry(G, [s[0] for s in shard], [s[1] for s in shard], K, S, sharded)
        lo = g["out_off"]
        hi = [o + e for o, e in zip(g["out_off"], g["out_ext"])]
        sl = (slice(None), slice(None)) + tuple(slice(l, h) for l, h in zip(lo, hi))
        total += conv.conv_wgrad(x, dy[sl], K, S, lo, hi)
    assert np.array_equal(total, full)


def _exchange_all(x, G, K, S, parts):
    """Simulate the sequential per-axis halo exchange between all shards, each
    starting from its interior only, using only pack/unpack on tiles."""
    nd = len(G)
    sharded = [p > 1 for p in parts]
    grid = [_splits(G[a], parts[a]) for a in range(nd)]
    tiles, meta = {}, {}
    for idx in itertools.product(*[range(len(g)) for g in grid]):
        off = [grid[a][idx[a]][0] for a in range(nd)]
        ext = [grid[a][idx[a]][1] for a in range(nd)]
        g = geometry.shard_geometry(G, off, ext, K, S, sharded)
        lo, hi = g["halo_lo"], g["halo_hi"]
        tile = np.full([x.shape[0], x.shape[1]] + [l + e + h for l, e, h in zip(lo, ext, hi)], np.nan)
        inner = (slice(None), slice(None)) + tuple(slice(l, l + e) for l, e in zip(lo, ext))
        tile[inner] = x[(slice(None), slice(None)) + tuple(slice(o, o + e) for o, e in zip(off, ext))]
        tiles[idx] = tile
        meta[idx] = (off, ext, g)
    for axis in range(nd):
        for idx in tiles:
            off, ext, g = meta[idx]
            for side in (0, 1):
                width = g["halo_lo"][axis] if side == 0 else g["halo_hi"][axis]
                if width == 0:
                    continue
                nb = list(idx)
                nb[axis] += -1 if side == 0 else 1
                nb = tuple(nb)
                if nb in tiles:
                    noff, next_, ng = meta[nb]
                    slab = halo.pack(tiles[nb], axis, 1 - side, width, ng["halo_lo"], next_, ng["halo_hi"])
                else:
                    slab = None
                tiles[idx] = halo.unpack(tiles[idx], axis, side, slab, g["halo_lo"], ext, g["halo_hi"])
    return tiles, meta


@pytest.mark.parametrize("case", [c for c in CASES if max(c[3]) > 1])
def test_sequential_exchange_fills_padded_tiles(case):
    """After exchanging axes in ascending order with pack/unpack only, every tile
    equals the zero-extended full domain over its box, corners included; and the
    slab a neighbour sends equals the slab cut from the full domain."""
    G, K, S, parts = case
    rng = np.random.default_rng(42)
    x = rng.uniform(-1, 1, size=(1, 2) + G)
    tiles, meta = _exchange_all(x, G, K, S, parts)
    for idx, tile in tiles.items():
        off, ext, g = meta[idx]
        assert not np.isnan(tile).any()
        assert np.array_equal(tile, conv.padded_tile(x, g, off, ext))
        for axis in range(len(G)):
            for side in (0, 1):
                rs = halo.received_slab(x, axis, side, off, g["halo_lo"], ext, g["halo_hi"])
                lo, hi = halo.face_box(axis, halo.margin_rows(axis, side, g["halo_lo"], ext, g["halo_hi"]),
                                       g["halo_lo"], ext, g["halo_hi"])
                sl = (slice(None), slice(None)) + tuple(slice(l, h) for l, h in zip(lo, hi))
                assert np.array_equal(rs, tile[sl])
                assert list(rs.shape) == halo.slab_shape(1, 2, axis, hi[axis] - lo[axis], g["halo_lo"], ext,
                                                         g["halo_hi"])


def test_pack_then_unpack_round_trip():
    rng = np.random.default_rng(8)
    lo, ext, hi = [2, 1, 0], [5, 4, 6], [1, 2, 0]
    tile = rng.uniform(-1, 1, size=[1, 3] + [a + b + c for a, b, c in zip(lo, ext, hi)])
    for axis in range(2):
        for side in (0, 1):
            width = lo[axis] if side == 0 else hi[axis]
            s = halo.pack(tile, axis, side, width, lo, ext, hi)
            assert list(s.shape) == halo.slab_shape(1, 3, axis, width, lo, ext, hi)
            t2 = halo.unpack(tile, axis, side, s, lo, ext, hi)
            r0, r1 = halo.margin_rows(axis, side, lo, ext, hi)
            b0, b1 = halo.face_box(axis, (r0, r1), lo, ext, hi)
            sl = (slice(None), slice(None)) + tuple(slice(a, b) for a, b in zip(b0, b1))
            assert np.array_equal(t2[sl], s)
