"""Pins for the oracle's input gradient and reverse halo exchange (CPU only).

The input gradient is tied to hand-worked values, a scalar-loop transcription,
the transpose of the dense Toeplitz matrix of the forward convolution, torch's
float64 autograd (a library routine), closed forms, and the adjoint identity
with the forward convolution read off a tile. The reverse exchange is pinned by
running it between every shard of split domains: afterwards each shard's
interior must equal the full-domain input gradient over its box.
"""
import itertools
import json
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import brute, conv, geometry, halo

GOLDEN = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "worked_examples.json")))

# (nd, N, Ci, Co, G, K, S)
TINY = [
    (1, 1, 2, 3, (7,), (3,), (1,)),
    (1, 2, 1, 2, (9,), (5,), (2,)),
    (1, 1, 3, 1, (8,), (1,), (3,)),
    (2, 1, 2, 2, (5, 6), (3, 3), (1, 1)),
    (2, 1, 1, 2, (7, 5), (3, 5), (2, 1)),
    (2, 2, 2, 1, (6, 6), (5, 1), (1, 3)),
    (3, 1, 2, 2, (4, 5, 3), (3, 3, 3), (1, 1, 1)),
    (3, 1, 1, 2, (5, 4, 6), (3, 1, 3), (2, 1, 2)),
]
TORCH_CASES = TINY + [
    (2, 1, 4, 5, (17, 13), (3, 3), (1, 1)),
    (3, 1, 3, 4, (9, 8, 10), (5, 5, 5), (1, 1, 1)),
    (3, 2, 4, 3, (11, 9, 7), (3, 3, 3), (2, 2, 2)),
    (2, 1, 3, 2, (10, 11), (7, 3), (3, 2)),
]


def rnd(rng, shape, integer=False):
    if integer:
        return rng.integers(-2, 3, size=shape).astype(np.float64)
    return rng.uniform(-1, 1, size=shape)


def n_out(G, K, S):
    return tuple(geometry.out_len(g, k, s) for g, k, s in zip(G, K, S))


@pytest.mark.parametrize("case", GOLDEN["dgrad1d"], ids=lambda c: c["what"][:40])
def test_hand_worked_1d(case):
    w = np.array(case["w"], dtype=np.float64).reshape(1, 1, -1)
    dy = np.array(case["dy"], dtype=np.float64).reshape(1, 1, -1)
    dx = conv.conv_dgrad(dy, w, (case["G"],), (case["stride"],))
    assert dx.reshape(-1).tolist() == case["dx"]


@pytest.mark.parametrize("shape", TINY)
@pytest.mark.parametrize("integer", [True, False])
def test_dgrad_vs_scalar_loops(shape, integer):
    nd, N, Ci, Co, G, K, S = shape
    rng = np.random.default_rng(hash((shape, integer, "dgrad")) % 2**32)
    w = rnd(rng, (Co, Ci) + K, integer)
    dy = rnd(rng, (N, Co) + n_out(G, K, S), integer)
    dx = conv.conv_dgrad(dy, w, G, S)
    db = brute.dgrad_scalar(dy, w, G, S)
    if integer:
        assert np.array_equal(dx, db)
    else:
        np.testing.assert_allclose(dx, db, rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("shape", TINY[:6])
def test_dgrad_is_the_toeplitz_transpose(shape):
    nd, N, Ci, Co, G, K, S = shape
    rng = np.random.default_rng(11)
    w = rnd(rng, (Co, Ci) + K)
    dy = rnd(rng, (N, Co) + n_out(G, K, S))
    T = brute.toeplitz(w, G, S)
    dx = conv.conv_dgrad(dy, w, G, S)
    for n in range(N):
        np.testing.assert_allclose(dx[n].reshape(-1), T.T @ dy[n].reshape(-1), rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("shape", TORCH_CASES)
def test_dgrad_vs_torch_autograd_float64(shape):
    nd, N, Ci, Co, G, K, S = shape
    rng = np.random.default_rng(5)
    x = rnd(rng, (N, Ci) + G)
    w = rnd(rng, (Co, Ci) + K)
    dy = rnd(rng, (N, Co) + n_out(G, K, S))
    fn = {1: F.conv1d, 2: F.conv2d, 3: F.conv3d}[nd]
    xt = torch.tensor(x, requires_grad=True)
    yt = fn(xt, torch.tensor(w), stride=S, padding=[(k - 1) // 2 for k in K])
    (yt * torch.tensor(dy)).sum().backward()
    np.testing.assert_allclose(conv.conv_dgrad(dy, w, G, S), xt.grad.numpy(), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("nd,S", [(1, 1), (2, 2), (3, 1), (3, 2)])
def test_delta_kernel_scatters_dy(nd, S):
    """w = e(co=1, ci=0, tap t): dx[ci=0][j*S - P + t] = dy[co=1][j], every other
    input gradient zero."""
    rng = np.random.default_rng(nd * 10 + S)
    G = (9, 7, 6)[:nd]
    K = (3, 5, 3)[:nd]
    Sv = (S,) * nd
    t = tuple(k - 1 for k in K)
    w = np.zeros((2, 2) + K)
    w[(1, 0) + t] = 1.0
    dy = rnd(rng, (1, 2) + n_out(G, K, Sv))
    dx = conv.conv_dgrad(dy, w, G, Sv)
    ref = np.zeros((1, 2) + G)
    for j in itertools.product(*[range(m) for m in n_out(G, K, Sv)]):
        i = tuple(j[a] * S - (K[a] - 1) // 2 + t[a] for a in range(nd))
        if all(0 <= i[a] < G[a] for a in range(nd)):
            ref[(0, 0) + i] = dy[(0, 1) + j]
    assert np.array_equal(dx, ref)


@pytest.mark.parametrize("nd,S", [(1, 2), (2, 1), (3, 1), (3, 2)])
def test_ones_count_the_outputs_reading_each_input(nd, S):
    """dy = 1, w = 1: dx[i] = Co * prod over axes of #{(j, t): j*S - P + t = i}."""
    G = (8, 7, 5)[:nd]
    K = (3, 3, 5)[:nd]
    Sv = (S,) * nd
    Co = 3
    w = np.ones((Co, 2) + K)
    dy = np.ones((1, Co) + n_out(G, K, Sv))
    dx = conv.conv_dgrad(dy, w, G, Sv)
    per_axis = []
    for a in range(nd):
        P = (K[a] - 1) // 2
        cnt = np.zeros(G[a])
        for j in range(n_out(G, K, Sv)[a]):
            for tt in range(K[a]):
                i = j * S - P + tt
                if 0 <= i < G[a]:
                    cnt[i] += 1
        per_axis.append(cnt)
    ref = Co * np.ones(G)
    for a, cnt in enumerate(per_axis):
        shp = [1] * nd
        shp[a] = -1
        ref = ref * cnt.reshape(shp)
    assert np.array_equal(dx[0, 0], ref) and np.array_equal(dx[0, 1], ref)


@pytest.mark.parametrize("pad,S", [((1, 1), (1, 1)), ((0, 2), (2, 1)), ((-1, 1), (3, 1)), ((2, 0), (1, 2))])
def test_tile_dgrad_is_the_adjoint_of_tile_conv(pad, S):
    """<tile_conv(T), dy> = <T, tile_dgrad(dy)> for any tile T and dy."""
    rng = np.random.default_rng(abs(hash((pad, S))) % 2**32)
    tile_ext = (11, 9)
    K = (3, 5)
    out_ext = (4, 6)
    T = rnd(rng, (2, 3) + tile_ext)
    w = rnd(rng, (4, 3) + K)
    dy = rnd(rng, (2, 4) + out_ext)
    lhs = float(np.sum(conv.tile_conv(T, w, S, pad, out_ext) * dy))
    rhs = float(np.sum(T * conv.tile_dgrad(dy, w, S, pad, tile_ext)))
    assert abs(lhs - rhs) <= 1e-11 * max(1.0, abs(lhs))


def _splits(G, parts):
    sizes = geometry.chunk_sizes(G, parts)
    return list(zip(geometry.offsets(sizes), sizes))


CASES = [
    # (G, K, S, parts per axis)
    ((16,), (3,), (1,), (3,)),
    ((19,), (5,), (2,), (4,)),
    ((12, 10), (3, 3), (1, 1), (2, 1)),
    ((13, 11), (5, 3), (1, 2), (3, 2)),
    ((10, 9, 8), (3, 3, 3), (1, 1, 1), (2, 2, 1)),
    ((12, 7, 9), (3, 3, 3), (2, 1, 2), (3, 1, 1)),
    ((9, 10, 7), (5, 5, 5), (1, 1, 1), (2, 2, 1)),
    ((11, 8, 6), (3, 5, 1), (3, 1, 1), (4, 1, 2)),
]


def reverse_exchange(G, K, S, parts, dy, w, rounding=None):
    """Every shard computes tile_dgrad of its owned dy onto its padded tile, then
    the margins are returned axis by axis in descending order with
    pack_margin / accumulate. Returns {shard: (tile gradient, geometry, ext)}."""
    nd = len(G)
    sharded = [p > 1 for p in parts]
    grid = [_splits(G[a], parts[a]) for a in range(nd)]
    tiles, meta = {}, {}
    for idx in itertools.product(*[range(len(g)) for g in grid]):
        off = [grid[a][idx[a]][0] for a in range(nd)]
        ext = [grid[a][idx[a]][1] for a in range(nd)]
        g = geometry.shard_geometry(G, off, ext, K, S, sharded)
        P = [l + e + h for l, e, h in zip(g["halo_lo"], ext, g["halo_hi"])]
        sl = (slice(None), slice(None)) + tuple(slice(o, o + e) for o, e in zip(g["out_off"], g["out_ext"]))
        tg = conv.tile_dgrad(dy[sl], w, S, g["pad_lo"], P)
        tiles[idx] = tg if rounding is None else rounding(tg)
        meta[idx] = (off, ext, g)
    for axis in reversed(range(nd)):
        sends = []
        for idx in tiles:
            off, ext, g = meta[idx]
            for side in (0, 1):
                width = g["halo_lo"][axis] if side == 0 else g["halo_hi"][axis]
                nb = list(idx)
                nb[axis] += -1 if side == 0 else 1
                nb = tuple(nb)
                if width == 0 or nb not in tiles:
                    continue  # no margin, or a global boundary: the gradient on the zero padding is dropped
                sends.append((nb, 1 - side, width, halo.pack_margin(tiles[idx], axis, side, g["halo_lo"], ext,
                                                                    g["halo_hi"])))
        for nb, side, width, slab in sends:
            noff, next_, ng = meta[nb]
            tiles[nb] = halo.accumulate(tiles[nb], axis, side, width, slab, ng["halo_lo"], next_, ng["halo_hi"],
                                        rounding)
    return tiles, meta


@pytest.mark.parametrize("case", CASES)
@pytest.mark.parametrize("integer", [True, False])
def test_reverse_exchange_gives_the_full_input_gradient(case, integer):
    G, K, S, parts = case
    nd = len(G)
    rng = np.random.default_rng(sum(G) * 3 + nd)
    w = rnd(rng, (3, 2) + K, integer)
    dy = rnd(rng, (2, 3) + n_out(G, K, S), integer)
    full = conv.conv_dgrad(dy, w, G, S)
    covered = np.zeros(full.shape, dtype=bool)
    tiles, meta = reverse_exchange(G, K, S, parts, dy, w)
    for idx, tg in tiles.items():
        off, ext, g = meta[idx]
        inner = (slice(None), slice(None)) + tuple(slice(l, l + e) for l, e in zip(g["halo_lo"], ext))
        box = (slice(None), slice(None)) + tuple(slice(o, o + e) for o, e in zip(off, ext))
        if integer:
            assert np.array_equal(tg[inner], full[box])
        else:
            np.testing.assert_allclose(tg[inner], full[box], rtol=1e-12, atol=1e-12)
        covered[box] = True
    assert covered.all()


def test_margins_of_an_unsplit_axis_keep_their_gradient_out():
    """On an unsplit axis the tile has no margin: taps that fall on the zero padding
    drop out of tile_dgrad exactly as they drop out of the full-domain gradient."""
    rng = np.random.default_rng(3)
    G, K, S = (9, 8), (3, 5), (1, 1)
    w = rnd(rng, (2, 2) + K, True)
    dy = rnd(rng, (1, 2) + n_out(G, K, S), True)
    g = geometry.shard_geometry(G, [0, 0], list(G), K, S, [False, False])
    assert g["halo_lo"] == [0, 0] and g["pad_lo"] == [1, 2]
    assert np.array_equal(conv.tile_dgrad(dy, w, S, g["pad_lo"], G), conv.conv_dgrad(dy, w, G, S))


@pytest.mark.parametrize("case", GOLDEN["bf16_accumulate"], ids=lambda c: c["what"][:40])
def test_bf16_accumulate_rounding(case):
    """accumulate with the bf16 rounding (binary32 sum, then nearest-even) on the
    hand-worked ties."""
    lo, ext, hi = [1], [3], [1]
    tile = np.full((1, 1, 5), case["tile"])
    slab = np.full((1, 1, 1), case["slab"])
    rnd_bf16 = lambda v: conv.bf16_value(conv.round_bf16(v))
    out = halo.accumulate(tile, 0, 0, 1, slab, lo, ext, hi, rnd_bf16)
    assert out[0, 0, 1] == case["sum"]
    assert out[0, 0, 0] == case["tile"] and out[0, 0, 2] == case["tile"]
