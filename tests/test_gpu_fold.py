"""GPU parity of the forward with the halo folded into its tile loads
(shard_conv_fwd_folded) and of the interior / boundary split.

Every tile here keeps NaN canaries in all its margins: the folded call must read
each margin voxel from the received slab (or take zero at a global boundary),
so a margin read would poison the outputs. Bars: bit-identical to unpacking the
slabs and calling shard_conv_fwd (the same kernels and summation order), and
within the tolerance of the float64 oracle (bitwise on integer data); the
interior call writes exactly the outputs shard_conv_interior names, and
interior then boundary writes what the whole call writes.
"""
import os

import numpy as np
import pytest

import synth
import shard_cases as cases
from gpu_util import build_tile, canary_for, dev, empty_like_dtype, host, log, run_fwd, weights, window_from_tile
from oracle import halo as ohalo

pytestmark = pytest.mark.gpu

INT_DIST = (synth.INT, (-2.0, 2.0))


@pytest.fixture(scope="module")
def sc():
    import torch
    assert torch.cuda.is_available()
    from paper_2605_11111_amd import shardconv
    return shardconv


def _canary_tile_and_slabs(sc, w, idx, dist=None):
    """The padded tile with only its interior filled (NaN canaries in every
    margin) and the slabs the neighbours would send, cut from the same seeded
    full domain (None at a global boundary)."""
    sg = cases.shard_geom(w, idx)
    full_h = cases.x_box(w, sg.tile_lo, sg.tile_hi, cases.out_code(w), dist)
    lo, hi = sg.g["halo_lo"], sg.g["halo_hi"]
    tile_h = np.full_like(full_h, canary_for(w))
    inner = (slice(None),) + tuple(slice(l, l + e) for l, e in zip(lo, sg.ext)) + (slice(None),)
    tile_h[inner] = full_h[inner]
    slabs = {}
    for axis in range(w.nd):
        for side in (0, 1):
            width = lo[axis] if side == 0 else hi[axis]
            if width == 0:
                continue
            if cases.neighbour_exists(w, idx, axis, side):
                b0, b1 = ohalo.face_box(axis, ohalo.margin_rows(axis, side, lo, sg.ext, hi), lo, sg.ext, hi)
                box = (slice(None),) + tuple(slice(a, b) for a, b in zip(b0, b1)) + (slice(None),)
                slabs[(axis, side)] = dev(np.ascontiguousarray(full_h[box]))
            else:
                slabs[(axis, side)] = None
    desc = sc.tile_desc(w.N, w.cin, sg.ext, lo, hi)
    return desc, dev(tile_h), slabs, sg, full_h


def _folded(sc, w, desc, tile, slabs, sg, wt, region, y=None):
    import torch
    O = sg.g["out_ext"]
    if y is None:
        y = empty_like_dtype([w.N] + list(O) + [w.cout], w)
        y.view(torch.int16 if w.dtype == "bf16" else torch.int32).fill_(
            int(np.array(canary_for(w)).view(np.int16 if w.dtype == "bf16" else np.int32)))
    code = sc.SHARD_F32 if w.dtype == "f32" else sc.SHARD_BF16
    n = sc.shard_conv_workspace_bytes(0, desc, code, w.cout, w.K, w.S, O)
    ws = torch.empty(max(n, 16), dtype=torch.uint8, device="cuda")
    sc.shard_conv_fwd_folded(desc, tile, slabs, region, wt, w.cout, w.K, w.S, sg.g["pad_lo"], O, y, ws)
    return y


def _interior_mask(sc, w, desc, sg):
    lo, hi = sc.shard_conv_interior(desc, w.K, w.S, sg.g["pad_lo"], sg.g["out_ext"])
    m = np.zeros([w.N] + list(sg.g["out_ext"]) + [w.cout], dtype=bool)
    m[(slice(None),) + tuple(slice(a, b) for a, b in zip(lo, hi)) + (slice(None),)] = True
    return m


def _bits(a):
    return a.view(np.uint16 if a.dtype == np.uint16 else np.uint32)


@pytest.mark.parametrize("name", list(cases.REDUCED))
def test_folded_equals_unpacked_every_shard_reduced(sc, name):
    w = cases.REDUCED[name]
    w_host, w64 = weights(w)
    wt = dev(w_host)
    for idx in w.shards():
        log(f"folded {name} shard {idx}")
        desc, tile, slabs, sg, full_h = _canary_tile_and_slabs(sc, w, idx)
        got = host(_folded(sc, w, desc, tile, slabs, sg, wt, sc.SHARD_REGION_ALL))
        d2, t2, _, _ = build_tile(sc, w, idx)
        want = host(run_fwd(sc, w, d2, t2, sg, wt))
        assert np.array_equal(_bits(got), _bits(want)), idx
        xw, origin = window_from_tile(w, sg, full_h)
        ref = cases.expected_fwd(w, sg, xw, origin, w64)
        assert cases.norm_max_err(cases.as_f64(got, w), ref) <= cases.TOL[w.dtype], idx


@pytest.mark.parametrize("name", list(cases.REDUCED))
def test_interior_then_boundary(sc, name):
    """The interior call (no slabs at all) writes exactly the interior outputs;
    the boundary call then completes the tensor bit for bit."""
    w = cases.REDUCED[name]
    w_host, _ = weights(w)
    wt = dev(w_host)
    for idx in w.shards():
        log(f"split {name} shard {idx}")
        desc, tile, slabs, sg, _ = _canary_tile_and_slabs(sc, w, idx)
        whole = host(_folded(sc, w, desc, tile, slabs, sg, wt, sc.SHARD_REGION_ALL))
        inner = _interior_mask(sc, w, desc, sg)
        y = _folded(sc, w, desc, tile, None, sg, wt, sc.SHARD_REGION_INTERIOR)
        part = host(y)
        assert np.array_equal(_bits(part)[inner], _bits(whole)[inner]), idx
        assert np.all(_bits(part)[~inner] == _bits(np.array([canary_for(w)]))[0]), idx
        _folded(sc, w, desc, tile, slabs, sg, wt, sc.SHARD_REGION_BOUNDARY, y)
        assert np.array_equal(_bits(host(y)), _bits(whole)), idx
        # the boundary alone leaves the interior untouched
        yb = host(_folded(sc, w, desc, tile, slabs, sg, wt, sc.SHARD_REGION_BOUNDARY))
        assert np.array_equal(_bits(yb)[~inner], _bits(whole)[~inner]), idx
        assert np.all(_bits(yb)[inner] == _bits(np.array([canary_for(w)]))[0]), idx


@pytest.mark.parametrize("name", ["c3r", "c2r", "c4r", "c5r", "c1"])
@pytest.mark.parametrize("algo", ["", "tiled", "generic"])
def test_folded_kernel_variants_integer_exact(sc, name, algo):
    """Every kernel family folds the halo: integer data bit for bit against the
    oracle on the last shard along every axis (two neighbours where there are)."""
    sc.shard_set_call_opts(kernels=cases.KERNELS[algo])
    w = cases.REDUCED[name]
    idx = tuple(min(1, len(w.splits(a)) - 1) for a in range(w.nd))
    w_host, w64 = weights(w, INT_DIST)
    desc, tile, slabs, sg, full_h = _canary_tile_and_slabs(sc, w, idx, INT_DIST)
    got = host(_folded(sc, w, desc, tile, slabs, sg, dev(w_host), sc.SHARD_REGION_ALL))
    xw, origin = window_from_tile(w, sg, full_h)
    ref = cases.expected_fwd(w, sg, xw, origin, w64)
    if w.dtype == "bf16":
        assert np.array_equal(got, cases.bf16_rne_of_f64(ref))
    else:
        assert np.array_equal(got.astype(np.float64), ref)


FULL = ["c3_3d_bf16", "c2_2d_bf16", "c4_3d_bf16_k5", "c5_3d_fp32_s2"]


@pytest.mark.parametrize("name", FULL)
def test_full_size_folded_and_split_equal_unpacked(sc, name):
    """At full size, in the launch configuration the benchmark times: the folded
    call on a tile whose margins hold canaries, and the interior + boundary pair,
    equal the unpacked tile's forward bit for bit (compared on the device)."""
    import torch
    w = cases.WORKLOADS[name]
    w_host, _ = weights(w)
    wt = dev(w_host)
    log(f"full folded {name}: building tiles")
    desc, tile, slabs, sg, full_h = _canary_tile_and_slabs(sc, w, w.shard)
    del full_h
    d2, t2, _, _ = build_tile(sc, w, w.shard)
    log(f"full folded {name}: running")
    want = run_fwd(sc, w, d2, t2, sg, wt)
    del t2
    got = _folded(sc, w, desc, tile, slabs, sg, wt, sc.SHARD_REGION_ALL)
    assert torch.equal(got.view(torch.int16 if w.dtype == "bf16" else torch.int32),
                       want.view(torch.int16 if w.dtype == "bf16" else torch.int32))
    del got
    y = _folded(sc, w, desc, tile, None, sg, wt, sc.SHARD_REGION_INTERIOR)
    _folded(sc, w, desc, tile, slabs, sg, wt, sc.SHARD_REGION_BOUNDARY, y)
    torch.cuda.synchronize()
    assert torch.equal(y.view(torch.int16 if w.dtype == "bf16" else torch.int32),
                       want.view(torch.int16 if w.dtype == "bf16" else torch.int32))
    log(f"full folded {name}: ok")


def _wgrad_folded(sc, w, desc, tile, slabs, sg, dy):
    import torch
    O = sg.g["out_ext"]
    dw = torch.full((w.cout, w.cin) + tuple(w.K), float("nan"), device="cuda")
    code = sc.SHARD_F32 if w.dtype == "f32" else sc.SHARD_BF16
    n = sc.shard_conv_workspace_bytes(1, desc, code, w.cout, w.K, w.S, O)
    ws = torch.empty(max(n, 16), dtype=torch.uint8, device="cuda")
    sc.shard_conv_wgrad_folded(desc, tile, slabs, dy, w.cout, w.K, w.S, sg.g["pad_lo"], O, dw, ws)
    return dw


@pytest.mark.parametrize("name", list(cases.REDUCED))
def test_folded_wgrad_equals_unpacked_every_shard_reduced(sc, name):
    """The weight gradient reading the halo from the slabs (NaN canaries in every
    margin) equals unpack + shard_conv_wgrad: bit for bit with the general tiled
    kernels on both sides, to the tolerance with the fastest ones (the unpacked
    call may take a shape-specialised kernel that sums in another order), and
    matches the oracle."""
    from gpu_util import dy_box, run_wgrad
    w = cases.REDUCED[name]
    for idx in w.shards():
        log(f"folded wgrad {name} shard {idx}")
        desc, tile, slabs, sg, full_h = _canary_tile_and_slabs(sc, w, idx)
        dyh = dy_box(w, sg)
        dy = dev(dyh)
        d2, t2, _, _ = build_tile(sc, w, idx)
        xw, origin = window_from_tile(w, sg, full_h)
        ref = cases.expected_wgrad(w, sg, xw, origin, cases.to_ncdhw(cases.as_f64(dyh, w)))
        for algo in ("tiled", ""):
            with sc.call_opts(kernels=cases.KERNELS[algo]):
                got = _wgrad_folded(sc, w, desc, tile, slabs, sg, dy).cpu().numpy()
                want = run_wgrad(sc, w, d2, t2, sg, dy).cpu().numpy()
            if algo == "tiled":
                assert np.array_equal(got.view(np.uint32), want.view(np.uint32)), idx
            else:
                assert cases.norm_max_err(got.astype(np.float64), want.astype(np.float64)) <= cases.TOL[w.dtype], idx
            assert cases.norm_max_err(got.astype(np.float64), ref) <= cases.TOL[w.dtype], (idx, algo)


@pytest.mark.parametrize("name", ["c3r", "c2r", "c4r", "c5r", "c1"])
@pytest.mark.parametrize("algo", ["", "tiled", "generic"])
def test_folded_wgrad_kernel_variants_integer_exact(sc, name, algo):
    from gpu_util import dy_box
    sc.shard_set_call_opts(kernels=cases.KERNELS[algo])
    w = cases.REDUCED[name]
    idx = tuple(min(1, len(w.splits(a)) - 1) for a in range(w.nd))
    desc, tile, slabs, sg, full_h = _canary_tile_and_slabs(sc, w, idx, INT_DIST)
    dyh = dy_box(w, sg, INT_DIST)
    got = _wgrad_folded(sc, w, desc, tile, slabs, sg, dev(dyh)).cpu().numpy().astype(np.float64)
    xw, origin = window_from_tile(w, sg, full_h)
    ref = cases.expected_wgrad(w, sg, xw, origin, cases.to_ncdhw(cases.as_f64(dyh, w)))
    assert np.max(np.abs(ref)) < 2 ** 24
    assert np.array_equal(got, ref)


@pytest.mark.parametrize("name", ["c3_3d_bf16", "c2_2d_bf16", "c4_3d_bf16_k5"])
def test_full_size_folded_wgrad_equals_unpacked(sc, name):
    import torch
    from gpu_util import dy_box, run_wgrad
    w = cases.WORKLOADS[name]
    log(f"full folded wgrad {name}: building tiles")
    desc, tile, slabs, sg, full_h = _canary_tile_and_slabs(sc, w, w.shard)
    del full_h
    dy = dev(dy_box(w, sg))
    d2, t2, _, _ = build_tile(sc, w, w.shard)
    want = run_wgrad(sc, w, d2, t2, sg, dy)
    del t2
    got = _wgrad_folded(sc, w, desc, tile, slabs, sg, dy)
    assert torch.equal(got.view(torch.int32), want.view(torch.int32))
    log(f"full folded wgrad {name}: ok")


EDGE = [
    # (name, dtype, N, cin, cout, G, parts, K, S)
    ("1d_bf16", "bf16", 2, 16, 32, (301,), (3,), (5,), (1,)),
    ("1d_f32_s3", "f32", 1, 8, 8, (97,), (4,), (3,), (3,)),
    ("2d_k7_ragged_c", "bf16", 1, 24, 40, (29, 37), (3, 1), (7, 7), (1, 1)),
    ("2d_f32_two_axes", "f32", 2, 5, 7, (19, 21), (2, 2), (3, 3), (2, 1)),
    ("3d_s3_negative_pad", "f32", 1, 8, 16, (25, 9, 14), (2, 1, 1), (3, 3, 3), (3, 1, 2)),
    ("3d_thin_w", "bf16", 1, 32, 32, (10, 11, 3), (2, 1, 1), (3, 3, 3), (1, 1, 1)),
    ("3d_long_rows", "bf16", 1, 32, 32, (6, 5, 700), (2, 1, 1), (3, 3, 3), (1, 1, 1)),
    ("3d_three_axes", "bf16", 1, 16, 16, (12, 10, 40), (2, 2, 2), (3, 3, 3), (1, 1, 1)),
    ("2d_long_rows_h_split", "bf16", 2, 64, 64, (9, 1100), (2, 1), (3, 3), (1, 1)),
    # two batch items, three shards along D: both boundary planes of the middle
    # shard go in one W-march launch
    ("3d_batch2_split_d", "bf16", 2, 32, 32, (12, 10, 40), (3, 1, 1), (3, 3, 3), (1, 1, 1)),
    # the row-pair weight gradient's per-lane slab loads: margins on two axes,
    # a W split, a 5x5x5 corner shard
    ("2d_c16_k3_two_axes", "bf16", 2, 16, 64, (26, 40), (2, 2), (3, 3), (1, 1)),
    ("1d_c16_k5_split_w", "bf16", 1, 16, 64, (200,), (3,), (5,), (1,)),
    ("3d_c16_k5_two_axes", "bf16", 1, 16, 64, (12, 14, 36), (2, 2, 1), (5, 5, 5), (1, 1, 1)),
]


@pytest.mark.parametrize("case", EDGE, ids=lambda c: c[0])
def test_folded_edge_shapes_every_shard_integer_exact(sc, case):
    """Folded forward (whole, and interior then boundary) and folded weight
    gradient on edge shapes - 1D, strides 2 and 3, negative pads, margins on two
    and three axes (corners from the later axis's slab), odd channel counts, long
    rows - bit for bit against the oracle on integer data, every shard."""
    from gpu_util import dy_box
    name, dt, N, cin, cout, G, parts, K, S = case
    wl = cases.Workload(name, dt, N, cin, cout, G, parts, K, S, (0,) * len(G),
                        x_dist=(synth.UNIFORM, (-1.0, 1.0)), w_dist=(synth.UNIFORM, (-0.5, 0.5)),
                        dy_dist=(synth.UNIFORM, (-1.0, 1.0)))
    w_host, w64 = weights(wl, INT_DIST)
    wt = dev(w_host)
    for idx in wl.shards():
        log(f"folded edge {name} shard {idx}")
        desc, tile, slabs, sg, full_h = _canary_tile_and_slabs(sc, wl, idx, INT_DIST)
        xw, origin = window_from_tile(wl, sg, full_h)
        ref = cases.expected_fwd(wl, sg, xw, origin, w64)
        want = cases.bf16_rne_of_f64(ref) if dt == "bf16" else ref
        for parts_ in ((sc.SHARD_REGION_ALL,), (sc.SHARD_REGION_INTERIOR, sc.SHARD_REGION_BOUNDARY)):
            y = None
            for region in parts_:
                y = _folded(sc, wl, desc, tile, None if region == sc.SHARD_REGION_INTERIOR else slabs, sg, wt,
                            region, y)
            got = host(y)
            if dt == "bf16":
                assert np.array_equal(got, want), (idx, parts_)
            else:
                assert np.array_equal(got.astype(np.float64), want), (idx, parts_)
        dyh = dy_box(wl, sg, INT_DIST)
        dref = cases.expected_wgrad(wl, sg, xw, origin, cases.to_ncdhw(cases.as_f64(dyh, wl)))
        assert np.max(np.abs(dref)) < 2 ** 24
        dw = _wgrad_folded(sc, wl, desc, tile, slabs, sg, dev(dyh)).cpu().numpy().astype(np.float64)
        assert np.array_equal(dw, dref), idx
