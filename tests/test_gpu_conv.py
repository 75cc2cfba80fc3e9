"""GPU parity of the shard convolution (forward and weight gradient) against
the float64 oracle.

Bars: fp32 normalised max error <= 1e-5, bf16 (fp32 accumulation) <= 2e-2;
integer-valued inputs (exact in bf16 and fp32, partial sums below 2^24) must
match bit for bit, a bf16 output being the oracle's round-to-nearest-even of
the exact sum. Reduced domains check every shard; full-size workloads run the
launch configuration the benchmark times and are checked on sampled output
planes (forward) and on a weight gradient whose dy is supported on sampled
planes (its exact value is the oracle's sum over those planes).
"""
import os

import numpy as np
import pytest

import synth
import shard_cases as cases
from gpu_util import build_tile, dev, dy_box, host, log, run_fwd, run_wgrad, weights, window_from_tile
from oracle import conv as oconv

pytestmark = pytest.mark.gpu

INT_DIST = (synth.INT, (-2.0, 2.0))


@pytest.fixture(scope="module")
def sc():
    import torch
    assert torch.cuda.is_available()
    from paper_2605_11111_amd import shardconv
    return shardconv


def _fwd_case(sc, w, idx, x_dist=None, w_dist=None):
    desc, tile, sg, full_h = build_tile(sc, w, idx, x_dist, keep_host=True)
    w_host, w64 = weights(w, w_dist)
    y = host(run_fwd(sc, w, desc, tile, sg, dev(w_host)))
    xw, origin = window_from_tile(w, sg, full_h)
    ref = cases.expected_fwd(w, sg, xw, origin, w64)
    return y, ref, sg


def _wgrad_case(sc, w, idx, x_dist=None, dy_dist=None):
    desc, tile, sg, full_h = build_tile(sc, w, idx, x_dist, keep_host=True)
    dyh = dy_box(w, sg, dy_dist)
    dw = host(run_wgrad(sc, w, desc, tile, sg, dev(dyh)))
    xw, origin = window_from_tile(w, sg, full_h)
    ref = cases.expected_wgrad(w, sg, xw, origin, cases.to_ncdhw(cases.as_f64(dyh, w)))
    return dw, ref


@pytest.mark.parametrize("name", list(cases.REDUCED))
def test_forward_every_shard_reduced(sc, name):
    w = cases.REDUCED[name]
    for idx in w.shards():
        log(f"fwd {name} shard {idx}")
        y, ref, _ = _fwd_case(sc, w, idx)
        err = cases.norm_max_err(cases.as_f64(y, w), ref)
        assert err <= cases.TOL[w.dtype], (idx, err)


@pytest.mark.parametrize("name", list(cases.REDUCED))
def test_forward_integer_exact_reduced(sc, name):
    w = cases.REDUCED[name]
    for idx in w.shards():
        y, ref, _ = _fwd_case(sc, w, idx, INT_DIST, INT_DIST)
        if w.dtype == "bf16":
            assert np.array_equal(y, cases.bf16_rne_of_f64(ref)), idx
        else:
            assert np.array_equal(y.astype(np.float64), ref), idx


@pytest.mark.parametrize("name", list(cases.REDUCED))
def test_wgrad_every_shard_reduced(sc, name):
    w = cases.REDUCED[name]
    for idx in w.shards():
        log(f"wgrad {name} shard {idx}")
        dw, ref = _wgrad_case(sc, w, idx)
        err = cases.norm_max_err(dw.astype(np.float64), ref)
        assert err <= cases.TOL[w.dtype], (idx, err)


@pytest.mark.parametrize("name", list(cases.REDUCED))
def test_wgrad_integer_exact_reduced(sc, name):
    w = cases.REDUCED[name]
    for idx in w.shards():
        dw, ref = _wgrad_case(sc, w, idx, INT_DIST, INT_DIST)
        assert np.max(np.abs(ref)) < 2 ** 24
        assert np.array_equal(dw.astype(np.float64), ref), idx


def test_c1_concatenated_shards_equal_full_domain(sc):
    w = cases.C1
    x = cases.to_ncdhw(cases.as_f64(cases.field(w, "x").box(out=cases.out_code(w)), w))
    _, w64 = weights(w)
    full = cases.to_cl(oconv.conv_forward(x, w64, w.S))
    pieces = []
    for idx in w.shards():
        y, _, sg = _fwd_case(sc, w, idx)
        pieces.append(y.astype(np.float64))
    got = np.concatenate(pieces, axis=1)
    assert got.shape == full.shape
    assert cases.norm_max_err(got, full) <= cases.TOL["f32"]


@pytest.mark.parametrize("name", ["c3r", "c2r", "c4r", "c5r", "c1"])
def test_kernel_variants_agree(sc, name):
    """The shape-specialised kernels (default), the general tiled MFMA kernels
    (SHARD_KERNELS_TILED) and the direct kernels (SHARD_KERNELS_DIRECT) give
    the same result: bitwise on integer data, to the tolerance otherwise."""
    w = cases.REDUCED[name]
    idx = tuple(len(w.splits(a)) - 1 for a in range(w.nd))
    for dist in (INT_DIST, None):
        desc, tile, sg, _ = build_tile(sc, w, idx, dist)
        w_host, _ = weights(w, dist)
        wt, dyh = dev(w_host), dev(dy_box(w, sg, dist))
        res = {}
        for algo in ("", "tiled", "generic"):
            with sc.call_opts(kernels=cases.KERNELS[algo]):
                res[algo] = (host(run_fwd(sc, w, desc, tile, sg, wt)), host(run_wgrad(sc, w, desc, tile, sg, dyh)))
        y0, d0 = res[""]
        for algo in ("tiled", "generic"):
            y1, d1 = res[algo]
            if dist is INT_DIST:
                assert np.array_equal(y0, y1) and np.array_equal(d0, d1), (name, algo)
            else:
                assert cases.norm_max_err(cases.as_f64(y1, w), cases.as_f64(y0, w)) <= cases.TOL[w.dtype]
                assert cases.norm_max_err(d1.astype(np.float64), d0.astype(np.float64)) <= cases.TOL[w.dtype]


def test_repeat_runs_are_bitwise_identical(sc):
    for name in ("c3r", "c5r"):
        w = cases.REDUCED[name]
        idx = w.shards()[1]
        desc, tile, sg, _ = build_tile(sc, w, idx)
        w_host, _ = weights(w)
        dyh = dev(dy_box(w, sg))
        wt = dev(w_host)
        a = [host(run_fwd(sc, w, desc, tile, sg, wt)) for _ in range(2)]
        b = [host(run_wgrad(sc, w, desc, tile, sg, dyh)) for _ in range(2)]
        assert np.array_equal(a[0], a[1]) and np.array_equal(b[0], b[1])


# --- edge cases ----------------------------------------------------------------

EDGE = [
    # (name, dtype, N, cin, cout, G, parts, K, S)
    ("1d_bf16", "bf16", 2, 16, 32, (301,), (3,), (5,), (1,)),
    ("1d_f32_s3", "f32", 1, 8, 8, (97,), (4,), (3,), (3,)),
    ("2d_k1", "bf16", 1, 32, 48, (33, 45), (2, 1), (1, 1), (1, 1)),
    ("2d_k7_ragged_c", "bf16", 1, 24, 40, (29, 37), (3, 1), (7, 7), (1, 1)),
    ("2d_odd_channels", "bf16", 1, 3, 5, (20, 23), (2, 1), (3, 3), (1, 1)),
    ("2d_f32_odd_channels", "f32", 2, 5, 7, (19, 21), (2, 2), (3, 3), (2, 1)),
    ("3d_s3_negative_pad", "f32", 1, 8, 16, (25, 9, 14), (2, 1, 1), (3, 3, 3), (3, 1, 2)),
    ("3d_wide_channels", "bf16", 1, 96, 80, (9, 10, 40), (2, 1, 1), (3, 3, 3), (1, 1, 1)),
    ("3d_thin_w", "bf16", 1, 32, 32, (10, 11, 3), (2, 1, 1), (3, 3, 3), (1, 1, 1)),
    # few long rows: the W-march kernels split rows into segments
    ("3d_long_rows", "bf16", 1, 32, 32, (6, 5, 700), (2, 1, 1), (3, 3, 3), (1, 1, 1)),
    ("2d_long_rows", "bf16", 2, 64, 64, (9, 1100), (2, 1), (3, 3), (1, 1)),
    # 16 or fewer output channels: 16 x 16 output tiles (cin not a multiple of
    # the 32-channel K chunk in the second)
    ("3d_narrow_out", "bf16", 1, 64, 16, (10, 12, 40), (2, 1, 1), (3, 3, 3), (1, 1, 1)),
    ("2d_narrow_out_k5", "bf16", 2, 48, 12, (21, 33), (2, 1), (5, 5), (1, 1)),
    # 16 input channels, output channels in blocks of 64: the row-pair weight
    # gradient (row pairs and W pairs; a 1x1 kernel leaves half the waves
    # without tiles; ragged W runs; two output-channel blocks)
    ("2d_c16_k3_rowpair", "bf16", 2, 16, 64, (34, 50), (2, 1), (3, 3), (1, 1)),
    ("2d_c16_k1_rowpair", "bf16", 1, 16, 64, (33, 45), (2, 1), (1, 1), (1, 1)),
    ("1d_c16_k5_rowpair", "bf16", 1, 16, 128, (300,), (3,), (5,), (1,)),
    ("3d_c16_k5_ragged", "bf16", 1, 16, 64, (11, 13, 37), (2, 1, 1), (5, 5, 5), (1, 1, 1)),
    # shards of 8 x 16 x 24 outputs: the general forward takes bricks 8 voxels
    # wide whose rows lie 10 voxels apart in LDS, read with the transposed
    # M-row order (one and two N tiles; a ragged N tile of 40 channels)
    ("3d_bricks_8_wide", "bf16", 1, 16, 32, (16, 16, 24), (2, 1, 1), (3, 3, 3), (1, 1, 1)),
    ("3d_bricks_8_wide_c48", "bf16", 2, 48, 40, (16, 16, 24), (2, 1, 1), (3, 3, 3), (1, 1, 1)),
    # one N tile over 8x8x8 bricks, ragged along H and W: a partial channel
    # chunk (24), output channels ending inside a 16-byte run (20), three chunks (40)
    ("3d_one_ntile_k5_c24", "bf16", 1, 24, 24, (16, 14, 14), (2, 1, 1), (3, 5, 3), (1, 1, 1)),
    ("3d_one_ntile_k5_c20", "bf16", 1, 16, 20, (16, 14, 14), (2, 1, 1), (5, 5, 5), (1, 1, 1)),
    ("3d_one_ntile_k3_c40", "bf16", 1, 40, 16, (16, 14, 14), (2, 1, 1), (3, 3, 5), (1, 1, 1)),
]


@pytest.mark.parametrize("case", EDGE, ids=lambda c: c[0])
def test_edge_shapes_every_shard(sc, case):
    name, dt, N, cin, cout, G, parts, K, S = case
    wl = cases.Workload(name, dt, N, cin, cout, G, parts, K, S, (0,) * len(G),
                        x_dist=(synth.UNIFORM, (-1.0, 1.0)), w_dist=(synth.UNIFORM, (-0.5, 0.5)),
                        dy_dist=(synth.UNIFORM, (-1.0, 1.0)))
    for idx in wl.shards():
        log(f"edge {name} shard {idx}")
        y, ref, sg = _fwd_case(sc, wl, idx)
        assert cases.norm_max_err(cases.as_f64(y, wl), ref) <= cases.TOL[dt], idx
        dw, dref = _wgrad_case(sc, wl, idx)
        assert cases.norm_max_err(dw.astype(np.float64), dref) <= cases.TOL[dt], idx
        yi, refi, _ = _fwd_case(sc, wl, idx, INT_DIST, INT_DIST)
        if dt == "bf16":
            assert np.array_equal(yi, cases.bf16_rne_of_f64(refi)), idx
        else:
            assert np.array_equal(yi.astype(np.float64), refi), idx


def test_empty_outputs(sc):
    import torch
    w = cases.REDUCED["c4r"]
    sg = cases.shard_geom(w, (0, 0, 0))
    desc = sc.tile_desc(w.N, w.cin, sg.ext, sg.g["halo_lo"], sg.g["halo_hi"])
    tile = torch.zeros([1] + [l + e + h for l, e, h in zip(sg.g["halo_lo"], sg.ext, sg.g["halo_hi"])] + [w.cin],
                       dtype=torch.bfloat16, device="cuda")
    O = [0, sg.g["out_ext"][1], sg.g["out_ext"][2]]
    sc.shard_conv_fwd(desc, tile, torch.zeros(1, dtype=torch.bfloat16, device="cuda"), w.cout, w.K, w.S,
                      sg.g["pad_lo"], O, torch.zeros(1, dtype=torch.bfloat16, device="cuda"), None)
    dw = torch.full((w.cout, w.cin) + tuple(w.K), 7.0, device="cuda")
    n = sc.shard_conv_workspace_bytes(1, desc, sc.SHARD_BF16, w.cout, w.K, w.S, O)
    ws = torch.empty(max(n, 16), dtype=torch.uint8, device="cuda")
    sc.shard_conv_wgrad(desc, tile, torch.zeros(1, dtype=torch.bfloat16, device="cuda"), w.cout, w.K, w.S,
                        sg.g["pad_lo"], O, dw, ws)
    assert float(dw.abs().max()) == 0.0


# --- full-size workloads (the launch configuration the benchmark times) ---------

FULL = ["c1_2d_fp32", "c2_2d_bf16", "c4_3d_bf16_k5", "c5_3d_fp32_s2", "c3_3d_bf16"]


def _planes(L, rng):
    extra = sorted(set(int(v) for v in rng.integers(2, max(3, L - 2), size=2)))
    return sorted(set([0, 1, L - 2, L - 1] + extra))


@pytest.mark.parametrize("name", FULL)
def test_full_size_forward_sampled_planes(sc, name):
    w = cases.WORKLOADS[name]
    log(f"full fwd {name}: building tile")
    desc, tile, sg, full_h = build_tile(sc, w, w.shard, keep_host=True)
    w_host, w64 = weights(w)
    log(f"full fwd {name}: running")
    y = run_fwd(sc, w, desc, tile, sg, dev(w_host))
    L = sg.g["out_ext"][0]
    planes = _planes(L, np.random.default_rng(1))
    yh = host(y[:, planes])
    del y, tile
    for k, p in enumerate(planes):
        r0 = p * w.S[0] - sg.g["pad_lo"][0]
        xw, origin = window_from_tile(w, sg, full_h, (r0, r0 + w.K[0]))
        lo, hi = cases.owned_box(sg)
        lo[0], hi[0] = lo[0] + p, lo[0] + p + 1
        ref = cases.to_cl(oconv.conv_forward_window(xw, origin, w.G, w64, w.S, lo, hi))
        err = cases.norm_max_err(cases.as_f64(yh[:, k:k + 1], w), ref)
        log(f"  plane {p}: normalised max err {err:.3e}")
        assert err <= cases.TOL[w.dtype], (p, err)


@pytest.mark.parametrize("name", FULL)
def test_full_size_forward_integer_exact_sampled_planes(sc, name):
    w = cases.WORKLOADS[name]
    desc, tile, sg, full_h = build_tile(sc, w, w.shard, INT_DIST, keep_host=True)
    w_host, w64 = weights(w, INT_DIST)
    y = run_fwd(sc, w, desc, tile, sg, dev(w_host))
    L = sg.g["out_ext"][0]
    planes = _planes(L, np.random.default_rng(2))
    yh = host(y[:, planes])
    del y, tile
    for k, p in enumerate(planes):
        r0 = p * w.S[0] - sg.g["pad_lo"][0]
        xw, origin = window_from_tile(w, sg, full_h, (r0, r0 + w.K[0]))
        lo, hi = cases.owned_box(sg)
        lo[0], hi[0] = lo[0] + p, lo[0] + p + 1
        ref = cases.to_cl(oconv.conv_forward_window(xw, origin, w.G, w64, w.S, lo, hi))
        got = yh[:, k:k + 1]
        if w.dtype == "bf16":
            assert np.array_equal(got, cases.bf16_rne_of_f64(ref)), p
        else:
            assert np.array_equal(got.astype(np.float64), ref), p


@pytest.mark.parametrize("name", FULL)
@pytest.mark.parametrize("integer", [False, True])
def test_full_size_wgrad_with_plane_supported_dy(sc, name, integer):
    """dy is the seeded field on a few output planes and zero elsewhere; the
    kernel still sweeps the whole shard, and its result must equal the oracle's
    weight gradient summed over those planes only."""
    import torch
    w = cases.WORKLOADS[name]
    dist = INT_DIST if integer else None
    desc, tile, sg, full_h = build_tile(sc, w, w.shard, dist, keep_host=True)
    L = sg.g["out_ext"][0]
    planes = _planes(L, np.random.default_rng(3))
    lo, hi = cases.owned_box(sg)
    f = cases.field(w, "dy", dist)
    dy = torch.zeros([w.N] + list(sg.g["out_ext"]) + [w.cout], dtype=cases.torch_dtype(w), device="cuda")
    ref = np.zeros((w.cout, w.cin) + tuple(w.K))
    for p in planes:
        l2, h2 = list(lo), list(hi)
        l2[0], h2[0] = lo[0] + p, lo[0] + p + 1
        dyp = f.box((0, 0, *l2), (w.N, w.cout, *h2), out=cases.out_code(w))
        dy[:, p:p + 1] = dev(dyp)
        r0 = p * w.S[0] - sg.g["pad_lo"][0]
        xw, origin = window_from_tile(w, sg, full_h, (r0, r0 + w.K[0]))
        ref += oconv.conv_wgrad_window(xw, origin, w.G, cases.to_ncdhw(cases.as_f64(dyp, w)), w.K, w.S, l2, h2)
    dw = host(run_wgrad(sc, w, desc, tile, sg, dy)).astype(np.float64)
    if integer:
        assert np.max(np.abs(ref)) < 2 ** 24
        assert np.array_equal(dw, ref)
    else:
        err = cases.norm_max_err(dw, ref)
        log(f"  wgrad {name}: normalised max err {err:.3e}")
        assert err <= cases.TOL[w.dtype]


# the shapes of the three weight-gradient kernel families at full size: the
# W-march kernel (C3), the tiled bf16 kernel (C4) and the tiled fp32 kernel (C5)
DENSE_WGRAD = ["c3_3d_bf16", "c4_3d_bf16_k5", "c5_3d_fp32_s2"]


@pytest.mark.parametrize("name", DENSE_WGRAD)
@pytest.mark.timeout(900)
def test_full_size_wgrad_dense_dy(sc, name):
    """The weight gradient of the whole shard on the full seeded dy (every owned
    output voxel contributes: the full split-K accumulation), against the oracle
    summed over chunks of output planes on the host (the oracle's sum over the
    owned box, taken chunk by chunk, is the same sum)."""
    w = cases.WORKLOADS[name]
    log(f"dense wgrad {name}: building tile")
    desc, tile, sg, full_h = build_tile(sc, w, w.shard, keep_host=True)
    dyh = dy_box(w, sg)
    log(f"dense wgrad {name}: running")
    dw = host(run_wgrad(sc, w, desc, tile, sg, dev(dyh))).astype(np.float64)
    del tile
    lo, hi = cases.owned_box(sg)
    L = sg.g["out_ext"][0]
    ref = np.zeros((w.cout, w.cin) + tuple(w.K))
    CH = 8
    for p0 in range(0, L, CH):
        p1 = min(L, p0 + CH)
        l2, h2 = list(lo), list(hi)
        l2[0], h2[0] = lo[0] + p0, lo[0] + p1
        r0 = p0 * w.S[0] - sg.g["pad_lo"][0]
        r1 = (p1 - 1) * w.S[0] - sg.g["pad_lo"][0] + w.K[0]
        xw, origin = window_from_tile(w, sg, full_h, (r0, r1))
        ref += oconv.conv_wgrad_window(xw, origin, w.G, cases.to_ncdhw(cases.as_f64(dyh[:, p0:p1], w)), w.K, w.S,
                                       l2, h2)
        if p0 % (8 * CH) == 0:
            log(f"  oracle planes {p0}..{p1} of {L}")
    err = cases.norm_max_err(dw, ref)
    log(f"  dense wgrad {name}: normalised max err {err:.3e}")
    assert err <= cases.TOL[w.dtype]


def test_wgrad_status_word_reports_a_wait_that_gave_up(sc):
    """The W-march weight gradient hands stage buffers between its waves through
    bounded waits. With the bound forced down to one poll the waits give up at
    once (every kernel still runs to its end): the status word at the start of
    the workspace must say so and every dw element must be NaN. With the default
    bound the same call is clean and matches the first result."""
    import torch
    w = cases.REDUCED["c3r"]
    idx = w.shards()[1]
    desc, tile, sg, _ = build_tile(sc, w, idx)
    dyh = dev(dy_box(w, sg))
    O = sg.g["out_ext"]
    dw = torch.empty((w.cout, w.cin) + tuple(w.K), dtype=torch.float32, device="cuda")
    nbytes = sc.shard_conv_workspace_bytes(1, desc, sc.SHARD_BF16, w.cout, w.K, w.S, O)
    ws = torch.empty(nbytes, dtype=torch.uint8, device="cuda")

    def call():
        ws[:4].fill_(0xA5)
        sc.shard_conv_wgrad(desc, tile, dyh, w.cout, w.K, w.S, sg.g["pad_lo"], O, dw, ws)
        torch.cuda.synchronize()
        return int(ws[:4].view(torch.int32).item()), dw.clone()

    s0, d0 = call()
    assert s0 == 0 and bool(torch.isfinite(d0).all())
    with sc.call_opts(wait_polls=1):
        s1, d1 = call()
    assert s1 != 0
    assert bool(torch.isnan(d1).all())
    s2, d2 = call()
    assert s2 == 0 and torch.equal(d2, d0)
