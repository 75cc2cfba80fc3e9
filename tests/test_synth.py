"""The seeded generator: reproducible, box-consistent, with the stated moments.

These checks concern input generation only (no method arithmetic)."""
import numpy as np
import pytest

import synth


def test_same_seed_same_bits_and_streams_differ():
    f = synth.Field((1, 3, 9, 10), synth.NORMAL, (0, 1), stream=synth.STREAM_X)
    a, b = f.box(), f.box()
    assert np.array_equal(a, b)
    g = synth.Field((1, 3, 9, 10), synth.NORMAL, (0, 1), stream=synth.STREAM_DY)
    assert not np.array_equal(a, g.box())
    h = synth.Field((1, 3, 9, 10), synth.NORMAL, (0, 1), seed=1)
    assert not np.array_equal(a, h.box())


@pytest.mark.parametrize("dist,params", [(synth.UNIFORM, (-1, 1)), (synth.NORMAL, (0, 1)),
                                         (synth.SMOOTH, (0, 1, 1.5)), (synth.INT, (-2, 2)),
                                         (synth.SPARSE_INT, (-2, 2, 0.1))])
@pytest.mark.parametrize("out", [synth.OUT_F64, synth.OUT_F32, synth.OUT_BF16])
def test_sub_box_equals_slice_of_full(dist, params, out):
    f = synth.Field((2, 3, 11, 9, 13), dist, params)
    full = f.box(out=out)
    part = f.box(lo=(1, 1, 2, 0, 5), hi=(2, 3, 9, 7, 13), out=out)
    assert np.array_equal(part, full[1:2, 2:9, 0:7, 5:13, 1:3])


def test_outside_domain_is_zero_and_inside_matches():
    f = synth.Field((1, 2, 6, 7), synth.SMOOTH, (0, 1, 1.0))
    full = f.box()
    ext = f.box(lo=(0, 0, -2, -1), hi=(1, 2, 8, 7))
    assert np.all(ext[:, :2] == 0) and np.all(ext[:, 8:] == 0) and np.all(ext[:, :, :1] == 0)
    assert np.array_equal(ext[:, 2:8, 1:8], full)


def test_moments():
    u = synth.Field((1, 4, 128, 128), synth.UNIFORM, (-1, 1)).box()
    assert abs(u.mean()) < 0.01 and abs(u.var() - 1 / 3) < 0.01 and u.min() >= -1 and u.max() < 1
    n = synth.Field((1, 4, 128, 128), synth.NORMAL, (0, 1)).box()
    assert abs(n.mean()) < 0.01 and abs(n.std() - 1) < 0.01
    m4 = np.mean(n ** 4)
    assert abs(m4 - 3) < 0.1
    w = synth.Field((1, 4, 128, 128), synth.NORMAL, (0, 1 / 24)).box()
    assert abs(w.std() * 24 - 1) < 0.02
    i = synth.Field((1, 4, 64, 64), synth.INT, (-2, 2)).box()
    assert set(np.unique(i).tolist()) == {-2, -1, 0, 1, 2}
    sp = synth.Field((1, 4, 128, 128), synth.SPARSE_INT, (1, 2, 1 / 64)).box()
    frac = np.count_nonzero(sp) / sp.size
    assert abs(frac - 1 / 64) < 0.003


def test_smooth_field_unit_variance_and_correlated():
    f = synth.Field((1, 2, 64, 64, 64), synth.SMOOTH, (0, 1, 2.0))
    s = f.box()
    assert abs(s.std() - 1) < 0.15 and abs(s.mean()) < 0.15
    # neighbours along every axis are strongly correlated (Gaussian width 2 voxels)
    for ax in (1, 2, 3):
        a = np.take(s, np.arange(0, 63), axis=ax).reshape(-1)
        b = np.take(s, np.arange(1, 64), axis=ax).reshape(-1)
        assert np.corrcoef(a, b)[0, 1] > 0.8
    # periodic: the field wraps, so the first and last planes are neighbours too
    a = s[:, 0].reshape(-1)
    b = s[:, -1].reshape(-1)
    assert np.corrcoef(a, b)[0, 1] > 0.8


def test_bf16_round_to_nearest_even_ties():
    vals = np.array([
        1.0,
        1.0 + 2 ** -8,                # exact tie between 1.0 and 1.0078125 -> even (1.0)
        1.0 + 3 * 2 ** -8,            # tie between 1.0078125 and 1.015625 -> even (1.015625)
        1.0 + 2 ** -8 + 2 ** -20,     # just above the tie -> up
        -(1.0 + 2 ** -8),             # negative tie -> even
        3.0e38,                        # rounds to the largest finite bfloat16 neighbour
    ], dtype=np.float32)
    got = synth.bf16_to_f64(synth.round_bf16(vals))
    want = [1.0, 1.0, 1.015625, 1.0078125, -1.0]
    assert got[:5].tolist() == want
    assert np.isfinite(got[5]) or got[5] == np.inf


def test_bf16_output_is_rounded_f32_output():
    f = synth.Field((1, 3, 17, 19), synth.NORMAL, (0, 1))
    f32 = f.box(out=synth.OUT_F32)
    b = f.box(out=synth.OUT_BF16)
    assert np.array_equal(b, synth.round_bf16(f32))
    np.testing.assert_allclose(synth.bf16_to_f64(b), f32, rtol=2 ** -8)


def test_oracle_output_rounding_matches_generator_rounding_and_ties():
    """Two independent bf16 rounding implementations (oracle numpy, generator C)
    agree on random values and on hand-picked ties."""
    from oracle import conv
    rng = np.random.default_rng(0)
    v = np.concatenate([rng.normal(size=5000) * 10.0 ** rng.integers(-5, 6, size=5000),
                        [1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -(1.0 + 2 ** -8), 255.0, 257.0, 259.0]])
    assert np.array_equal(conv.round_bf16(v), synth.round_bf16(v.astype(np.float32)))
    got = conv.bf16_value(conv.round_bf16(np.array([257.0, 259.0, 1.0 + 2 ** -8])))
    assert got.tolist() == [256.0, 260.0, 1.0]   # ties to even: 257 -> 256, 259 -> 260
