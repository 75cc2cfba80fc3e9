"""Pins for the oracle's convolution and weight gradient (CPU only).

Each check ties the vectorised oracle to something other than itself: values
worked by hand, a scalar-loop transcription, a dense Toeplitz matrix, torch's
float64 CPU convolution (a library routine), closed forms and invariants.
"""
import itertools
import json
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import brute, conv, geometry

GOLDEN = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "worked_examples.json")))


def rnd(rng, shape, integer=False):
    if integer:
        return rng.integers(-2, 3, size=shape).astype(np.float64)
    return rng.uniform(-1, 1, size=shape)


# shapes: (nd, N, Ci, Co, G, K, S)
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


@pytest.mark.parametrize("case", GOLDEN["conv1d"], ids=lambda c: c["what"][:40])
def test_hand_worked_1d(case):
    x = np.array(case["x"], dtype=np.float64).reshape(1, 1, -1)
    w = np.array(case["w"], dtype=np.float64).reshape(1, 1, -1)
    y = conv.conv_forward(x, w, (case["stride"],))
    assert y.reshape(-1).tolist() == case["y"]


@pytest.mark.parametrize("shape", TINY)
@pytest.mark.parametrize("integer", [True, False])
def test_forward_vs_scalar_loops(shape, integer):
    nd, N, Ci, Co, G, K, S = shape
    rng = np.random.default_rng(hash((shape, integer)) % 2**32)
    x = rnd(rng, (N, Ci) + G, integer)
    w = rnd(rng, (Co, Ci) + K, integer)
    y = conv.conv_forward(x, w, S)
    yb = brute.conv_scalar(x, w, S)
    if integer:
        assert np.array_equal(y, yb)
    else:
        np.testing.assert_allclose(y, yb, rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("shape", TINY[:6])
def test_forward_vs_toeplitz(shape):
    nd, N, Ci, Co, G, K, S = shape
    rng = np.random.default_rng(7)
    x = rnd(rng, (N, Ci) + G)
    w = rnd(rng, (Co, Ci) + K)
    T = brute.toeplitz(w, G, S)
    y = conv.conv_forward(x, w, S)
    for n in range(N):
        np.testing.assert_allclose(y[n].reshape(-1), T @ x[n].reshape(-1), rtol=1e-12, atol=1e-13)


TORCH_CASES = TINY + [
    (2, 1, 4, 5, (17, 13), (3, 3), (1, 1)),
    (3, 1, 3, 4, (9, 8, 10), (5, 5, 5), (1, 1, 1)),
    (3, 2, 4, 3, (11, 9, 7), (3, 3, 3), (2, 2, 2)),
    (2, 1, 3, 2, (10, 11), (7, 3), (3, 2)),
]


@pytest.mark.parametrize("shape", TORCH_CASES)
def test_forward_vs_torch_float64(shape):
    nd, N, Ci, Co, G, K, S = shape
    rng = np.random.default_rng(11)
    x = rnd(rng, (N, Ci) + G)
    w = rnd(rng, (Co, Ci) + K)
    fn = {1: F.conv1d, 2: F.conv2d, 3: F.conv3d}[nd]
    ref = fn(torch.from_numpy(x), torch.from_numpy(w), stride=S, padding=tuple((k - 1) // 2 for k in K)).numpy()
    np.testing.assert_allclose(conv.conv_forward(x, w, S), ref, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("shape", TORCH_CASES)
def test_wgrad_vs_torch_float64(shape):
    nd, N, Ci, Co, G, K, S = shape
    rng = np.random.default_rng(13)
    x = rnd(rng, (N, Ci) + G)
    n_out = [geometry.out_len(G[a], K[a], S[a]) for a in range(nd)]
    dy = rnd(rng, (N, Co) + tuple(n_out))
    fn = {1: torch.nn.grad.conv1d_weight, 2: torch.nn.grad.conv2d_weight, 3: torch.nn.grad.conv3d_weight}[nd]
    ref = fn(torch.from_numpy(x), (Co, Ci) + K, torch.from_numpy(dy), stride=S,
             padding=tuple((k - 1) // 2 for k in K)).numpy()
    np.testing.assert_allclose(conv.conv_wgrad(x, dy, K, S), ref, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("shape", TINY)
def test_wgrad_vs_scalar_loops_on_a_box(shape):
    nd, N, Ci, Co, G, K, S = shape
    rng = np.random.default_rng(17)
    x = rnd(rng, (N, Ci) + G, integer=True)
    n_out = [geometry.out_len(G[a], K[a], S[a]) for a in range(nd)]
    lo = [m // 3 for m in n_out]
    hi = [max(l + 1, m - m // 4) for l, m in zip(lo, n_out)]
    dy = rnd(rng, (N, Co) + tuple(h - l for l, h in zip(lo, hi)), integer=True)
    got = conv.conv_wgrad(x, dy, K, S, lo, hi)
    assert np.array_equal(got, brute.wgrad_scalar(x, dy, K, S, lo, hi))


@pytest.mark.parametrize("nd,S", [(1, 1), (2, 2), (3, 1), (3, 2), (2, 3)])
def test_delta_kernel_gives_a_shift(nd, S):
    """w = e_{co=ci, t}: y[n, c, j] = x[n, c, j*S + t - P] (0 outside the domain)."""
    rng = np.random.default_rng(nd * 10 + S)
    G = (9, 7, 8)[:nd]
    K = (5, 3, 3)[:nd]
    x = rnd(rng, (1, 2) + G)
    for t in itertools.product(*[range(k) for k in K]):
        w = np.zeros((2, 2) + K)
        for c in range(2):
            w[(c, c) + t] = 1.0
        y = conv.conv_forward(x, w, (S,) * nd)
        for j in itertools.product(*[range(m) for m in y.shape[2:]]):
            src = [j[a] * S + t[a] - (K[a] - 1) // 2 for a in range(nd)]
            inside = all(0 <= src[a] < G[a] for a in range(nd))
            for c in range(2):
                want = x[(0, c) + tuple(src)] if inside else 0.0
                assert y[(0, c) + j] == want


@pytest.mark.parametrize("nd,S", [(1, 2), (2, 1), (3, 1), (3, 2)])
def test_constant_input_counts_in_bounds_taps(nd, S):
    """x = c, w = 1: y = c * Ci * prod_a #{t : 0 <= j*S - P + t < G}."""
    G = (6, 9, 5)[:nd]
    K = (3, 5, 3)[:nd]
    Ci, c = 3, 1.5
    x = np.full((1, Ci) + G, c)
    w = np.ones((2, Ci) + K)
    y = conv.conv_forward(x, w, (S,) * nd)
    for j in itertools.product(*[range(m) for m in y.shape[2:]]):
        cnt = 1
        for a in range(nd):
            P = (K[a] - 1) // 2
            cnt *= sum(1 for t in range(K[a]) if 0 <= j[a] * S - P + t < G[a])
        assert y[(0, 0) + j] == c * Ci * cnt and y[(0, 1) + j] == c * Ci * cnt


def test_linearity():
    rng = np.random.default_rng(3)
    x1, x2 = rnd(rng, (1, 3, 8, 7, 6)), rnd(rng, (1, 3, 8, 7, 6))
    w1, w2 = rnd(rng, (2, 3, 3, 3, 3)), rnd(rng, (2, 3, 3, 3, 3))
    S = (1, 2, 1)
    f = lambda x, w: conv.conv_forward(x, w, S)
    np.testing.assert_allclose(f(2 * x1 - x2, w1), 2 * f(x1, w1) - f(x2, w1), atol=1e-12)
    np.testing.assert_allclose(f(x1, w1 + 3 * w2), f(x1, w1) + 3 * f(x1, w2), atol=1e-12)


@pytest.mark.parametrize("nd,S", [(1, 1), (2, 2), (3, 1), (3, 3)])
def test_adjoint_identity(nd, S):
    """<conv(x; w), dy> = <w, wgrad(x, dy)> (the weight gradient is the adjoint in w)."""
    rng = np.random.default_rng(nd + 100 * S)
    G = (10, 9, 8)[:nd]
    K = (3, 5, 3)[:nd]
    x = rnd(rng, (2, 3) + G)
    w = rnd(rng, (4, 3) + K)
    y = conv.conv_forward(x, w, (S,) * nd)
    dy = rnd(rng, y.shape)
    lhs = float(np.sum(y * dy))
    rhs = float(np.sum(w * conv.conv_wgrad(x, dy, K, (S,) * nd)))
    assert abs(lhs - rhs) <= 1e-11 * max(1.0, abs(lhs))


@pytest.mark.parametrize("nd,S", [(1, 2), (2, 1), (3, 2)])
def test_wgrad_ones_closed_form(nd, S):
    """x = 1, dy = 1 over a box: dW[co, ci, t] = prod_a #{j in box : 0 <= j*S - P + t_a < G}."""
    G = (9, 8, 7)[:nd]
    K = (3, 5, 3)[:nd]
    n_out = [geometry.out_len(G[a], K[a], S) for a in range(nd)]
    lo = [1] * nd
    hi = [m for m in n_out]
    x = np.ones((1, 2) + G)
    dy = np.ones((1, 3) + tuple(h - l for l, h in zip(lo, hi)))
    dw = conv.conv_wgrad(x, dy, K, (S,) * nd, lo, hi)
    for t in itertools.product(*[range(k) for k in K]):
        cnt = 1
        for a in range(nd):
            P = (K[a] - 1) // 2
            cnt *= sum(1 for j in range(lo[a], hi[a]) if 0 <= j * S - P + t[a] < G[a])
        assert np.all(dw[(slice(None), slice(None)) + t] == cnt)


def test_output_box_restriction_matches_full():
    """Computing only a box of outputs (what the big workloads do) equals slicing
    the full result: bitwise on integer data, to rounding on real data."""
    rng = np.random.default_rng(5)
    for integer in (True, False):
        x = rnd(rng, (1, 3, 12, 10, 9), integer)
        w = rnd(rng, (2, 3, 3, 3, 3), integer)
        S = (1, 1, 2)
        full = conv.conv_forward(x, w, S)
        lo, hi = (3, 0, 1), (8, 10, 4)
        part = conv.conv_forward(x, w, S, lo, hi)
        want = full[:, :, 3:8, 0:10, 1:4]
        if integer:
            assert np.array_equal(part, want)
        else:
            np.testing.assert_allclose(part, want, rtol=1e-14, atol=1e-14)


def test_window_with_outside_values_is_zeroed():
    """A window that reaches outside the domain is treated as zero there, whatever
    values the caller put in it (the definition's zero padding)."""
    rng = np.random.default_rng(9)
    x = rnd(rng, (1, 2, 8, 6))
    w = rnd(rng, (3, 2, 3, 3))
    full = conv.conv_forward(x, w, (1, 1))
    xw = np.full((1, 2, 10, 8), 123.0)
    xw[:, :, 1:9, 1:7] = x
    part = conv.conv_forward_window(xw, (-1, -1), (8, 6), w, (1, 1), (0, 0), (8, 6))
    np.testing.assert_allclose(part, full, rtol=1e-14, atol=1e-14)
