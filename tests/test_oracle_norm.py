"""Pins for the oracle's domain-parallel group normalisation (CPU only): hand-
worked values, torch's float64 group_norm (a library routine), closed forms,
and the sharded pipeline (per-shard sums added over all shards, then each
interior normalised) against the whole-domain result.
"""
import itertools
import json
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import geometry, norm

GOLDEN = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "worked_examples.json")))


def test_hand_worked_values():
    c0, c1 = GOLDEN["group_norm"]
    x = np.array(c0["x"], dtype=np.float64).reshape(1, 1, -1)
    assert norm.sums(x, 1).reshape(-1).tolist() == c0["sums"]
    y = norm.group_norm(x, 1, c0["eps"], c0["gamma"], c0["beta"])
    np.testing.assert_allclose(y.reshape(-1) * np.sqrt(5.0), c0["y_times_sqrt5"], rtol=0, atol=1e-12)
    x = np.array(c1["x"], dtype=np.float64).reshape(1, 2, 2)
    assert norm.sums(x, 1).reshape(-1).tolist() == c1["sums"]
    y = norm.group_norm(x, 1, c1["eps"], c1["gamma"], c1["beta"])
    assert y.reshape(2, 2).tolist() == c1["y"]


@pytest.mark.parametrize("shape,groups", [((2, 6, 9), 3), ((1, 8, 5, 7), 2), ((2, 4, 3, 5, 6), 4),
                                          ((1, 32, 6, 5, 4), 8), ((1, 5, 11), 1), ((3, 6, 4, 4), 6)])
def test_vs_torch_group_norm_float64(shape, groups):
    rng = np.random.default_rng(len(shape) * 10 + groups)
    x = rng.normal(0.5, 2.0, size=shape)
    c = shape[1]
    gamma, beta = rng.uniform(0.5, 2, c), rng.uniform(-1, 1, c)
    ref = F.group_norm(torch.tensor(x), groups, torch.tensor(gamma), torch.tensor(beta), eps=1e-5).numpy()
    np.testing.assert_allclose(norm.group_norm(x, groups, 1e-5, gamma, beta), ref, rtol=1e-10, atol=1e-10)


def test_constant_input_gives_beta():
    x = np.full((2, 4, 5, 6), 3.25)
    beta = np.array([0.5, -1.0, 2.0, 0.0])
    y = norm.group_norm(x, 2, 1e-5, np.ones(4), beta)
    assert np.array_equal(y, np.broadcast_to(beta.reshape(1, 4, 1, 1), y.shape))


def test_two_values_give_unit_variance():
    """Half +a, half -a per group: mean 0, variance a^2."""
    a = 1.5
    x = np.tile(np.array([a, -a]), (1, 2, 8)).reshape(1, 2, 16)
    y = norm.group_norm(x, 1, 0.0, np.ones(2), np.zeros(2))
    np.testing.assert_allclose(np.abs(y), 1.0, rtol=0, atol=1e-15)


def _splits(G, parts):
    sizes = geometry.chunk_sizes(G, parts)
    return list(zip(geometry.offsets(sizes), sizes))


@pytest.mark.parametrize("G,parts,groups", [((16,), (3,), 2), ((12, 10), (2, 3), 4), ((9, 10, 7), (2, 2, 1), 1),
                                            ((11, 8, 6), (4, 1, 2), 8)])
@pytest.mark.parametrize("integer", [True, False])
def test_shard_sums_and_normalisation_match_the_whole_domain(G, parts, groups, integer):
    rng = np.random.default_rng(sum(G) + groups)
    shape = (2, 8) + G
    x = rng.integers(-2, 3, size=shape).astype(np.float64) if integer else rng.normal(size=shape)
    gamma, beta = rng.uniform(0.5, 2, 8), rng.uniform(-1, 1, 8)
    full = norm.sums(x, groups)
    boxes = [tuple(slice(o, o + e) for o, e in s) for s in itertools.product(*[_splits(G[a], parts[a])
                                                                              for a in range(len(G))])]
    total = np.zeros_like(full)
    for b in boxes:
        total += norm.sums(x[(slice(None), slice(None)) + b], groups)
    if integer:
        assert np.array_equal(total, full)
    else:
        np.testing.assert_allclose(total, full, rtol=1e-13, atol=1e-12)
    count = x.size // (x.shape[0] * groups)
    y = norm.group_norm(x, groups, 1e-5, gamma, beta)
    for b in boxes:
        sl = (slice(None), slice(None)) + b
        np.testing.assert_allclose(norm.normalise(x[sl], total, count, 1e-5, gamma, beta, groups), y[sl],
                                   rtol=1e-12, atol=1e-12)
