"""Domain-parallel group normalisation (oracle; test infrastructure only).

A normalisation layer on a sharded tensor must aggregate its statistics over
all shards before it can normalise (ShardTensor section "PyTorch Dispatch",
next to the halo operation). Reading used here: group normalisation of a
[N][C][*spatial] tensor with G groups of C / G consecutive channels - per batch
item and group, the mean and variance run over the group's channels and the
whole spatial domain (G = C is instance normalisation, G = 1 normalises over
all channels and space); with domain parallelism below batch size one this is
the statistic a layer needs across ranks. Definition:

    mean[n, g] = S1 / cnt,   var[n, g] = S2 / cnt - mean^2   (biased variance)
    S1 = sum x,  S2 = sum x^2  over c in group g and all spatial positions
    y[n, c, i] = (x[n, c, i] - mean[n, g(c)]) / sqrt(var[n, g(c)] + eps) * gamma[c] + beta[c]

A shard contributes the sums S1, S2 over its interior; the sums of all shards
are the full-domain sums (the all-reduce), after which each shard normalises
its interior. Everything is float64 NumPy.
"""
from __future__ import annotations

import numpy as np


def _groups(x, groups):
    n, c = x.shape[:2]
    if groups < 1 or c % groups != 0:
        raise ValueError("groups must divide the channel count")
    return x.reshape((n, groups, c // groups) + x.shape[2:])


def sums(x, groups) -> np.ndarray:
    """[N][G][2]: the sums S1, S2 of x (logical [N][C][*spatial]) per batch item
    and channel group, over the group's channels and every position of x."""
    xg = _groups(np.asarray(x, dtype=np.float64), groups)
    red = tuple(range(2, xg.ndim))
    return np.stack([xg.sum(axis=red), (xg * xg).sum(axis=red)], axis=-1)


def normalise(x, s, count, eps, gamma, beta, groups) -> np.ndarray:
    """y from x and the full-domain sums s ([N][G][2]) over `count` elements per
    (batch item, group)."""
    x = np.asarray(x, dtype=np.float64)
    n, c = x.shape[:2]
    mean = s[..., 0] / count
    var = np.maximum(s[..., 1] / count - mean * mean, 0.0)
    rstd = 1.0 / np.sqrt(var + eps)
    per_c = c // groups
    m = np.repeat(mean, per_c, axis=1).reshape((n, c) + (1,) * (x.ndim - 2))
    r = np.repeat(rstd, per_c, axis=1).reshape((n, c) + (1,) * (x.ndim - 2))
    g = np.asarray(gamma, dtype=np.float64).reshape((1, c) + (1,) * (x.ndim - 2))
    b = np.asarray(beta, dtype=np.float64).reshape((1, c) + (1,) * (x.ndim - 2))
    return (x - m) * r * g + b


def group_norm(x, groups, eps, gamma, beta) -> np.ndarray:
    """Group normalisation of the whole domain."""
    x = np.asarray(x, dtype=np.float64)
    count = x.size // (x.shape[0] * groups)
    return normalise(x, sums(x, groups), count, eps, gamma, beta, groups)
