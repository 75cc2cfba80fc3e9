"""Scalar-loop and dense-matrix restatements of the convolution (oracle; test
infrastructure only). Pure Python loops, for tiny inputs: they pin the
vectorised oracle in ``conv`` by a second, independent transcription of the
same definition (see ``conv`` for the definition and its citation).
"""
from __future__ import annotations

import itertools

import numpy as np


def _out_len(G, K, S):
    return (G + (K - 1) - K) // S + 1


def conv_scalar(x, w, stride):
    """y[n][co][j] = sum over ci, t of w[co][ci][t] * x[n][ci][j*S - P + t], x = 0 outside."""
    N, Ci = x.shape[:2]
    Co = w.shape[0]
    G, K = x.shape[2:], w.shape[2:]
    nd = len(G)
    n_out = [_out_len(G[a], K[a], stride[a]) for a in range(nd)]
    y = np.zeros([N, Co] + n_out)
    for n in range(N):
        for co in range(Co):
            for j in itertools.product(*[range(m) for m in n_out]):
                acc = 0.0
                for ci in range(Ci):
                    for t in itertools.product(*[range(k) for k in K]):
                        src = [j[a] * stride[a] - (K[a] - 1) // 2 + t[a] for a in range(nd)]
                        if all(0 <= src[a] < G[a] for a in range(nd)):
                            acc += float(w[(co, ci) + t]) * float(x[(n, ci) + tuple(src)])
                y[(n, co) + j] = acc
    return y


def wgrad_scalar(x, dy, kernel, stride, out_lo, out_hi):
    """dW[co][ci][t] = sum over n and owned outputs j of dy[n][co][j] * x[n][ci][j*S - P + t]."""
    N, Ci = x.shape[:2]
    Co = dy.shape[1]
    G = x.shape[2:]
    nd = len(G)
    dw = np.zeros([Co, Ci] + list(kernel))
    for co in range(Co):
        for ci in range(Ci):
            for t in itertools.product(*[range(k) for k in kernel]):
                acc = 0.0
                for n in range(N):
                    for j in itertools.product(*[range(l, h) for l, h in zip(out_lo, out_hi)]):
                        src = [j[a] * stride[a] - (kernel[a] - 1) // 2 + t[a] for a in range(nd)]
                        if all(0 <= src[a] < G[a] for a in range(nd)):
                            jj = tuple(j[a] - out_lo[a] for a in range(nd))
                            acc += float(dy[(n, co) + jj]) * float(x[(n, ci) + tuple(src)])
                dw[(co, ci) + t] = acc
    return dw


def dgrad_scalar(dy, w, G, stride):
    """dx[n][ci][i] = sum over co, t and outputs j with j*S - P + t = i of
    w[co][ci][t] * dy[n][co][j]: every (output, tap) pair adds its term to the
    input it was read from, inputs outside the domain dropped."""
    N, Co = dy.shape[:2]
    Ci = w.shape[1]
    K = w.shape[2:]
    nd = len(G)
    n_out = dy.shape[2:]
    dx = np.zeros([N, Ci] + list(G))
    for n in range(N):
        for co in range(Co):
            for j in itertools.product(*[range(m) for m in n_out]):
                for t in itertools.product(*[range(k) for k in K]):
                    src = [j[a] * stride[a] - (K[a] - 1) // 2 + t[a] for a in range(nd)]
                    if all(0 <= src[a] < G[a] for a in range(nd)):
                        for ci in range(Ci):
                            dx[(n, ci) + tuple(src)] += float(w[(co, ci) + t]) * float(dy[(n, co) + j])
    return dx


def toeplitz(w, G, stride):
    """Dense matrix T with vec(y[n]) = T @ vec(x[n]) for one batch item, built entry
    by entry: T[(co, j), (ci, i)] = w[co, ci, i - j*S + P] when that tap exists."""
    Co, Ci = w.shape[:2]
    K = w.shape[2:]
    nd = len(G)
    n_out = [_out_len(G[a], K[a], stride[a]) for a in range(nd)]
    rows = Co * int(np.prod(n_out))
    cols = Ci * int(np.prod(G))
    T = np.zeros((rows, cols))
    out_idx = list(itertools.product(*[range(m) for m in n_out]))
    in_idx = list(itertools.product(*[range(g) for g in G]))
    for co in range(Co):
        for r, j in enumerate(out_idx):
            for ci in range(Ci):
                for c, i in enumerate(in_idx):
                    t = [i[a] - j[a] * stride[a] + (K[a] - 1) // 2 for a in range(nd)]
                    if all(0 <= t[a] < K[a] for a in range(nd)):
                        T[co * len(out_idx) + r, ci * len(in_idx) + c] = w[(co, ci) + tuple(t)]
    return T
