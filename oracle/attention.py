"""One block step of ring attention (oracle; test infrastructure only).

Ring attention (section "Performance Benchmarks", subsection "Ring Attention")
shards the sequence: each device keeps its queries Q and computes scaled
dot-product attention against one key/value block at a time, passing K and V
around a ring of devices, and accumulates the softmax in log space so that
partial results over different blocks combine stably. One step on one device
is therefore: attention of the local queries against the block it holds, then
a log-space merge into the running result.

Definitions, per batch item, head and query row i (float64 NumPy; the only
library steps are matrix products):

    s[i, j]   = scale * q[i] . k[j]                     (j over the block's keys)
    lse_b[i]  = log sum_j exp(s[i, j])                  (-inf for an empty block)
    o_b[i]    = sum_j exp(s[i, j] - lse_b[i]) v[j]      (0 for an empty block)

and the merge of a running state (o, lse) with a block (o_b, lse_b):

    lse'[i]   = log(exp(lse[i]) + exp(lse_b[i]))
    o'[i]     = exp(lse[i] - lse'[i]) o[i] + exp(lse_b[i] - lse'[i]) o_b[i]

with the empty state o = 0, lse = -inf (a first step merges into it). After
the blocks of every device have been merged, o is softmax(scale q k^T) v over
the whole sequence and lse its log-normaliser. Arrays are [B][H][S][D] for
q, k, v, o and [B][H][S] for lse.
"""
from __future__ import annotations

import numpy as np


def block_attention(q, k, v, scale):
    """(o_b, lse_b) of queries q against the keys/values k, v of one block."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    shape = q.shape[:-1]
    if k.shape[-2] == 0:
        return np.zeros(shape + (v.shape[-1],)), np.full(shape, -np.inf)
    s = scale * np.matmul(q, np.swapaxes(k, -1, -2))
    m = s.max(axis=-1, keepdims=True)
    e = np.exp(s - m)
    tot = e.sum(axis=-1, keepdims=True)
    lse = (m + np.log(tot))[..., 0]
    return np.matmul(e / tot, v), lse


def merge(o, lse, o_b, lse_b):
    """Log-space merge of a running state with a block's result."""
    o, lse = np.asarray(o, dtype=np.float64), np.asarray(lse, dtype=np.float64)
    o_b, lse_b = np.asarray(o_b, dtype=np.float64), np.asarray(lse_b, dtype=np.float64)
    hi = np.maximum(lse, lse_b)
    safe = np.where(np.isneginf(hi), 0.0, hi)      # both empty: stay empty
    a = np.exp(lse - safe)
    b = np.exp(lse_b - safe)
    tot = a + b
    new_lse = np.where(tot > 0, safe + np.log(np.where(tot > 0, tot, 1.0)), -np.inf)
    wa = np.where(tot > 0, a / np.where(tot > 0, tot, 1.0), 0.0)[..., None]
    wb = np.where(tot > 0, b / np.where(tot > 0, tot, 1.0), 0.0)[..., None]
    return wa * o + wb * o_b, new_lse


def empty_state(q_shape, d_v):
    """The state before any block: o = 0, lse = -inf."""
    return np.zeros(tuple(q_shape[:-1]) + (d_v,)), np.full(tuple(q_shape[:-1]), -np.inf)


def ring_step(o, lse, q, k, v, scale):
    """One device's step: attention against the held block, merged in log space."""
    o_b, lse_b = block_attention(q, k, v, scale)
    return merge(o, lse, o_b, lse_b)


def full_attention(q, k, v, scale):
    """softmax(scale q k^T) v and its log-normaliser over all keys at once."""
    return block_attention(q, k, v, scale)
