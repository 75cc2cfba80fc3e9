"""Pins of the ring-attention oracle (oracle.attention) against things other
than itself: a hand-worked two-key example in closed form, scalar loops over
the definition, torch's float64 CPU scaled-dot-product attention, the ring
invariant (merging the blocks of any split of the keys, in any order, gives
attention over all keys), and the degenerate cases."""
import itertools
import math

import numpy as np
import pytest

from oracle import attention as oat


def test_hand_worked_two_keys():
    # q = (1, 0), keys e0 and e1, scale 1: scores 1 and 0
    q = np.array([[[[1.0, 0.0]]]])
    k = np.array([[[[1.0, 0.0], [0.0, 1.0]]]])
    v = np.array([[[[1.0, 2.0], [3.0, 4.0]]]])
    o, lse = oat.block_attention(q, k, v, 1.0)
    e = math.e
    w0, w1 = e / (1 + e), 1 / (1 + e)
    assert lse[0, 0, 0] == pytest.approx(math.log(1 + e), abs=1e-15)
    assert o[0, 0, 0] == pytest.approx([w0 * 1 + w1 * 3, w0 * 2 + w1 * 4], abs=1e-15)


def _loops(q, k, v, scale):
    B, H, S, D = q.shape
    o = np.zeros((B, H, S, v.shape[-1]))
    lse = np.zeros((B, H, S))
    for b, h, i in itertools.product(range(B), range(H), range(S)):
        s = [scale * sum(q[b, h, i, d] * k[b, h, j, d] for d in range(D)) for j in range(k.shape[2])]
        m = max(s)
        z = sum(math.exp(x - m) for x in s)
        lse[b, h, i] = m + math.log(z)
        for e in range(v.shape[-1]):
            o[b, h, i, e] = sum(math.exp(s[j] - m) / z * v[b, h, j, e] for j in range(len(s)))
    return o, lse


def _rand(rng, *shape):
    return rng.standard_normal(shape)


def test_scalar_loops():
    rng = np.random.default_rng(0)
    q, k, v = _rand(rng, 1, 2, 3, 4), _rand(rng, 1, 2, 5, 4), _rand(rng, 1, 2, 5, 3)
    o, lse = oat.block_attention(q, k, v, 0.7)
    o2, lse2 = _loops(q, k, v, 0.7)
    assert np.allclose(o, o2, atol=1e-13) and np.allclose(lse, lse2, atol=1e-13)


def test_torch_sdpa_float64():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(1)
    q, k, v = _rand(rng, 2, 3, 17, 16), _rand(rng, 2, 3, 29, 16), _rand(rng, 2, 3, 29, 16)
    scale = 1 / math.sqrt(16)
    o, lse = oat.block_attention(q, k, v, scale)
    tq, tk, tv = (torch.from_numpy(a) for a in (q, k, v))
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, scale=scale).numpy()
    ref_lse = torch.logsumexp(scale * tq @ tk.transpose(-1, -2), dim=-1).numpy()
    assert np.allclose(o, ref, atol=1e-12) and np.allclose(lse, ref_lse, atol=1e-12)


@pytest.mark.parametrize("seed", range(6))
def test_ring_of_blocks_equals_full_attention(seed):
    """Any split of the keys into blocks (empty and one-key blocks included),
    merged in any order from the empty state, gives full attention."""
    rng = np.random.default_rng(10 + seed)
    S, D = 37, 8
    q, k, v = _rand(rng, 1, 2, 11, D), 3 * _rand(rng, 1, 2, S, D), _rand(rng, 1, 2, S, D)
    scale = 0.5
    cuts = sorted(rng.choice(np.arange(0, S + 1), size=5, replace=True))
    bounds = [0] + list(cuts) + [S]
    blocks = [(a, b) for a, b in zip(bounds[:-1], bounds[1:])]
    rng.shuffle(blocks)
    o, lse = oat.empty_state(q.shape, D)
    for a, b in blocks:
        o, lse = oat.ring_step(o, lse, q, k[:, :, a:b], v[:, :, a:b], scale)
    full_o, full_lse = oat.full_attention(q, k, v, scale)
    assert np.allclose(o, full_o, atol=1e-12) and np.allclose(lse, full_lse, atol=1e-12)


def test_degenerate_cases():
    rng = np.random.default_rng(3)
    q, v = _rand(rng, 1, 1, 4, 6), _rand(rng, 1, 1, 1, 6)
    k = _rand(rng, 1, 1, 1, 6)
    o, lse = oat.block_attention(q, k, v, 0.3)
    assert np.allclose(o, np.broadcast_to(v, o.shape), atol=1e-15)          # one key: its value
    assert np.allclose(lse, 0.3 * (q @ k[0, 0, 0])[..., ], atol=1e-15)
    k8, v8 = _rand(rng, 1, 1, 8, 6), _rand(rng, 1, 1, 8, 6)
    o, lse = oat.block_attention(np.zeros((1, 1, 4, 6)), k8, v8, 1.0)     # equal scores: the mean
    assert np.allclose(o, v8.mean(axis=2, keepdims=True), atol=1e-15)
    assert np.allclose(lse, math.log(8), atol=1e-15)
    e_o, e_lse = oat.block_attention(q, np.zeros((1, 1, 0, 6)), np.zeros((1, 1, 0, 6)), 1.0)
    assert np.all(e_o == 0) and np.all(np.isneginf(e_lse))                  # empty block
    s_o, s_lse = oat.block_attention(q, k8, v8, 1.0)
    o2, l2 = oat.merge(s_o, s_lse, e_o, e_lse)                              # merging nothing
    assert np.array_equal(o2, s_o) and np.array_equal(l2, s_lse)
    o3, l3 = oat.merge(*oat.empty_state(q.shape, 6), s_o, s_lse)             # into the empty state
    assert np.array_equal(o3, s_o) and np.array_equal(l3, s_lse)
    o4, l4 = oat.merge(*oat.empty_state(q.shape, 6), e_o, e_lse)             # empty and empty
    assert np.all(o4 == 0) and np.all(np.isneginf(l4))


def test_merge_is_symmetric_and_associative():
    rng = np.random.default_rng(4)
    st = [(rng.standard_normal((2, 3, 5)), rng.standard_normal((2, 3)) * 4) for _ in range(3)]
    ab = oat.merge(*st[0], *st[1])
    ba = oat.merge(*st[1], *st[0])
    assert np.allclose(ab[0], ba[0], atol=1e-14) and np.allclose(ab[1], ba[1], atol=1e-14)
    left = oat.merge(*ab, *st[2])
    right = oat.merge(*st[0], *oat.merge(*st[1], *st[2]))
    assert np.allclose(left[0], right[0], atol=1e-13) and np.allclose(left[1], right[1], atol=1e-13)
