"""GPU parity of the ring-attention block step (shard_attn_block) against the
float64 oracle (oracle.attention).

The oracle runs on the same bf16-rounded q, k, v. Bars: the output to the bf16
tolerance (normalised max error <= 2e-2: the probabilities enter the second
product rounded to bf16), the log-normaliser to 1e-4 relative; a ring of
several blocks (empty and one-key blocks included) merged step by step equals
attention over the whole key sequence.
"""
import math

import numpy as np
import pytest

import shard_cases as cases
from gpu_util import log
from oracle import attention as oat

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sc():
    import torch
    assert torch.cuda.is_available()
    from paper_2605_11111_amd import shardconv
    return shardconv


def _bf16(rng, shape, scale=1.0):
    """bf16 device tensor and its exact float64 values."""
    import torch
    t = (torch.from_numpy(rng.standard_normal(shape) * scale).float()).to(torch.bfloat16)
    return t.cuda(), t.double().numpy()


def _state(B, H, S, D):
    import torch
    return (torch.full((B, H, S, D), float("nan"), device="cuda"),
            torch.full((B, H, S), float("nan"), device="cuda"))


def _check(o, lse, ref_o, ref_lse):
    got_o = o.cpu().double().numpy()
    got_l = lse.cpu().double().numpy()
    err = cases.norm_max_err(got_o, ref_o)
    lerr = float(np.max(np.abs(got_l - ref_lse) / np.maximum(1.0, np.abs(ref_lse))))
    assert np.all(np.isfinite(got_o)) and err <= 2e-2, err
    assert lerr <= 1e-4, lerr
    return err, lerr


SHAPES = [
    # (B, H, Sq, Sk, D)
    (1, 2, 256, 256, 128),
    (2, 3, 300, 77, 128),      # ragged queries and keys
    (1, 1, 5, 1000, 64),       # few queries, many keys
    (2, 2, 513, 33, 64),
    (1, 4, 1, 1, 128),         # one query, one key
]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_single_block_from_empty_state(sc, shape):
    B, H, Sq, Sk, D = shape
    rng = np.random.default_rng(sum(shape))
    q, q64 = _bf16(rng, (B, H, Sq, D))
    k, k64 = _bf16(rng, (B, H, Sk, D))
    v, v64 = _bf16(rng, (B, H, Sk, D))
    scale = 1 / math.sqrt(D)
    o, lse = _state(B, H, Sq, D)
    sc.shard_attn_block(q, k, v, o, lse, scale, True)
    ref_o, ref_l = oat.block_attention(q64, k64, v64, scale)
    log(f"attn {shape}: err {_check(o, lse, ref_o, ref_l)}")


@pytest.mark.parametrize("D", [64, 128])
def test_ring_of_blocks_equals_full_attention(sc, D):
    """The K/V sequence split in uneven blocks (an empty one and a one-key one
    among them) and merged step by step gives attention over all keys; the
    oracle's own ring of the same blocks agrees."""
    import torch
    B, H, Sq, S = 1, 3, 400, 700
    rng = np.random.default_rng(D)
    q, q64 = _bf16(rng, (B, H, Sq, D))
    k, k64 = _bf16(rng, (B, H, S, D), 1.5)
    v, v64 = _bf16(rng, (B, H, S, D))
    scale = 1 / math.sqrt(D)
    bounds = [0, 130, 130, 131, 400, 700]
    o, lse = _state(B, H, Sq, D)
    ro, rl = oat.empty_state(q64.shape, D)
    for i, (a, b) in enumerate(zip(bounds[:-1], bounds[1:])):
        sc.shard_attn_block(q, k[:, :, a:b].contiguous(), v[:, :, a:b].contiguous(), o, lse, scale, i == 0)
        ro, rl = oat.ring_step(ro, rl, q64, k64[:, :, a:b], v64[:, :, a:b], scale)
    torch.cuda.synchronize()
    full_o, full_l = oat.full_attention(q64, k64, v64, scale)
    assert np.allclose(ro, full_o, atol=1e-12)
    _check(o, lse, full_o, full_l)


def test_empty_block(sc):
    """An empty first block gives the empty state; an empty later block leaves
    the state as it was (bit for bit)."""
    import torch
    B, H, Sq, D = 1, 2, 70, 64
    rng = np.random.default_rng(5)
    q, _ = _bf16(rng, (B, H, Sq, D))
    e = torch.zeros((B, H, 0, D), dtype=torch.bfloat16, device="cuda")
    o, lse = _state(B, H, Sq, D)
    sc.shard_attn_block(q, e, e, o, lse, 0.125, True)
    assert float(o.abs().max()) == 0.0 and bool(torch.all(torch.isneginf(lse)))
    k, _ = _bf16(rng, (B, H, 9, D))
    sc.shard_attn_block(q, k, k, o, lse, 0.125, False)     # merge into the empty state
    o1, l1 = o.clone(), lse.clone()
    sc.shard_attn_block(q, e, e, o, lse, 0.125, False)
    assert torch.equal(o, o1) and torch.equal(lse, l1)


def test_repeatable(sc):
    import torch
    rng = np.random.default_rng(6)
    q, _ = _bf16(rng, (1, 2, 300, 128))
    k, _ = _bf16(rng, (1, 2, 500, 128))
    outs = []
    for _ in range(2):
        o, lse = _state(1, 2, 300, 128)
        sc.shard_attn_block(q, k, k, o, lse, 0.1, True)
        outs.append((o, lse))
    assert torch.equal(outs[0][0], outs[1][0]) and torch.equal(outs[0][1], outs[1][1])


def test_full_size_sampled_queries(sc):
    """The benchmarked block step at full size (1 x 16 heads x 16384 queries
    against 16384 keys, head dim 128), two steps (the second merging a second
    block), checked on sampled query rows of every head."""
    import torch
    B, H, S, D = 1, 16, 16384, 128
    g = torch.Generator(device="cuda").manual_seed(7)
    q = torch.randn((B, H, S, D), generator=g, device="cuda").to(torch.bfloat16)
    k = torch.randn((B, H, 2 * S, D), generator=g, device="cuda").to(torch.bfloat16)
    v = torch.randn((B, H, 2 * S, D), generator=g, device="cuda").to(torch.bfloat16)
    scale = 1 / math.sqrt(D)
    o, lse = _state(B, H, S, D)
    sc.shard_attn_block(q, k[:, :, :S].contiguous(), v[:, :, :S].contiguous(), o, lse, scale, True)
    sc.shard_attn_block(q, k[:, :, S:].contiguous(), v[:, :, S:].contiguous(), o, lse, scale, False)
    rows = np.array(sorted(set([0, 1, 255, 256, S - 1] + list(np.random.default_rng(8).integers(0, S, 11)))))
    q64 = q[:, :, rows].cpu().double().numpy()
    k64, v64 = k.cpu().double().numpy(), v.cpu().double().numpy()
    ref_o, ref_l = oat.full_attention(q64, k64, v64, scale)
    err = _check(o[:, :, rows], lse[:, :, rows], ref_o, ref_l)
    log(f"full-size attention: err {err}")
