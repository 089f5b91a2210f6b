"""Pins for the ring-decode oracle (CPU only).

oracle/decode.py folds the cache blocks into the queries' running softmax state in ring
order.  These tests tie it to things other than itself: torch's fp64 attention with an
explicit position mask, the scalar brute force on a full sequence whose last rows are the
decode queries, closed forms (zero queries), the reduction to full attention when the
queries are the whole sequence, and invariance under every order of the blocks.
"""
import itertools
import math

import numpy as np
import pytest
import torch

from oracle import brute
from oracle import decode as OD


def _rand(seed, *shape):
    return np.random.default_rng(seed).standard_normal(shape)


def _sdpa_last_rows(q, k, v, causal):
    """torch fp64 attention of q (the last Tq positions) over k, v with a boolean mask."""
    S, Tq = k.shape[1], q.shape[1]
    t = lambda x: torch.from_numpy(x).permute(0, 2, 1, 3)
    mask = None
    if causal:
        qpos = torch.arange(S - Tq, S)[:, None]
        mask = torch.arange(S)[None, :] <= qpos
    o = torch.nn.functional.scaled_dot_product_attention(t(q), t(k), t(v), attn_mask=mask)
    s = torch.einsum("bhqd,bhkd->bhqk", t(q), t(k)) / math.sqrt(q.shape[3])
    if causal:
        s = s.masked_fill(~mask, float("-inf"))
    return o.permute(0, 2, 1, 3).numpy(), torch.logsumexp(s, dim=-1).numpy()


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("S,N,Tq", [(64, 4, 1), (64, 4, 5), (96, 3, 32), (40, 1, 7), (48, 8, 48)])
def test_matches_torch_sdpa_fp64(S, N, Tq, causal):
    q = _rand(1, 2, Tq, 3, 16)
    k, v = _rand(2, 2, S, 3, 16), _rand(3, 2, S, 3, 16)
    o, lse = OD.ring_decode_fwd(q, k, v, N, causal)
    o_ref, lse_ref = _sdpa_last_rows(q, k, v, causal)
    np.testing.assert_allclose(o, o_ref, rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, lse_ref, rtol=0, atol=1e-12)


@pytest.mark.parametrize("causal", [False, True])
def test_matches_brute_force_last_rows(causal):
    """Queries = the last Tq rows of a full sequence: decode equals those rows of full
    (causal) attention computed by scalar loops."""
    S, Tq, N, D = 12, 4, 3, 3
    qfull, k, v = _rand(4, S, D), _rand(5, S, D), _rand(6, S, D)
    o, lse = OD.ring_decode_fwd(qfull[None, S - Tq:, None], k[None, :, None], v[None, :, None], N, causal)
    ob, lb = brute.attention_brute(qfull.tolist(), k.tolist(), v.tolist(), causal)
    np.testing.assert_allclose(o[0, :, 0], np.array(ob)[S - Tq:], atol=1e-12)
    np.testing.assert_allclose(lse[0, 0], np.array(lb)[S - Tq:], atol=1e-12)


def test_zero_query_gives_visible_mean():
    """All scores tie when q = 0: causal query t (position S - Tq + t) returns the mean of
    V over positions 0 .. S - Tq + t and lse = ln(S - Tq + t + 1); without the mask the
    mean over the whole cache and ln S."""
    S, Tq, N = 48, 6, 4
    v = _rand(7, 1, S, 2, 8)
    k = _rand(8, 1, S, 2, 8)
    q = np.zeros((1, Tq, 2, 8))
    o, lse = OD.ring_decode_fwd(q, k, v, N, True)
    n_vis = np.arange(S - Tq, S) + 1
    prefix = np.cumsum(v, axis=1)[:, S - Tq:] / n_vis[None, :, None, None]
    np.testing.assert_allclose(o, prefix, atol=1e-13)
    np.testing.assert_allclose(lse, np.broadcast_to(np.log(n_vis), lse.shape), atol=1e-13)
    o, lse = OD.ring_decode_fwd(q, k, v, N, False)
    np.testing.assert_allclose(o, np.broadcast_to(v.mean(axis=1, keepdims=True), o.shape), atol=1e-13)
    np.testing.assert_allclose(lse, math.log(S), atol=1e-13)


def test_single_query_sees_its_own_key_last():
    """With one query whose key is the only one far above the rest, causal decode puts
    (almost) all weight on the newest cache row: o -> V[S-1]."""
    S, N, D = 32, 4, 8
    k = _rand(9, 1, S, 1, D) * 0.01
    v = _rand(10, 1, S, 1, D)
    q = np.ones((1, 1, 1, D)) * 40.0
    k[0, S - 1, 0] = 40.0  # q.k = 40*40*8/sqrt(8) for the newest key, ~0 elsewhere
    o, _ = OD.ring_decode_fwd(q, k, v, N, True)
    np.testing.assert_allclose(o[0, 0, 0], v[0, S - 1, 0], atol=1e-12)


@pytest.mark.parametrize("N", [1, 2, 3, 4])
def test_every_block_order_gives_the_same_result(N):
    S, Tq = 12 * N, 5
    q = _rand(11, 1, Tq, 2, 4)
    k, v = _rand(12, 1, S, 2, 4), _rand(13, 1, S, 2, 4)
    o0, l0 = OD.ring_decode_fwd(q, k, v, N, True)
    for order in itertools.permutations(range(N)):
        o, lse = OD.ring_decode_fwd(q, k, v, N, True, order=order)
        np.testing.assert_allclose(o, o0, atol=1e-12)
        np.testing.assert_allclose(lse, l0, atol=1e-12)


def test_rejects_bad_shapes():
    q, k = np.zeros((1, 3, 1, 4)), np.zeros((1, 10, 1, 4))
    with pytest.raises(ValueError):
        OD.ring_decode_fwd(q, k, k, 4, True)  # 10 % 4 != 0
    with pytest.raises(ValueError):
        OD.ring_decode_fwd(np.zeros((1, 11, 1, 4)), k, k, 5, True)  # Tq > S
