"""Pins for the naive attention oracle (CPU only).

Each pin ties oracle/attention.py to something other than itself: the scalar brute
force, torch's own fp64 attention routine and autograd, closed forms of the Section 2
definition, and central finite differences.
"""
import math

import numpy as np
import pytest
import torch

from oracle import attention as A
from oracle import brute


def _rand(seed, *shape):
    return np.random.default_rng(seed).standard_normal(shape)


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("S,D", [(1, 1), (5, 3), (16, 8), (11, 4)])
def test_naive_matches_brute_force(S, D, causal):
    q, k, v = (_rand(s, 2, S, 2, D) for s in (1, 2, 3))
    o, lse = A.attention_fwd(q, k, v, causal)
    for b in range(2):
        for h in range(2):
            ob, lb = brute.attention_brute(q[b, :, h].tolist(), k[b, :, h].tolist(),
                                           v[b, :, h].tolist(), causal)
            np.testing.assert_allclose(o[b, :, h], np.array(ob), rtol=0, atol=1e-12)
            np.testing.assert_allclose(lse[b, h], np.array(lb), rtol=0, atol=1e-12)


@pytest.mark.parametrize("causal", [False, True])
def test_naive_matches_torch_sdpa_fp64(causal):
    q, k, v = (_rand(s, 2, 67, 3, 16) for s in (4, 5, 6))
    o, lse = A.attention_fwd(q, k, v, causal, row_chunk=17)
    t = lambda x: torch.from_numpy(x).permute(0, 2, 1, 3)  # [B,H,S,D]
    ref = torch.nn.functional.scaled_dot_product_attention(t(q), t(k), t(v), is_causal=causal)
    np.testing.assert_allclose(o, ref.permute(0, 2, 1, 3).numpy(), rtol=0, atol=1e-12)
    # lse against torch.logsumexp of the scaled, masked scores
    s = torch.einsum("bhqd,bhkd->bhqk", t(q), t(k)) / math.sqrt(16)
    if causal:
        s = s.masked_fill(torch.ones(67, 67, dtype=torch.bool).triu(1), float("-inf"))
    np.testing.assert_allclose(lse, torch.logsumexp(s, dim=-1).numpy(), rtol=0, atol=1e-12)


def test_rows_and_offset_match_full():
    q, k, v = (_rand(s, 1, 48, 2, 8) for s in (7, 8, 9))
    o, lse = A.attention_fwd(q, k, v, True)
    rows = np.array([0, 5, 17, 47])
    orow, lrow = A.attention_rows(q, k, v, rows, True)
    np.testing.assert_allclose(orow, o[:, rows], atol=1e-13)
    np.testing.assert_allclose(lrow, lse[:, :, rows], atol=1e-13)
    # a later query block evaluated against the whole sequence (global positions)
    ob, lb = A.attention_fwd(q[:, 32:], k, v, True, q_offset=32)
    np.testing.assert_allclose(ob, o[:, 32:], atol=1e-13)
    np.testing.assert_allclose(lb, lse[:, :, 32:], atol=1e-13)


def test_zero_query_gives_prefix_mean():
    """All scores tie when Q = 0: causal row r is the mean of V_0..V_r, lse = ln(r+1);
    without the mask every row is mean(V) and lse = ln S."""
    S = 40
    v = _rand(11, 1, S, 2, 8)
    k = _rand(12, 1, S, 2, 8)
    q = np.zeros_like(v)
    o, lse = A.attention_fwd(q, k, v, True)
    prefix = np.cumsum(v, axis=1) / np.arange(1, S + 1)[None, :, None, None]
    np.testing.assert_allclose(o, prefix, atol=1e-13)
    np.testing.assert_allclose(lse, np.broadcast_to(np.log(np.arange(1, S + 1)), lse.shape), atol=1e-13)
    o, lse = A.attention_fwd(q, k, v, False)
    np.testing.assert_allclose(o, np.broadcast_to(v.mean(axis=1, keepdims=True), o.shape), atol=1e-13)
    np.testing.assert_allclose(lse, math.log(S), atol=1e-13)


def test_first_causal_token():
    """Row 0 of a causal attention sees only key 0: O_0 = V_0, lse_0 = q_0.k_0/sqrt(D),
    and dQ_0 = 0 (its softmax has a single entry)."""
    q, k, v, do = (_rand(s, 2, 9, 3, 8) for s in (13, 14, 15, 16))
    o, lse = A.attention_fwd(q, k, v, True)
    np.testing.assert_array_equal(o[:, 0], v[:, 0])
    np.testing.assert_allclose(lse[:, :, 0], (q[:, 0] * k[:, 0]).sum(-1) / math.sqrt(8), atol=1e-14)
    dq, _, _ = A.attention_bwd(q, k, v, do, True)
    np.testing.assert_allclose(dq[:, 0], 0.0, atol=1e-14)


def test_constant_values_and_identical_keys():
    q, k = _rand(17, 1, 20, 2, 8), _rand(18, 1, 20, 2, 8)
    o, _ = A.attention_fwd(q, k, np.ones((1, 20, 2, 8)), True)
    np.testing.assert_allclose(o, 1.0, atol=1e-14)
    # identical key rows: scores do not depend on q, so dQ = 0
    kk = np.broadcast_to(k[:, :1], k.shape).copy()
    v, do = _rand(19, 1, 20, 2, 8), _rand(20, 1, 20, 2, 8)
    dq, _, _ = A.attention_bwd(q, kk, v, do, False)
    np.testing.assert_allclose(dq, 0.0, atol=1e-13)


@pytest.mark.parametrize("causal", [False, True])
def test_backward_matches_torch_autograd_fp64(causal):
    q, k, v, do = (_rand(s, 2, 33, 2, 16) for s in (21, 22, 23, 24))
    dq, dk, dv = A.attention_bwd(q, k, v, do, causal, row_chunk=7)
    tq, tk, tv = (torch.from_numpy(x).permute(0, 2, 1, 3).requires_grad_() for x in (q, k, v))
    out = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, is_causal=causal)
    out.backward(torch.from_numpy(do).permute(0, 2, 1, 3))
    for mine, ref in ((dq, tq), (dk, tk), (dv, tv)):
        np.testing.assert_allclose(mine, ref.grad.permute(0, 2, 1, 3).numpy(), atol=1e-12)


@pytest.mark.parametrize("causal", [False, True])
def test_backward_finite_differences(causal):
    q, k, v, do = (_rand(s, 1, 6, 1, 3) for s in (25, 26, 27, 28))
    dq, dk, dv = A.attention_bwd(q, k, v, do, causal)

    def loss(q_, k_, v_):
        return float((A.attention_fwd(q_, k_, v_, causal)[0] * do).sum())

    eps = 1e-6
    for idx, (x, g) in enumerate(((q, dq), (k, dk), (v, dv))):
        num = np.zeros_like(x)
        for pos in np.ndindex(x.shape):
            xp, xm = x.copy(), x.copy()
            xp[pos] += eps
            xm[pos] -= eps
            args_p = [q, k, v]
            args_m = [q, k, v]
            args_p[idx], args_m[idx] = xp, xm
            num[pos] = (loss(*args_p) - loss(*args_m)) / (2 * eps)
        np.testing.assert_allclose(g, num, atol=1e-8)


@pytest.mark.parametrize("causal", [False, True])
def test_gradient_invariants(causal):
    """Rows of dS sum to zero, so sum_s dK_s = 0; and sum_s dV_s = sum_r dO_r."""
    q, k, v, do = (_rand(s, 2, 30, 3, 8) for s in (29, 30, 31, 32))
    dq, dk, dv = A.attention_bwd(q, k, v, do, causal)
    np.testing.assert_allclose(dk.sum(axis=1), 0.0, atol=1e-12)
    np.testing.assert_allclose(dv.sum(axis=1), do.sum(axis=1), atol=1e-12)


def test_gradient_rows_match_full_backward():
    q, k, v, do = (_rand(s, 2, 40, 2, 8) for s in (33, 34, 35, 36))
    dq, _, _ = A.attention_bwd(q, k, v, do, True)
    rows = np.array([0, 3, 17, 39])
    np.testing.assert_allclose(A.attention_bwd_rows(q, k, v, do, rows, True), dq[:, rows], atol=1e-13)
    # a later query block against all keys (global positions)
    dqb, dkb, dvb = A.attention_bwd(q[:, 24:], k, v, do[:, 24:], True, q_offset=24)
    np.testing.assert_allclose(dqb, dq[:, 24:], atol=1e-13)
    np.testing.assert_allclose(A.attention_bwd_rows(q[:, 24:], k, v, do[:, 24:], [0, 15], True, q_offset=24),
                               dq[:, [24, 39]], atol=1e-13)


def _torch_host_share_grads(q, k, v, do, causal, q_offset):
    """torch fp64 autograd of sum(do * attention(q, k, v)) for a query block at global
    positions q_offset.. against every key (explicit boolean mask for the offset)."""
    tq, tk, tv = (torch.from_numpy(x).permute(0, 2, 1, 3).requires_grad_() for x in (q, k, v))
    mask = None
    if causal:
        qpos = q_offset + torch.arange(q.shape[1])[:, None]
        mask = torch.arange(k.shape[1])[None, :] <= qpos
    out = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, attn_mask=mask)
    out.backward(torch.from_numpy(do).permute(0, 2, 1, 3))
    return [t.grad.permute(0, 2, 1, 3).numpy() for t in (tq, tk, tv)]


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("q_offset,chunk", [(0, 5), (24, 7), (24, 512)])
def test_key_row_gradients_match_torch_autograd(causal, q_offset, chunk):
    """dK / dV rows of chosen keys (the host-share view: a query block at an offset adds its
    contribution to every key's gradient) against torch autograd, and the host-share
    backward with its causal key limit against the same."""
    q, k, v, do = (_rand(s, 2, 40, 2, 8) for s in (37, 38, 39, 40))
    qb, dob = q[:, q_offset:], do[:, q_offset:]
    tdq, tdk, tdv = _torch_host_share_grads(qb, k, v, dob, causal, q_offset)
    rows = np.array([0, 1, 13, 23, 24, 25, 39])
    dk, dv = A.attention_bwd_key_rows(qb, k, v, dob, rows, causal, q_offset=q_offset, row_chunk=chunk)
    np.testing.assert_allclose(dk, tdk[:, rows], atol=1e-12)
    np.testing.assert_allclose(dv, tdv[:, rows], atol=1e-12)
    dq, dk_all, dv_all = A.attention_bwd(qb, k, v, dob, causal, q_offset=q_offset, row_chunk=chunk)
    for mine, ref in ((dq, tdq), (dk_all, tdk), (dv_all, tdv)):
        np.testing.assert_allclose(mine, ref, atol=1e-12)
    o, lse = A.attention_fwd(qb, k, v, causal, q_offset=q_offset, row_chunk=chunk)
    tq, tk, tv = (torch.from_numpy(x).permute(0, 2, 1, 3) for x in (qb, k, v))
    mask = None
    if causal:
        mask = torch.arange(40)[None, :] <= (q_offset + torch.arange(qb.shape[1])[:, None])
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, attn_mask=mask)
    np.testing.assert_allclose(o, ref.permute(0, 2, 1, 3).numpy(), atol=1e-12)
