"""Pins for the ring-order blockwise oracle (CPU only).

The ring emulation must reach exactly the plain softmax attention result whatever the
number of hosts, the tile sizes and the order in which key/value blocks are folded in
(the permutation invariance Section 3 relies on).  It is checked against the naive
definition, which is itself pinned in test_oracle_attention.py.
"""
import itertools

import numpy as np
import pytest

from oracle import attention as A
from oracle import ring as R


def _rand(seed, *shape):
    return np.random.default_rng(seed).standard_normal(shape)


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("n_hosts", [1, 2, 4, 8])
def test_ring_forward_equals_naive(n_hosts, causal):
    q, k, v = (_rand(s, 2, 64, 2, 8) for s in (1, 2, 3))
    o_ref, lse_ref = A.attention_fwd(q, k, v, causal)
    o, lse, mx, den = R.ring_attention_fwd(q, k, v, n_hosts, causal)
    np.testing.assert_allclose(o, o_ref, atol=1e-12)
    np.testing.assert_allclose(lse, lse_ref, atol=1e-12)
    np.testing.assert_allclose(mx + np.log(den), lse_ref, atol=1e-12)


@pytest.mark.parametrize("qc,kc", [(1, 1), (2, 4), (4, 2), (3, 5), (8, 8), (16, 16)])
def test_ring_forward_invariant_to_tile_sizes(qc, kc):
    q, k, v = (_rand(s, 1, 64, 2, 4) for s in (4, 5, 6))
    o_ref, lse_ref = A.attention_fwd(q, k, v, True)
    o, lse, _, _ = R.ring_attention_fwd(q, k, v, 4, True, query_chunk=qc, key_chunk=kc)
    np.testing.assert_allclose(o, o_ref, atol=1e-12)
    np.testing.assert_allclose(lse, lse_ref, atol=1e-12)


@pytest.mark.parametrize("n_hosts", [2, 3, 4])
def test_ring_forward_invariant_to_every_block_order(n_hosts):
    S = 12 * n_hosts
    q, k, v = (_rand(s, 1, S, 1, 4) for s in (7, 8, 9))
    o_ref, lse_ref = A.attention_fwd(q, k, v, True)
    for perm in itertools.permutations(range(n_hosts)):
        # host i folds blocks in the order perm, shifted by i (a different order per host)
        order = [[perm[(t + i) % n_hosts] for t in range(n_hosts)] for i in range(n_hosts)]
        o, lse, _, _ = R.ring_attention_fwd(q, k, v, n_hosts, True, query_chunk=5,
                                            key_chunk=3, order=order)
        np.testing.assert_allclose(o, o_ref, atol=1e-12)
        np.testing.assert_allclose(lse, lse_ref, atol=1e-12)


def test_ring_forward_random_orders_eight_hosts():
    rng = np.random.default_rng(10)
    q, k, v = (_rand(s, 1, 64, 2, 4) for s in (11, 12, 13))
    o_ref, _ = A.attention_fwd(q, k, v, True)
    for _ in range(5):
        order = [list(rng.permutation(8)) for _ in range(8)]
        o, _, _, _ = R.ring_attention_fwd(q, k, v, 8, True, order=order)
        np.testing.assert_allclose(o, o_ref, atol=1e-12)


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("n_hosts,qc,kc", [(1, 16, 16), (2, 4, 8), (4, 16, 16), (8, 3, 2)])
def test_ring_backward_equals_naive(n_hosts, qc, kc, causal):
    q, k, v, do = (_rand(s, 2, 48, 2, 8) for s in (14, 15, 16, 17))
    ref = A.attention_bwd(q, k, v, do, causal)
    got = R.ring_attention_bwd(q, k, v, do, n_hosts, causal, query_chunk=qc, key_chunk=kc)
    for g, r in zip(got, ref):
        np.testing.assert_allclose(g, r, atol=1e-12)


def test_ring_backward_invariant_to_block_order():
    q, k, v, do = (_rand(s, 1, 32, 2, 4) for s in (18, 19, 20, 21))
    ref = A.attention_bwd(q, k, v, do, True)
    for perm in itertools.permutations(range(4)):
        order = [[perm[(t + 2 * i) % 4] for t in range(4)] for i in range(4)]
        got = R.ring_attention_bwd(q, k, v, do, 4, True, order=order)
        for g, r in zip(got, ref):
            np.testing.assert_allclose(g, r, atol=1e-12)


@pytest.mark.parametrize("host", [0, 3, 7])
def test_one_host_share_equals_rows_of_full_attention(host):
    q, k, v = (_rand(s, 1, 128, 2, 8) for s in (22, 23, 24))
    o_ref, lse_ref = A.attention_fwd(q, k, v, True)
    c = 16
    o, lse = R.ring_host_fwd(q[:, host * c:(host + 1) * c], k, v, 8, host, True,
                             query_chunk=4, key_chunk=8)
    np.testing.assert_allclose(o, o_ref[:, host * c:(host + 1) * c], atol=1e-12)
    np.testing.assert_allclose(lse, lse_ref[:, :, host * c:(host + 1) * c], atol=1e-12)
