"""Ring decode, emulated on the CPU (oracle; test only).

Follows the paper's appendix on the inference requirement: in autoregressive decoding
only a few query tokens (one per generated token) attend to a long key/value cache, and
ring attention serves a cache far larger than one device holds by keeping it split in
blocks over a ring of hosts and circulating the blocks past the queries.  Written out in
float64:

  * The cache of S tokens is split into N = n_hosts blocks of c = S / N tokens; block j
    holds positions [j c, (j + 1) c).
  * The Tq query tokens are the newest tokens: they sit at positions S - Tq .. S - 1,
    inside the last host's block, and their own keys and values are already the last
    Tq rows of the cache.  Under causal masking query t sees keys at positions <= its
    own; without it every query sees the whole cache.
  * The queries stay on the last host (host N - 1).  At step t the key/value block it
    holds is (N - 1 - t) mod N -- the ring order of Section 3: its own block first, then
    its predecessors' -- and the block is folded into the queries' running maximum,
    numerator and denominator with the online-softmax recurrence of Section 2 (the
    same fold as the training forward pass).  After N steps, o = numerator /
    denominator and lse = max + ln(denominator).

The result is exactly softmax attention of the last Tq rows over the whole cache; the
tests pin this against the plain definition in ``oracle.attention``.
"""
import math

import numpy as np


def _as64(x):
    return np.asarray(x, dtype=np.float64)


def ring_decode_fwd(q, k_cache, v_cache, n_hosts, causal=True, order=None, scale=None):
    """Decode attention of q [B, Tq, H, D] against a cache k_cache/v_cache [B, S, H, D].

    ``order`` (optional) replaces the ring order (N-1, N-2, ..., 0) with any sequence of
    the N block indices, to check that the fold does not depend on it.
    Returns (o [B, Tq, H, D], lse [B, H, Tq]).
    """
    q, k, v = _as64(q), _as64(k_cache), _as64(v_cache)
    B, Tq, H, D = q.shape
    S = k.shape[1]
    N = int(n_hosts)
    if S % N or Tq > S or Tq < 1:
        raise ValueError("need S % n_hosts == 0 and 1 <= Tq <= S")
    c = S // N
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    q_pos = np.arange(S - Tq, S)
    blocks = [(N - 1 - t) % N for t in range(N)] if order is None else [int(j) for j in order]
    mx = np.full((B, H, Tq), -np.inf)
    num = np.zeros((B, H, Tq, D))
    den = np.zeros((B, H, Tq))
    for j in blocks:
        kb, vb = k[:, j * c:(j + 1) * c], v[:, j * c:(j + 1) * c]
        k_pos = j * c + np.arange(c)
        s = np.einsum("bqhd,bkhd->bhqk", q, kb) * scale
        if causal:
            s = np.where((k_pos[None, :] <= q_pos[:, None])[None, None], s, -np.inf)
        m_new = np.maximum(mx, s.max(axis=3))
        m_safe = np.where(np.isneginf(m_new), 0.0, m_new)  # nothing visible yet: shift 0
        p = np.exp(s - m_safe[..., None])
        corr = np.exp(mx - m_safe)
        den = den * corr + p.sum(axis=3)
        num = num * corr[..., None] + np.einsum("bhqk,bkhd->bhqd", p, vb)
        mx = m_new
    o = np.transpose(num / den[..., None], (0, 2, 1, 3))
    return o, mx + np.log(den)
