"""Exact softmax attention from its definition (oracle; test infrastructure only).

Section 2 of the paper defines attention as softmax(Q K^T / sqrt(d)) V with the softmax
taken row by row.  This module writes that definition out in float64: it builds the
score matrix of each (batch, head) pair (in row chunks when it would not fit in host
memory; every row is independent, so chunking is the same definition), masks it, and
normalises each row.

Conventions (shared with the library's C-ABI):
  * q, k, v, o, do, dq, dk, dv have layout [B, S, H, D] (the layout of the paper's
    Appendix A code: batch, length, heads, dim per head).
  * lse has layout [B, H, S] (the shape of the paper's running denominator) and holds
    max + ln(denominator) in natural-log units of the scaled scores.
  * Causal masking is by global token position: query at position p sees key at
    position p' iff p' <= p.  Masked keys contribute exactly zero.
  * ``q_offset`` is the global position of q's first row (keys always start at 0);
    it lets a caller evaluate one host's query block against the whole sequence.

Backward: the gradients of L = sum(dO * O) follow from the calculus of the definition:
  Phat = softmax rows, Delta_r = sum_d dO_rd O_rd, dP = dO V^T,
  dS = Phat * (dP - Delta), dQ = dS K / sqrt(d), dK = dS^T Q / sqrt(d), dV = Phat^T dO.
"""
import math

import numpy as np


def _as64(x):
    return np.asarray(x, dtype=np.float64)


def _masked_scores(qh, kh, scale, causal, q_pos0, r0):
    """Scores of query rows [r0, r0+len(qh)) against all keys, masked to -inf."""
    s = (qh @ kh.T) * scale
    if causal:
        qpos = q_pos0 + r0 + np.arange(qh.shape[0])[:, None]
        kpos = np.arange(kh.shape[0])[None, :]
        s = np.where(kpos > qpos, -np.inf, s)
    return s


def _key_end(n_keys, causal, q_offset, r1):
    """Number of leading keys that can be visible to query rows before r1.  Under the causal
    mask the keys at positions >= q_offset + r1 are masked for every such row and contribute
    exactly zero, so they are left out of the row chunk (the same definition, less work)."""
    return n_keys if not causal else max(0, min(n_keys, q_offset + r1))


def attention_fwd(q, k, v, causal, scale=None, q_offset=0, row_chunk=1024):
    """O = softmax(Q K^T * scale) V and lse, per (batch, head).  Returns (o, lse)."""
    q, k, v = _as64(q), _as64(k), _as64(v)
    B, S, H, D = q.shape
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    o = np.zeros((B, S, H, v.shape[3]))
    lse = np.zeros((B, H, S))
    for b in range(B):
        for h in range(H):
            for r0 in range(0, S, row_chunk):
                r1 = min(S, r0 + row_chunk)
                ke = _key_end(k.shape[1], causal, q_offset, r1)
                kh, vh = k[b, :ke, h, :], v[b, :ke, h, :]
                s = _masked_scores(q[b, r0:r1, h, :], kh, scale, causal, q_offset, r0)
                m = s.max(axis=1)
                p = np.exp(s - m[:, None])
                den = p.sum(axis=1)
                o[b, r0:r1, h, :] = (p @ vh) / den[:, None]
                lse[b, h, r0:r1] = m + np.log(den)
    return o, lse


def attention_rows(q, k, v, rows, causal, scale=None, q_offset=0):
    """Output rows ``rows`` of q only (each output row depends on its own query row).

    Returns (o_rows [B, len(rows), H, D], lse_rows [B, H, len(rows)]).
    """
    rows = np.asarray(rows, dtype=np.int64)
    qs = _as64(q)[:, rows]
    B, R, H, D = qs.shape
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    o = np.zeros((B, R, H, v.shape[3]))
    lse = np.zeros((B, H, R))
    for b in range(B):
        for h in range(H):
            kh, vh = _as64(k[b, :, h, :]), _as64(v[b, :, h, :])  # one head at a time
            s = (qs[b, :, h, :] @ kh.T) * scale
            if causal:
                qpos = (q_offset + rows)[:, None]
                kpos = np.arange(kh.shape[0])[None, :]
                s = np.where(kpos > qpos, -np.inf, s)
            m = s.max(axis=1)
            p = np.exp(s - m[:, None])
            den = p.sum(axis=1)
            o[b, :, h, :] = (p @ vh) / den[:, None]
            lse[b, h, :] = m + np.log(den)
    return o, lse


def attention_bwd(q, k, v, do, causal, scale=None, q_offset=0, row_chunk=1024):
    """Gradients (dq, dk, dv) of sum(do * O) with O = attention_fwd(q, k, v).

    O itself is recomputed here from the definition, never taken from elsewhere.
    """
    q, k, v, do = _as64(q), _as64(k), _as64(v), _as64(do)
    B, S, H, D = q.shape
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    dq = np.zeros_like(q)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    for b in range(B):
        for h in range(H):
            for r0 in range(0, S, row_chunk):
                r1 = min(S, r0 + row_chunk)
                ke = _key_end(k.shape[1], causal, q_offset, r1)
                kh, vh = k[b, :ke, h, :], v[b, :ke, h, :]
                qh, doh = q[b, r0:r1, h, :], do[b, r0:r1, h, :]
                s = _masked_scores(qh, kh, scale, causal, q_offset, r0)
                m = s.max(axis=1)
                p = np.exp(s - m[:, None])
                phat = p / p.sum(axis=1)[:, None]
                oh = phat @ vh
                delta = (doh * oh).sum(axis=1)
                dp = doh @ vh.T
                ds = phat * (dp - delta[:, None])
                dq[b, r0:r1, h, :] = (ds @ kh) * scale
                dk[b, :ke, h, :] += (ds.T @ qh) * scale
                dv[b, :ke, h, :] += phat.T @ doh
    return dq, dk, dv


def attention_bwd_rows(q, k, v, do, rows, causal, scale=None, q_offset=0):
    """Rows ``rows`` of dq only (row r of dq depends on query row r, its upstream gradient
    and every key/value).  Same definition as attention_bwd restricted to those rows;
    k and v are upcast one head at a time.  Returns dq_rows [B, len(rows), H, D]."""
    rows = np.asarray(rows, dtype=np.int64)
    qs, dos = _as64(q)[:, rows], _as64(do)[:, rows]
    B, R, H, D = qs.shape
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    dq = np.zeros((B, R, H, D))
    for b in range(B):
        for h in range(H):
            kh, vh = _as64(k[b, :, h, :]), _as64(v[b, :, h, :])
            s = (qs[b, :, h, :] @ kh.T) * scale
            if causal:
                qpos = (q_offset + rows)[:, None]
                s = np.where(np.arange(kh.shape[0])[None, :] > qpos, -np.inf, s)
            p = np.exp(s - s.max(axis=1)[:, None])
            phat = p / p.sum(axis=1)[:, None]
            oh = phat @ vh
            delta = (dos[b, :, h, :] * oh).sum(axis=1)
            ds = phat * (dos[b, :, h, :] @ vh.T - delta[:, None])
            dq[b, :, h, :] = (ds @ kh) * scale
    return dq


def attention_bwd_key_rows(q, k, v, do, key_rows, causal, scale=None, q_offset=0, row_chunk=512):
    """Rows ``key_rows`` of dk and dv only.  Row s of dk (of dv) sums, over every query row r,
    the term dS[r, s] q_r / sqrt(d) (Phat[r, s] dO_r), so it needs every query row's
    normalised probabilities and Delta_r = sum_d dO_rd O_rd: the forward definition is
    evaluated for all query rows (in row chunks, O recomputed from the definition), and only
    the columns ``key_rows`` of Phat and dP enter the sums.  Same definition as
    attention_bwd restricted to those rows.  Returns (dk_rows, dv_rows), each
    [B, len(key_rows), H, D]; q, k, v, do may be float32 and are upcast one head at a time."""
    key_rows = np.asarray(key_rows, dtype=np.int64)
    B, S, H, D = np.shape(q)
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    R = len(key_rows)
    dk = np.zeros((B, R, H, D))
    dv = np.zeros((B, R, H, np.shape(v)[3]))
    kpos = key_rows[None, :]
    for b in range(B):
        for h in range(H):
            kh_all, vh_all = k[b, :, h, :], v[b, :, h, :]
            ks, vs = _as64(kh_all[key_rows]), _as64(vh_all[key_rows])
            for r0 in range(0, S, row_chunk):
                r1 = min(S, r0 + row_chunk)
                ke = _key_end(np.shape(k)[1], causal, q_offset, r1)
                kh, vh = _as64(kh_all[:ke]), _as64(vh_all[:ke])
                qh, doh = _as64(q[b, r0:r1, h, :]), _as64(do[b, r0:r1, h, :])
                s = _masked_scores(qh, kh, scale, causal, q_offset, r0)
                m = s.max(axis=1)
                p = np.exp(s - m[:, None])
                den = p.sum(axis=1)
                oh = (p @ vh) / den[:, None]
                delta = (doh * oh).sum(axis=1)
                # the chosen columns: scores, probabilities and dP against those keys
                ss = (qh @ ks.T) * scale
                if causal:
                    qpos = (q_offset + r0 + np.arange(r1 - r0))[:, None]
                    ss = np.where(kpos > qpos, -np.inf, ss)
                phat = np.exp(ss - m[:, None]) / den[:, None]
                ds = phat * (doh @ vs.T - delta[:, None])
                dk[b, :, h, :] += (ds.T @ qh) * scale
                dv[b, :, h, :] += phat.T @ doh
    return dk, dv
