"""Exact softmax attention from its definition (oracle; test infrastructure only).

Section 2 of the paper defines attention as softmax(Q K^T / sqrt(d)) V with the softmax
taken row by row.  This module writes that definition out in float64: it builds the
score matrix of each (batch, head) pair (in row chunks; every row is independent, so
chunking is the same definition), masks it, and normalises each row.  The arithmetic is
plain PyTorch CPU operations in float64 (matrix products, exp, sums), which use all host
cores; arguments and results are NumPy arrays.

Conventions (shared with the library's C-ABI):
  * q, k, v, o, do, dq, dk, dv have layout [B, S, H, D] (the layout of the paper's
    Appendix A code: batch, length, heads, dim per head).
  * lse has layout [B, H, S] (the shape of the paper's running denominator) and holds
    max + ln(denominator) in natural-log units of the scaled scores.
  * Causal masking is by global token position: query at position p sees key at
    position p' iff p' <= p.  Masked keys contribute exactly zero, so a row chunk only
    takes the keys that can be visible to some row of it.
  * ``q_offset`` is the global position of q's first row (keys always start at 0);
    it lets a caller evaluate one host's query block against the whole sequence.

Backward: the gradients of L = sum(dO * O) follow from the calculus of the definition:
  Phat = softmax rows, Delta_r = sum_d dO_rd O_rd, dP = dO V^T,
  dS = Phat * (dP - Delta), dQ = dS K / sqrt(d), dK = dS^T Q / sqrt(d), dV = Phat^T dO.
"""
import math

import numpy as np
import torch


def _t64(x):
    """float64 CPU tensor of an array-like (NumPy array, torch tensor or nested list)."""
    if torch.is_tensor(x):
        return x.detach().to(device="cpu", dtype=torch.float64)
    return torch.from_numpy(np.ascontiguousarray(np.asarray(x, dtype=np.float64)))


def _np(t):
    return t.numpy()


def _masked_scores(qh, kh, scale, causal, q_pos0, r0):
    """Scores of query rows [r0, r0+len(qh)) against keys 0.., masked to -inf."""
    s = (qh @ kh.T) * scale
    if causal:
        qpos = q_pos0 + r0 + torch.arange(qh.shape[0])[:, None]
        kpos = torch.arange(kh.shape[0])[None, :]
        s = s.masked_fill(kpos > qpos, float("-inf"))
    return s


def _key_end(n_keys, causal, q_offset, r1):
    """Number of leading keys that can be visible to query rows before r1.  Under the causal
    mask the keys at positions >= q_offset + r1 are masked for every such row and contribute
    exactly zero, so they are left out of the row chunk (the same definition, less work)."""
    return n_keys if not causal else max(0, min(n_keys, q_offset + r1))


def attention_fwd(q, k, v, causal, scale=None, q_offset=0, row_chunk=1024):
    """O = softmax(Q K^T * scale) V and lse, per (batch, head).  Returns (o, lse)."""
    B, S, H, D = np.shape(q)
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    nk, Dv = np.shape(k)[1], np.shape(v)[3]
    o = torch.zeros((B, S, H, Dv), dtype=torch.float64)
    lse = torch.zeros((B, H, S), dtype=torch.float64)
    for b in range(B):
        for h in range(H):
            qh_all, kh_all, vh_all = _t64(q[b, :, h, :]), _t64(k[b, :, h, :]), _t64(v[b, :, h, :])
            for r0 in range(0, S, row_chunk):
                r1 = min(S, r0 + row_chunk)
                ke = _key_end(nk, causal, q_offset, r1)
                s = _masked_scores(qh_all[r0:r1], kh_all[:ke], scale, causal, q_offset, r0)
                m = s.max(dim=1).values
                p = torch.exp(s - m[:, None])
                den = p.sum(dim=1)
                o[b, r0:r1, h, :] = (p @ vh_all[:ke]) / den[:, None]
                lse[b, h, r0:r1] = m + torch.log(den)
    return _np(o), _np(lse)


def attention_rows(q, k, v, rows, causal, scale=None, q_offset=0):
    """Output rows ``rows`` of q only (each output row depends on its own query row).

    Returns (o_rows [B, len(rows), H, D], lse_rows [B, H, len(rows)]).
    """
    rows = np.asarray(rows, dtype=np.int64)
    B, _, H, D = np.shape(q)
    R = len(rows)
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    o = torch.zeros((B, R, H, np.shape(v)[3]), dtype=torch.float64)
    lse = torch.zeros((B, H, R), dtype=torch.float64)
    trows = torch.from_numpy(rows)
    for b in range(B):
        for h in range(H):
            qs = _t64(q[b, :, h, :])[trows]
            kh, vh = _t64(k[b, :, h, :]), _t64(v[b, :, h, :])  # one head at a time
            s = (qs @ kh.T) * scale
            if causal:
                s = s.masked_fill(torch.arange(kh.shape[0])[None, :] > (q_offset + trows)[:, None], float("-inf"))
            m = s.max(dim=1).values
            p = torch.exp(s - m[:, None])
            den = p.sum(dim=1)
            o[b, :, h, :] = (p @ vh) / den[:, None]
            lse[b, h, :] = m + torch.log(den)
    return _np(o), _np(lse)


def attention_bwd(q, k, v, do, causal, scale=None, q_offset=0, row_chunk=1024):
    """Gradients (dq, dk, dv) of sum(do * O) with O = attention_fwd(q, k, v).

    O itself is recomputed here from the definition, never taken from elsewhere.
    """
    B, S, H, D = np.shape(q)
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    nk = np.shape(k)[1]
    dq = torch.zeros((B, S, H, D), dtype=torch.float64)
    dk = torch.zeros((B, nk, H, D), dtype=torch.float64)
    dv = torch.zeros((B, nk, H, np.shape(v)[3]), dtype=torch.float64)
    for b in range(B):
        for h in range(H):
            q_all, do_all = _t64(q[b, :, h, :]), _t64(do[b, :, h, :])
            k_all, v_all = _t64(k[b, :, h, :]), _t64(v[b, :, h, :])
            for r0 in range(0, S, row_chunk):
                r1 = min(S, r0 + row_chunk)
                ke = _key_end(nk, causal, q_offset, r1)
                kh, vh = k_all[:ke], v_all[:ke]
                qh, doh = q_all[r0:r1], do_all[r0:r1]
                s = _masked_scores(qh, kh, scale, causal, q_offset, r0)
                m = s.max(dim=1).values
                p = torch.exp(s - m[:, None])
                phat = p / p.sum(dim=1)[:, None]
                oh = phat @ vh
                delta = (doh * oh).sum(dim=1)
                dp = doh @ vh.T
                ds = phat * (dp - delta[:, None])
                dq[b, r0:r1, h, :] = (ds @ kh) * scale
                dk[b, :ke, h, :] += (ds.T @ qh) * scale
                dv[b, :ke, h, :] += phat.T @ doh
    return _np(dq), _np(dk), _np(dv)


def attention_bwd_rows(q, k, v, do, rows, causal, scale=None, q_offset=0):
    """Rows ``rows`` of dq only (row r of dq depends on query row r, its upstream gradient
    and every key/value).  Same definition as attention_bwd restricted to those rows;
    k and v are upcast one head at a time.  Returns dq_rows [B, len(rows), H, D]."""
    rows = np.asarray(rows, dtype=np.int64)
    B, _, H, D = np.shape(q)
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    trows = torch.from_numpy(rows)
    dq = torch.zeros((B, len(rows), H, D), dtype=torch.float64)
    for b in range(B):
        for h in range(H):
            qs, dos = _t64(q[b, :, h, :])[trows], _t64(do[b, :, h, :])[trows]
            kh, vh = _t64(k[b, :, h, :]), _t64(v[b, :, h, :])
            s = (qs @ kh.T) * scale
            if causal:
                s = s.masked_fill(torch.arange(kh.shape[0])[None, :] > (q_offset + trows)[:, None], float("-inf"))
            p = torch.exp(s - s.max(dim=1).values[:, None])
            phat = p / p.sum(dim=1)[:, None]
            oh = phat @ vh
            delta = (dos * oh).sum(dim=1)
            ds = phat * (dos @ vh.T - delta[:, None])
            dq[b, :, h, :] = (ds @ kh) * scale
    return _np(dq)


def attention_bwd_key_rows(q, k, v, do, key_rows, causal, scale=None, q_offset=0, row_chunk=512):
    """Rows ``key_rows`` of dk and dv only.  Row s of dk (of dv) sums, over every query row r,
    the term dS[r, s] q_r / sqrt(d) (Phat[r, s] dO_r), so it needs every query row's
    normalised probabilities and Delta_r = sum_d dO_rd O_rd: the forward definition is
    evaluated for all query rows (in row chunks, O recomputed from the definition), and only
    the columns ``key_rows`` of Phat and dP enter the sums.  Same definition as
    attention_bwd restricted to those rows.  Returns (dk_rows, dv_rows), each
    [B, len(key_rows), H, D]; q, k, v, do are upcast one head at a time."""
    key_rows = np.asarray(key_rows, dtype=np.int64)
    B, S, H, D = np.shape(q)
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    nk = np.shape(k)[1]
    tkr = torch.from_numpy(key_rows)
    dk = torch.zeros((B, len(key_rows), H, D), dtype=torch.float64)
    dv = torch.zeros((B, len(key_rows), H, np.shape(v)[3]), dtype=torch.float64)
    for b in range(B):
        for h in range(H):
            q_all, do_all = _t64(q[b, :, h, :]), _t64(do[b, :, h, :])
            k_all, v_all = _t64(k[b, :, h, :]), _t64(v[b, :, h, :])
            ks, vs = k_all[tkr], v_all[tkr]
            for r0 in range(0, S, row_chunk):
                r1 = min(S, r0 + row_chunk)
                ke = _key_end(nk, causal, q_offset, r1)
                qh, doh = q_all[r0:r1], do_all[r0:r1]
                s = _masked_scores(qh, k_all[:ke], scale, causal, q_offset, r0)
                m = s.max(dim=1).values
                p = torch.exp(s - m[:, None])
                den = p.sum(dim=1)
                oh = (p @ v_all[:ke]) / den[:, None]
                delta = (doh * oh).sum(dim=1)
                # the chosen columns: scores, probabilities and dP against those keys
                ss = (qh @ ks.T) * scale
                if causal:
                    qpos = (q_offset + r0 + torch.arange(r1 - r0))[:, None]
                    ss = ss.masked_fill(tkr[None, :] > qpos, float("-inf"))
                phat = torch.exp(ss - m[:, None]) / den[:, None]
                ds = phat * (doh @ vs.T - delta[:, None])
                dk[b, :, h, :] += (ds.T @ qh) * scale
                dv[b, :, h, :] += phat.T @ doh
    return _np(dk), _np(dv)
