"""Ring attention with blockwise computation, emulated on the CPU (oracle; test only).

Follows Section 3 ("Ring-Based Blockwise Attention") and the forward/backward code of
Appendix A, written out with explicit per-host state in float64 (plain PyTorch CPU
operations; arguments and results are NumPy arrays):

  * The sequence of length S is split into N = n_hosts equal blocks of c = S / N
    tokens; host i owns query block i and, initially, key/value block i.
  * Forward: every host keeps a running row maximum, numerator (unnormalised output)
    and denominator.  At each of N steps it folds the key/value block it currently
    holds into them, tile by tile (query chunks x key chunks, as the paper's
    ``query_chunk_size`` / ``key_chunk_size``), then passes that block on to host
    i+1 (the ``ppermute`` with permutation i -> i+1 mod N).  At step t host i holds
    block (i - t) mod N.  The output is numerator / denominator.
  * Backward: dq accumulates on the host; dk and dv travel *with* their key/value
    block around the ring and are back at their home host after N rotations.
  * Causal masking uses global positions (query block index times c plus offset,
    key block index times c plus offset); tiles whose keys all lie after all of
    their queries are skipped, and masked keys contribute exactly zero.

Because the blocks are physically rotated (Python list rotation), the bookkeeping of
which block a host holds is independent of the (i - t) mod N formula used by the
library; ``order`` replaces the rotation with an explicit per-host sequence of blocks
to check that the result does not depend on the order in which blocks are folded in
(the permutation invariance the paper's ring relies on).
"""
import math

import numpy as np
import torch

_F64 = torch.float64


def _as64(x):
    """float64 CPU tensor of an array-like (NumPy array or torch tensor)."""
    if torch.is_tensor(x):
        return x.detach().to(device="cpu", dtype=_F64)
    return torch.from_numpy(np.ascontiguousarray(np.asarray(x, dtype=np.float64)))


def _scores(qc, kc, scale):
    """[B, cq, H, D] x [B, ck, H, D] -> [B, H, cq, ck]."""
    return torch.einsum("bqhd,bkhd->bhqk", qc, kc) * scale


def _visible(q_pos, k_pos, causal):
    """Boolean [cq, ck]: key k_pos[j] is visible to query q_pos[i]."""
    if not causal:
        return torch.ones((len(q_pos), len(k_pos)), dtype=torch.bool)
    return k_pos[None, :] <= q_pos[:, None]


def _fold_block_fwd(state, q, kblk, vblk, q_pos0, k_pos0, causal, scale, qchunk, kchunk):
    """Fold one key/value block into a host's (max, numerator, denominator)."""
    mx, num, den = state  # [B,H,c], [B,c,H,D], [B,H,c]
    c_q, c_k = q.shape[1], kblk.shape[1]
    for q0 in range(0, c_q, qchunk):
        q1 = min(c_q, q0 + qchunk)
        q_pos = q_pos0 + torch.arange(q0, q1)
        for k0 in range(0, c_k, kchunk):
            k1 = min(c_k, k0 + kchunk)
            k_pos = k_pos0 + torch.arange(k0, k1)
            vis = _visible(q_pos, k_pos, causal)
            if not bool(vis.any()):
                continue  # fully masked tile: contributes nothing
            s = _scores(q[:, q0:q1], kblk[:, k0:k1], scale)
            s = s.masked_fill(~vis[None, None], float("-inf"))
            m_old = mx[:, :, q0:q1]
            m_new = torch.maximum(m_old, s.amax(dim=3))
            # rows with no visible key so far keep m = -inf; shift by 0 there
            m_safe = torch.where(torch.isneginf(m_new), torch.zeros_like(m_new), m_new)
            p = torch.exp(s - m_safe[..., None])  # masked -> exp(-inf) = 0
            corr = torch.exp(m_old - m_safe)      # m_old = -inf -> 0
            den[:, :, q0:q1] = den[:, :, q0:q1] * corr + p.sum(dim=3)
            corr_o = corr.permute(0, 2, 1)[..., None]  # [B, cq, H, 1]
            pv = torch.einsum("bhqk,bkhd->bqhd", p, vblk[:, k0:k1])
            num[:, q0:q1] = num[:, q0:q1] * corr_o + pv
            mx[:, :, q0:q1] = m_new


def ring_attention_fwd(q, k, v, n_hosts, causal, query_chunk=None, key_chunk=None,
                       order=None, scale=None):
    """Ring-order blockwise attention over ``n_hosts`` virtual hosts.

    Returns (o [B,S,H,D], lse [B,H,S], max [B,H,S], denominator [B,H,S]).
    ``order[i][t]`` (optional) is the block host i folds in at step t; without it the
    blocks are rotated around the ring.
    """
    o, lse, mx, den = _ring_fwd(_as64(q), _as64(k), _as64(v), n_hosts, causal, query_chunk, key_chunk, order,
                                scale)
    return o.numpy(), lse.numpy(), mx.numpy(), den.numpy()


def _ring_fwd(q, k, v, n_hosts, causal, query_chunk, key_chunk, order, scale):
    B, S, H, D = q.shape
    N = int(n_hosts)
    if S % N:
        raise ValueError("sequence length must be a multiple of n_hosts")
    c = S // N
    qchunk = c if query_chunk is None else int(query_chunk)
    kchunk = c if key_chunk is None else int(key_chunk)
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    blk = lambda x, j: x[:, j * c:(j + 1) * c]
    # per-host state: the initial carry of the paper (max = -inf, zeros elsewhere)
    mx = [torch.full((B, H, c), float("-inf"), dtype=_F64) for _ in range(N)]
    num = [torch.zeros((B, c, H, D), dtype=_F64) for _ in range(N)]
    den = [torch.zeros((B, H, c), dtype=_F64) for _ in range(N)]
    # what each host currently holds: (block index, k block, v block)
    held = [(i, blk(k, i), blk(v, i)) for i in range(N)]
    for t in range(N):
        for i in range(N):
            if order is None:
                j, kb, vb = held[i]
            else:
                j = int(order[i][t])
                kb, vb = blk(k, j), blk(v, j)
            _fold_block_fwd((mx[i], num[i], den[i]), blk(q, i), kb, vb,
                            i * c, j * c, causal, scale, qchunk, kchunk)
        # ppermute: host i sends what it holds to host i+1 (receives from i-1)
        held = [held[(i - 1) % N] for i in range(N)]
    o = torch.cat([num[i] / den[i].permute(0, 2, 1)[..., None] for i in range(N)], dim=1)
    mx_all = torch.cat(mx, dim=2)
    den_all = torch.cat(den, dim=2)
    lse = mx_all + torch.log(den_all)
    return o, lse, mx_all, den_all


def _fold_block_bwd(q, kblk, vblk, o, do, lse, dq, dkblk, dvblk, q_pos0, k_pos0, causal,
                    scale, qchunk, kchunk):
    """Add one key/value block's contributions to dq (local) and dk, dv (travelling)."""
    c_q, c_k = q.shape[1], kblk.shape[1]
    delta = (do * o).sum(dim=3).permute(0, 2, 1)  # [B, H, c_q]
    for q0 in range(0, c_q, qchunk):
        q1 = min(c_q, q0 + qchunk)
        q_pos = q_pos0 + torch.arange(q0, q1)
        for k0 in range(0, c_k, kchunk):
            k1 = min(c_k, k0 + kchunk)
            k_pos = k_pos0 + torch.arange(k0, k1)
            vis = _visible(q_pos, k_pos, causal)
            if not bool(vis.any()):
                continue
            s = _scores(q[:, q0:q1], kblk[:, k0:k1], scale)
            # normalised probabilities straight from the saved log-sum-exp
            p = torch.exp(s - lse[:, :, q0:q1, None]).masked_fill(~vis[None, None], 0.0)
            dvblk[:, k0:k1] += torch.einsum("bhqk,bqhd->bkhd", p, do[:, q0:q1])
            dp = torch.einsum("bqhd,bkhd->bhqk", do[:, q0:q1], vblk[:, k0:k1])
            ds = p * (dp - delta[:, :, q0:q1, None])
            dq[:, q0:q1] += torch.einsum("bhqk,bkhd->bqhd", ds, kblk[:, k0:k1]) * scale
            dkblk[:, k0:k1] += torch.einsum("bhqk,bqhd->bkhd", ds, q[:, q0:q1]) * scale


def ring_attention_bwd(q, k, v, do, n_hosts, causal, query_chunk=None, key_chunk=None,
                       order=None, scale=None):
    """Gradients (dq, dk, dv) of sum(do * O) through the ring.

    The forward output and log-sum-exp used as residuals are recomputed here with the
    ring forward (the paper's residuals are output, denominator and max;
    lse = max + ln(denominator) carries the same information).
    """
    q, k, v, do = _as64(q), _as64(k), _as64(v), _as64(do)
    B, S, H, D = q.shape
    N = int(n_hosts)
    c = S // N
    qchunk = c if query_chunk is None else int(query_chunk)
    kchunk = c if key_chunk is None else int(key_chunk)
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    o, lse, _, _ = _ring_fwd(q, k, v, N, causal, qchunk, kchunk, order, scale)
    blk = lambda x, j: x[:, j * c:(j + 1) * c]
    lse_blk = lambda j: lse[:, :, j * c:(j + 1) * c]
    zeros = lambda: torch.zeros((B, c, H, D), dtype=_F64)
    dq = [zeros() for _ in range(N)]
    if order is None:
        # (block index, k, v, dk, dv) travel together around the ring
        held = [(i, blk(k, i), blk(v, i), zeros(), zeros()) for i in range(N)]
        for t in range(N):
            for i in range(N):
                j, kb, vb, dkb, dvb = held[i]
                _fold_block_bwd(blk(q, i), kb, vb, blk(o, i), blk(do, i), lse_blk(i), dq[i],
                                dkb, dvb, i * c, j * c, causal, scale, qchunk, kchunk)
            held = [held[(i - 1) % N] for i in range(N)]
        # after N rotations every block is back at its home host
        assert all(held[i][0] == i for i in range(N))
        dk = torch.cat([held[i][3] for i in range(N)], dim=1)
        dv = torch.cat([held[i][4] for i in range(N)], dim=1)
    else:
        dkb = [zeros() for _ in range(N)]
        dvb = [zeros() for _ in range(N)]
        for t in range(N):
            for i in range(N):
                j = int(order[i][t])
                _fold_block_bwd(blk(q, i), blk(k, j), blk(v, j), blk(o, i), blk(do, i),
                                lse_blk(i), dq[i], dkb[j], dvb[j], i * c, j * c, causal,
                                scale, qchunk, kchunk)
        dk = torch.cat(dkb, dim=1)
        dv = torch.cat(dvb, dim=1)
    return torch.cat(dq, dim=1).numpy(), dk.numpy(), dv.numpy()


def ring_host_fwd(q_blk, k, v, n_hosts, host_idx, causal, query_chunk=None,
                  key_chunk=None, scale=None, blocks=None):
    """One host's share: query block ``host_idx`` against all N key/value blocks, in
    the order they reach that host around the ring ((host_idx - t) mod N).  ``blocks``
    (optional) limits the fold to the first ``blocks`` steps of that order (a partial
    state, used to time a bounded part of the work).

    Returns (o_blk [B,c,H,D], lse_blk [B,H,c]).
    """
    q_blk, k, v = _as64(q_blk), _as64(k), _as64(v)
    B, c, H, D = q_blk.shape
    N = int(n_hosts)
    if k.shape[1] != N * c:
        raise ValueError("key length must be n_hosts * block")
    qchunk = c if query_chunk is None else int(query_chunk)
    kchunk = c if key_chunk is None else int(key_chunk)
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    i = int(host_idx)
    state = (torch.full((B, H, c), float("-inf"), dtype=_F64), torch.zeros((B, c, H, D), dtype=_F64),
             torch.zeros((B, H, c), dtype=_F64))
    for t in range(N if blocks is None else int(blocks)):
        j = (i - t) % N
        _fold_block_fwd(state, q_blk, k[:, j * c:(j + 1) * c], v[:, j * c:(j + 1) * c],
                        i * c, j * c, causal, scale, qchunk, kchunk)
    mx, num, den = state
    o = num / den.permute(0, 2, 1)[..., None]
    return o.numpy(), (mx + torch.log(den)).numpy()
