"""One transformer layer as Algorithm 1 composes it (oracle; test infrastructure only).

Algorithm 1 computes query, key and value for each host's input block, runs ring
attention over the hosts, then the blockwise feed-forward network on each host's
attention output.  The paper fixes neither normalisation, positional encoding, biases
nor where the residual connections go for this layer, so this module takes one
reading and the library follows the same one:

  Q = X Wq, K = X Wk, V = X Wv           (split into H heads of D = d_model / H)
  A = Attention(Q, K, V)                 (causal, scale 1/sqrt(D))
  Y = X + A Wo
  Z = Y + FFN(Y),  FFN(y) = GeLU_erf(y W1) W2   (no biases)

X has shape [S, d_model] (batch 1).  The backward pass returns the gradients of
sum(dZ * Z) with respect to X and every weight.  The composition is a reading of the
paper; the code is pinned to it by a restatement in torch library routines (scaled
dot-product attention, GeLU, autograd for the gradients), by the closed form that zero
query and key weights give (causal attention becomes the running mean of the value rows),
and by central finite differences; its attention and FFN parts have their own pins.
"""
import numpy as np

from . import attention as _attn
from . import ffn as _ffn


def _heads(x, H):
    S, dm = x.shape
    return x.reshape(1, S, H, dm // H)


def layer_fwd(x, wq, wk, wv, wo, w1, w2, n_heads, causal=True):
    """Returns Z [S, d_model]."""
    x = np.asarray(x, np.float64)
    S, dm = x.shape
    q, k, v = (_heads(x @ np.asarray(w, np.float64), n_heads) for w in (wq, wk, wv))
    a, _ = _attn.attention_fwd(q, k, v, causal)
    y = x + a.reshape(S, dm) @ np.asarray(wo, np.float64)
    return y + _ffn.ffn_fwd(y, w1, None, w2, None, _ffn.GELU_ERF)


def layer_bwd(x, wq, wk, wv, wo, w1, w2, dz, n_heads, causal=True):
    """Returns (dx, dwq, dwk, dwv, dwo, dw1, dw2) for upstream dz."""
    x, wq, wk, wv, wo, w1, w2, dz = (np.asarray(t, np.float64)
                                     for t in (x, wq, wk, wv, wo, w1, w2, dz))
    S, dm = x.shape
    q, k, v = (_heads(x @ w, n_heads) for w in (wq, wk, wv))
    a, _ = _attn.attention_fwd(q, k, v, causal)
    a2 = a.reshape(S, dm)
    y = x + a2 @ wo
    # Z = Y + FFN(Y): dY = dZ + FFN'(Y)^T dZ
    dy_ffn, dw1, _, dw2, _ = _ffn.ffn_bwd(y, w1, None, w2, dz, _ffn.GELU_ERF)
    dy = dz + dy_ffn
    # Y = X + A Wo
    dwo = a2.T @ dy
    da = (dy @ wo.T).reshape(1, S, n_heads, dm // n_heads)
    dq, dk, dv = _attn.attention_bwd(q, k, v, da, causal)
    dq, dk, dv = (t.reshape(S, dm) for t in (dq, dk, dv))
    dx = dy + dq @ wq.T + dk @ wk.T + dv @ wv.T
    return dx, x.T @ dq, x.T @ dk, x.T @ dv, dwo, dw1, dw2
