"""A LLaMA-style transformer layer around ring attention, and a stack of them (oracle;
test only).

The paper trains LLaMA models (Section 4, model configuration) with Ring Attention and
full gradient checkpointing of attention and FFN (Section 4 settings; the appendix on
training details).  The architecture pieces it inherits from LLaMA are not in the paper;
this module writes them out from their usual definitions, in float64:

  * RMSNorm:  y = x / sqrt(mean(x^2) + eps) * g   (row-wise, learned gain g)
  * rotary position embedding (RoPE) on each head of q and k, on interleaved pairs
    (2i, 2i+1) rotated by the angle p * base^(-2i / D) at global position p
  * SwiGLU feed-forward:  (silu(x W1) * (x W3)) W2,  silu(u) = u sigmoid(u)
  * pre-norm layer:
        n1 = RMSNorm(x; g1);  q, k, v = n1 Wq, n1 Wk, n1 Wv
        h  = x + Attention(RoPE(q), RoPE(k), v) Wo          (causal, global positions)
        n2 = RMSNorm(h; g2);  z = h + SwiGLU(n2)

The attention is the plain definition of ``oracle.attention`` (which the ring result
equals exactly).  Backward passes follow the chain rule, recomputing nothing that the
forward returns.  The composition (norm placement, eps, RoPE pairing and base) is a
reading, not fixed by the paper; the code is pinned to that reading by a restatement in
torch library routines (rms_norm, torch.polar rotary embedding, scaled dot-product
attention, silu) with autograd for every gradient, of the layer and of a two-layer stack,
and by finite differences; each piece is pinned to a library routine or to a property it
must satisfy (tests/test_oracle_llama.py).
"""
import numpy as np

from oracle import attention as OA

EPS = 1e-6
ROPE_BASE = 10000.0


def _as64(x):
    return np.asarray(x, dtype=np.float64)


# ---- RMSNorm --------------------------------------------------------------------------
def rmsnorm_fwd(x, g, eps=EPS):
    """x [T, d], g [d] -> (y [T, d], rstd [T])."""
    x, g = _as64(x), _as64(g)
    rstd = 1.0 / np.sqrt(np.mean(x * x, axis=1) + eps)
    return x * rstd[:, None] * g[None, :], rstd


def rmsnorm_bwd(x, g, dy, eps=EPS):
    """Gradients (dx [T, d], dg [d]) of y = rmsnorm(x, g) for upstream dy."""
    x, g, dy = _as64(x), _as64(g), _as64(dy)
    d = x.shape[1]
    rstd = 1.0 / np.sqrt(np.mean(x * x, axis=1) + eps)
    gdy = dy * g[None, :]
    # d rstd / d x_i = -rstd^3 x_i / d
    dx = gdy * rstd[:, None] - x * (rstd ** 3 / d * np.sum(gdy * x, axis=1))[:, None]
    dg = np.sum(dy * x * rstd[:, None], axis=0)
    return dx, dg


# ---- rotary position embedding ----------------------------------------------------------
def rope_angles(positions, D, base=ROPE_BASE):
    """[len(positions), D/2] angles p * base^(-2i/D)."""
    inv = base ** (-np.arange(0, D, 2, dtype=np.float64) / D)
    return np.asarray(positions, dtype=np.float64)[:, None] * inv[None, :]


def rope(x, positions, base=ROPE_BASE, inverse=False):
    """Rotate x [T, H, D] (or [T, H*D] with H given by the caller's reshape) pairwise:
    pair (2i, 2i+1) of row t by +angle (forward) or -angle (inverse = transpose)."""
    x = _as64(x)
    T, H, D = x.shape
    ang = rope_angles(positions, D, base)
    c, s = np.cos(ang)[:, None, :], np.sin(ang)[:, None, :]
    if inverse:
        s = -s
    x0, x1 = x[..., 0::2], x[..., 1::2]
    y = np.empty_like(x)
    y[..., 0::2] = x0 * c - x1 * s
    y[..., 1::2] = x0 * s + x1 * c
    return y


# ---- SwiGLU feed-forward ------------------------------------------------------------------
def _sigmoid(u):
    return 1.0 / (1.0 + np.exp(-u))


def silu(u):
    return u * _sigmoid(u)


def silu_grad(u):
    s = _sigmoid(u)
    return s * (1.0 + u * (1.0 - s))


def swiglu_fwd(x, w1, w3, w2):
    x, w1, w3, w2 = (_as64(t) for t in (x, w1, w3, w2))
    return (silu(x @ w1) * (x @ w3)) @ w2


def swiglu_bwd(x, w1, w3, w2, dy):
    """Returns (dx, dw1, dw3, dw2)."""
    x, w1, w3, w2, dy = (_as64(t) for t in (x, w1, w3, w2, dy))
    u, w = x @ w1, x @ w3
    gte = silu(u) * w
    dgte = dy @ w2.T
    du = dgte * w * silu_grad(u)
    dw = dgte * silu(u)
    return du @ w1.T + dw @ w3.T, x.T @ du, x.T @ dw, gte.T @ dy


# ---- the layer ---------------------------------------------------------------------------
def _heads(t, H):
    return t.reshape(1, t.shape[0], H, -1)


def layer_fwd(x, g1, wq, wk, wv, wo, g2, w1, w3, w2, n_heads, causal=True, eps=EPS, base=ROPE_BASE,
              return_all=False):
    """x [S, d] -> z [S, d] (batch 1).  With return_all, also the intermediates."""
    x = _as64(x)
    S, d = x.shape
    H = int(n_heads)
    D = d // H
    pos = np.arange(S)
    n1, _ = rmsnorm_fwd(x, g1, eps)
    q, k, v = n1 @ _as64(wq), n1 @ _as64(wk), n1 @ _as64(wv)
    qr = rope(q.reshape(S, H, D), pos, base)
    kr = rope(k.reshape(S, H, D), pos, base)
    a, _ = OA.attention_fwd(qr[None], kr[None], v.reshape(1, S, H, D), causal)
    a = a.reshape(S, d)
    h = x + a @ _as64(wo)
    n2, _ = rmsnorm_fwd(h, g2, eps)
    z = h + swiglu_fwd(n2, w1, w3, w2)
    if return_all:
        return z, dict(n1=n1, qr=qr, kr=kr, v=v, a=a, h=h, n2=n2)
    return z


def layer_bwd(x, g1, wq, wk, wv, wo, g2, w1, w3, w2, dz, n_heads, causal=True, eps=EPS, base=ROPE_BASE):
    """Returns (dx, dg1, dwq, dwk, dwv, dwo, dg2, dw1, dw3, dw2) for upstream dz."""
    x, dz = _as64(x), _as64(dz)
    S, d = x.shape
    H = int(n_heads)
    D = d // H
    pos = np.arange(S)
    _, it = layer_fwd(x, g1, wq, wk, wv, wo, g2, w1, w3, w2, H, causal, eps, base, return_all=True)
    dn2, dw1, dw3, dw2 = swiglu_bwd(it["n2"], w1, w3, w2, dz)
    dh_n, dg2 = rmsnorm_bwd(it["h"], g2, dn2, eps)
    dh = dz + dh_n
    dwo = it["a"].T @ dh
    da = dh @ _as64(wo).T
    dqr, dkr, dv = OA.attention_bwd(it["qr"][None], it["kr"][None], it["v"].reshape(1, S, H, D),
                                    da.reshape(1, S, H, D), causal)
    dq = rope(dqr[0], pos, base, inverse=True).reshape(S, d)
    dk = rope(dkr[0], pos, base, inverse=True).reshape(S, d)
    dv = dv[0].reshape(S, d)
    n1 = it["n1"]
    dwq, dwk, dwv = n1.T @ dq, n1.T @ dk, n1.T @ dv
    dn1 = dq @ _as64(wq).T + dk @ _as64(wk).T + dv @ _as64(wv).T
    dx_n, dg1 = rmsnorm_bwd(x, g1, dn1, eps)
    return dh + dx_n, dg1, dwq, dwk, dwv, dwo, dg2, dw1, dw3, dw2


def stack_fwd(x, layers, n_heads, causal=True):
    """Apply the layers (each a tuple (g1, wq, wk, wv, wo, g2, w1, w3, w2)) in order."""
    for p in layers:
        x = layer_fwd(x, *p, n_heads, causal)
    return x


def stack_bwd(x, layers, dz, n_heads, causal=True):
    """Training step of the stack with full recomputation: keep each layer's input, then
    run the layers' backward passes in reverse.  Returns (dx, [per-layer gradient tuples])."""
    inputs = []
    for p in layers:
        inputs.append(_as64(x))
        x = layer_fwd(x, *p, n_heads, causal)
    grads = [None] * len(layers)
    g = _as64(dz)
    for i in reversed(range(len(layers))):
        out = layer_bwd(inputs[i], *layers[i], g, n_heads, causal)
        g = out[0]
        grads[i] = out[1:]
    return g, grads
