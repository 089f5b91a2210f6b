"""Seeded synthetic inputs shared by the tests, the bench and the smoke check.

This module only draws random numbers; it holds none of the method's arithmetic.
Both the CPU oracle and the HIP library are fed the exact tensors produced here:
values are drawn in float32 from ``torch.Generator().manual_seed(seed)`` on the CPU in
a fixed order, then rounded to bfloat16 (round-to-nearest-even) where a bf16 workload
asks for it.  Weights are N(0, 0.02), activations and upstream gradients N(0, 1).
"""
import torch


def _gen(seed):
    g = torch.Generator(device="cpu")
    g.manual_seed(int(seed))
    return g


def _draw(g, shape, dtype, std=1.0):
    x = torch.randn(*shape, generator=g, dtype=torch.float32)
    if std != 1.0:
        x.mul_(std)
    return x.to(dtype)


def attention_inputs(seed, B, S, H, D, dtype=torch.bfloat16, with_grad=False, kv_len=None):
    """q [B,S,H,D], k, v [B,kv_len,H,D] (kv_len defaults to S), optionally dO [B,S,H,D].

    Drawn in the order q, k, v, dO.
    """
    g = _gen(seed)
    kv = S if kv_len is None else int(kv_len)
    q = _draw(g, (B, S, H, D), dtype)
    k = _draw(g, (B, kv, H, D), dtype)
    v = _draw(g, (B, kv, H, D), dtype)
    if not with_grad:
        return q, k, v
    do = _draw(g, (B, S, H, D), dtype)
    return q, k, v, do


def ffn_inputs(seed, T, d_model, d_ff, dtype=torch.bfloat16, with_bias=False, with_grad=False):
    """x [T,d_model], w1 [d_model,d_ff], b1 [d_ff] or None, w2 [d_ff,d_model],
    b2 [d_model] or None, dy [T,d_model] or None; drawn in that order."""
    g = _gen(seed)
    x = _draw(g, (T, d_model), dtype)
    w1 = _draw(g, (d_model, d_ff), dtype, 0.02)
    b1 = _draw(g, (d_ff,), dtype, 0.02) if with_bias else None
    w2 = _draw(g, (d_ff, d_model), dtype, 0.02)
    b2 = _draw(g, (d_model,), dtype, 0.02) if with_bias else None
    dy = _draw(g, (T, d_model), dtype) if with_grad else None
    return x, w1, b1, w2, b2, dy


def layer_inputs(seed, S, d_model, d_ff, dtype=torch.bfloat16):
    """x [S,d_model]; Wq, Wk, Wv, Wo [d_model,d_model]; W1 [d_model,d_ff];
    W2 [d_ff,d_model]; dZ [S,d_model]; drawn in that order."""
    g = _gen(seed)
    x = _draw(g, (S, d_model), dtype)
    wq, wk, wv, wo = (_draw(g, (d_model, d_model), dtype, 0.02) for _ in range(4))
    w1 = _draw(g, (d_model, d_ff), dtype, 0.02)
    w2 = _draw(g, (d_ff, d_model), dtype, 0.02)
    dz = _draw(g, (S, d_model), dtype)
    return x, wq, wk, wv, wo, w1, w2, dz


def llama_layer_inputs(seed, S, d_model, d_ff, n_layers=1, dtype=torch.bfloat16):
    """x [S,d_model]; per layer (g1 [d_model], Wq, Wk, Wv, Wo [d_model,d_model],
    g2 [d_model], W1, W3 [d_model,d_ff], W2 [d_ff,d_model]); dZ [S,d_model]; drawn in that
    order.  Gains are 1 + N(0, 0.1) (so that they matter), weights N(0, 0.02)."""
    g = _gen(seed)
    x = _draw(g, (S, d_model), dtype)
    layers = []
    for _ in range(n_layers):
        g1 = (1.0 + 0.1 * torch.randn(d_model, generator=g)).to(dtype)
        wq, wk, wv, wo = (_draw(g, (d_model, d_model), dtype, 0.02) for _ in range(4))
        g2 = (1.0 + 0.1 * torch.randn(d_model, generator=g)).to(dtype)
        w1 = _draw(g, (d_model, d_ff), dtype, 0.02)
        w3 = _draw(g, (d_model, d_ff), dtype, 0.02)
        w2 = _draw(g, (d_ff, d_model), dtype, 0.02)
        layers.append([g1, wq, wk, wv, wo, g2, w1, w3, w2])
    dz = _draw(g, (S, d_model), dtype)
    return x, layers, dz
