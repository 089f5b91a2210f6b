"""Error model behind the layer tolerances (test support; not the oracle, not the product).

Emulates, in float64 torch on the CPU, a transformer layer computed in exact arithmetic
except that every intermediate the GPU path stores in bf16 is rounded to bf16 there
(Q, K, V, the probabilities P, the attention output A, Y, the activation, Z; in the
backward pass dH, dY, dO, P, dS, dQ, dK, dV, dX).  Comparing it with the fp64 oracle
gives the error that bf16 storage alone causes -- the floor any bf16 implementation of
the layer faces -- from which the layer tests' tolerances are set.
"""
import math

import numpy as np
import torch

from oracle import layer as OL


def _bf(t):
    return t.to(torch.bfloat16).double()


def layer_rounding_errors(x, wq, wk, wv, wo, w1, w2, dz, n_heads):
    """Returns dict with max magnitude-scaled and relative-RMS errors of z and dx."""
    S, dm = x.shape
    H, D = n_heads, dm // n_heads
    X, Wq, Wk, Wv, Wo, W1, W2, dZ = (t.double() for t in (x, wq, wk, wv, wo, w1, w2, dz))
    mask = torch.ones(S, S, dtype=torch.bool).triu(1)
    heads = lambda t: t.view(S, H, D).transpose(0, 1)
    flat = lambda t: t.transpose(0, 1).reshape(S, dm)
    Q, K, V = (heads(_bf(X @ W)) for W in (Wq, Wk, Wv))
    s = (Q @ K.transpose(1, 2) / math.sqrt(D)).masked_fill(mask, float("-inf"))
    P = torch.softmax(s, dim=-1)
    Pb = _bf(torch.exp(s - s.max(-1, keepdim=True).values))
    A = _bf((Pb @ V) / Pb.sum(-1, keepdim=True))
    Y = _bf(X + flat(A) @ Wo)
    Hpre = Y @ W1
    Z = _bf(Y + _bf(torch.nn.functional.gelu(Hpre)) @ W2)
    # backward
    cdf = 0.5 * (1 + torch.erf(Hpre / math.sqrt(2)))
    pdf = torch.exp(-0.5 * Hpre ** 2) / math.sqrt(2 * math.pi)
    dH = _bf((dZ @ W2.T) * (cdf + Hpre * pdf))
    dY = _bf(dZ + dH @ W1.T)
    dO = heads(_bf(dY @ Wo.T))
    delta = (dO * A).sum(-1, keepdim=True)
    dS = _bf(P * (dO @ V.transpose(1, 2) - delta))
    dq = _bf(dS @ K / math.sqrt(D))
    dk = _bf(dS.transpose(1, 2) @ Q / math.sqrt(D))
    dv = _bf(_bf(P).transpose(1, 2) @ dO)
    dX = _bf(dY + flat(dq) @ Wq.T + flat(dk) @ Wk.T + flat(dv) @ Wv.T)
    np_in = [t.float().numpy() for t in (x, wq, wk, wv, wo, w1, w2)]
    z_ref = torch.from_numpy(OL.layer_fwd(*np_in, n_heads=H))
    dx_ref = torch.from_numpy(OL.layer_bwd(*np_in, dz.float().numpy(), n_heads=H)[0])
    out = {}
    for name, got, ref in (("z", Z, z_ref), ("dx", dX, dx_ref)):
        out[name + "_scaled_max"] = float(((got - ref).abs() / ref.abs().clamp(min=1.0)).max())
        out[name + "_rel_rms"] = float((got - ref).pow(2).mean().sqrt() / ref.pow(2).mean().sqrt())
    return out


def llama_layer_rounding_errors(x, params, dz, n_heads):
    """The LLaMA-style layer (oracle/llama.py) in exact arithmetic except for bf16 storage
    where the GPU path stores bf16: n1, q, k, v, the rotated q and k, P, the attention
    output, h, n2, the gate output, z; backward dh, dO, P, dS, the rotated-q/k gradients and
    dv, dq and dk after the inverse rotation, du, dw, dx (x W1, x W3 and the normalisation
    gradients stay float32, as there).  Returns, for z, dx and every parameter gradient,
    (max |err|, rms of the exact value, relative RMS error) against the fp64 oracle."""
    from oracle import llama as LL

    S, dm = x.shape
    H, D = n_heads, dm // n_heads
    X, dZ = x.double(), dz.double()
    g1, Wq, Wk, Wv, Wo, g2, W1, W3, W2 = (t.double() for t in params)
    pos = np.arange(S)
    rot = lambda t, inv=False: torch.from_numpy(LL.rope(t.view(S, H, D).numpy(), pos, inverse=inv)).reshape(S, dm)
    norm = lambda t, g: t / torch.sqrt((t * t).mean(1, keepdim=True) + LL.EPS) * g
    mask = torch.ones(S, S, dtype=torch.bool).triu(1)
    heads = lambda t: t.view(S, H, D).transpose(0, 1)
    flat = lambda t: t.transpose(0, 1).reshape(S, dm)
    n1 = _bf(norm(X, g1))
    q, k, v = (_bf(n1 @ W) for W in (Wq, Wk, Wv))
    qr, kr = _bf(rot(q)), _bf(rot(k))
    Q, K, V = heads(qr), heads(kr), heads(v)
    s = (Q @ K.transpose(1, 2) / math.sqrt(D)).masked_fill(mask, float("-inf"))
    P = torch.softmax(s, dim=-1)
    Pb = _bf(torch.exp(s - s.max(-1, keepdim=True).values))
    A = _bf((Pb @ V) / Pb.sum(-1, keepdim=True))
    a = flat(A)
    h = _bf(X + a @ Wo)
    n2 = _bf(norm(h, g2))
    u, w = n2 @ W1, n2 @ W3
    sig = torch.sigmoid(u)
    gte = _bf(u * sig * w)
    Z = _bf(h + gte @ W2)
    dgte = dZ @ W2.T
    du, dw = _bf(dgte * w * sig * (1 + u * (1 - sig))), _bf(dgte * u * sig)
    dW2, dW1, dW3 = gte.T @ dZ, n2.T @ du, n2.T @ dw
    dn2 = du @ W1.T + dw @ W3.T
    dh_n, dG2 = LL.rmsnorm_bwd(h.numpy(), g2.numpy(), dn2.numpy())
    dh = _bf(dZ + torch.from_numpy(dh_n))
    dWo = a.T @ dh
    dO = heads(_bf(dh @ Wo.T))
    delta = (dO * A).sum(-1, keepdim=True)
    dS = _bf(P * (dO @ V.transpose(1, 2) - delta))
    dqr = _bf(flat(dS @ K / math.sqrt(D)))
    dkr = _bf(flat(dS.transpose(1, 2) @ Q / math.sqrt(D)))
    dv = _bf(flat(_bf(P).transpose(1, 2) @ dO))
    dq, dk = _bf(rot(dqr, True)), _bf(rot(dkr, True))
    dWq, dWk, dWv = n1.T @ dq, n1.T @ dk, n1.T @ dv
    dn1 = dq @ Wq.T + dk @ Wk.T + dv @ Wv.T
    dx_n, dG1 = LL.rmsnorm_bwd(X.numpy(), g1.numpy(), dn1.numpy())
    dX = _bf(dh + torch.from_numpy(dx_n))
    p64 = [t.float().numpy() for t in params]
    z_ref = LL.layer_fwd(x.float().numpy(), *p64, H)
    ref = LL.layer_bwd(x.float().numpy(), *p64, dz.float().numpy(), H)
    got = [Z, dX, torch.from_numpy(dG1), dWq, dWk, dWv, dWo, torch.from_numpy(dG2), dW1, dW3, dW2]
    names = ["z", "dx", "g1", "wq", "wk", "wv", "wo", "g2", "w1", "w3", "w2"]
    out = {}
    for name, g_, r in zip(names, got, [z_ref] + list(ref)):
        g_ = g_.numpy() if torch.is_tensor(g_) else g_
        err = np.abs(g_ - r)
        rms = float(np.sqrt(np.mean(r * r)))
        out[name] = (float(err.max()), rms, float(np.sqrt(np.mean(err * err))) / max(rms, 1e-30))
        if name in ("z", "dx"):  # magnitude-scaled max, the metric of the z / dx bounds
            out[name + "_scaled_max"] = float((err / np.maximum(1.0, np.abs(r))).max())
    return out


def attention_rounding_errors(q, k, v, do, causal=True):
    """Ring attention forward and backward in exact arithmetic except for what the bf16 path
    stores in bf16: the probabilities P that multiply V (their row sum, the denominator, is
    taken over the rounded values), the output o -- which the backward entry point receives
    in bf16 and which enters Delta = rowsum(dO * o) --, the recomputed P and dS as product
    operands of the backward, and dq, dk, dv.  Inputs are bf16 tensors [B, S, H, D].
    Returns, for o and each gradient, (max |err|, max |err| / max(1, |ref|), relative RMS)
    against the fp64 oracle: the error that bf16 storage alone causes."""
    from oracle import attention as OA

    B, S, H, D = q.shape
    Q, K, V, dO = (t.double().permute(0, 2, 1, 3) for t in (q, k, v, do))  # [B, H, S, D]
    s = Q @ K.transpose(-1, -2) / math.sqrt(D)
    if causal:
        s = s.masked_fill(torch.ones(S, S, dtype=torch.bool).triu(1), float("-inf"))
    m = s.max(-1, keepdim=True).values
    Pb = _bf(torch.exp(s - m))
    den = Pb.sum(-1, keepdim=True)
    o = _bf((Pb @ V) / den)
    lse = m + torch.log(den)
    P = torch.exp(s - lse)
    delta = (dO * o).sum(-1, keepdim=True)
    dS = _bf(P * (dO @ V.transpose(-1, -2) - delta))
    dq = _bf(dS @ K / math.sqrt(D))
    dk = _bf(dS.transpose(-1, -2) @ Q / math.sqrt(D))
    dv = _bf(_bf(P).transpose(-1, -2) @ dO)
    f = [t.float().numpy() for t in (q, k, v, do)]
    o_ref, _ = OA.attention_fwd(*f[:3], causal)
    refs = (o_ref,) + tuple(OA.attention_bwd(*f, causal))
    out = {}
    for name, got, ref in zip(("o", "dq", "dk", "dv"), (o, dq, dk, dv), refs):
        g = got.permute(0, 2, 1, 3).numpy()
        err = np.abs(g - ref)
        out[name] = (float(err.max()), float((err / np.maximum(1.0, np.abs(ref))).max()),
                     float(np.sqrt((err ** 2).mean() / (ref ** 2).mean())))
    return out
