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
