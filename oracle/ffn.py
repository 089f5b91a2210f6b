"""Position-wise feed-forward network and projections (oracle; test infrastructure only).

Section 2 defines FFN(x) = act(x W1 + b1) W2 + b2 applied to every position separately
(the paper writes it with ReLU).  The blockwise form of Section 2 ("Blockwise Parallel
Transformers") applies the same network to one block of rows at a time so that the
[rows, d_ff] intermediate never exists for the whole sequence; since every row is
independent, it computes exactly the same values.

Activations (selected by ``act``):
  0  GeLU, exact:  x * Phi(x) = 0.5 x (1 + erf(x / sqrt 2)),  d/dx = Phi(x) + x phi(x)
  1  ReLU:         max(0, x),                                  d/dx = [x > 0]
  2  GeLU, tanh:   0.5 x (1 + tanh(u)), u = sqrt(2/pi) (x + 0.044715 x^3)

Backward of y = act(x W1 + b1) W2 + b2 for upstream dy (all float64):
  H = x W1 + b1, A = act(H), dA = dy W2^T, dH = dA * act'(H),
  dW2 = A^T dy, db2 = sum_rows dy, dW1 = x^T dH, db1 = sum_rows dH, dx = dH W1^T.
"""
import math

import numpy as np
from scipy.special import erf

GELU_ERF, RELU, GELU_TANH = 0, 1, 2
_K_TANH = math.sqrt(2.0 / math.pi)


def _as64(x):
    return None if x is None else np.asarray(x, dtype=np.float64)


def act_fwd(h, act):
    h = _as64(h)
    if act == GELU_ERF:
        return 0.5 * h * (1.0 + erf(h / math.sqrt(2.0)))
    if act == RELU:
        return np.maximum(h, 0.0)
    if act == GELU_TANH:
        return 0.5 * h * (1.0 + np.tanh(_K_TANH * (h + 0.044715 * h ** 3)))
    raise ValueError("unknown activation")


def act_grad(h, act):
    h = _as64(h)
    if act == GELU_ERF:
        cdf = 0.5 * (1.0 + erf(h / math.sqrt(2.0)))
        pdf = np.exp(-0.5 * h * h) / math.sqrt(2.0 * math.pi)
        return cdf + h * pdf
    if act == RELU:
        return (h > 0.0).astype(np.float64)
    if act == GELU_TANH:
        u = _K_TANH * (h + 0.044715 * h ** 3)
        t = np.tanh(u)
        du = _K_TANH * (1.0 + 3.0 * 0.044715 * h * h)
        return 0.5 * (1.0 + t) + 0.5 * h * (1.0 - t * t) * du
    raise ValueError("unknown activation")


def ffn_fwd(x, w1, b1, w2, b2, act=GELU_ERF):
    """y = act(x W1 + b1) W2 + b2 for x [T, d_model]."""
    x, w1, b1, w2, b2 = map(_as64, (x, w1, b1, w2, b2))
    h = x @ w1
    if b1 is not None:
        h = h + b1
    y = act_fwd(h, act) @ w2
    if b2 is not None:
        y = y + b2
    return y


def ffn_blockwise_fwd(x, w1, b1, w2, b2, block, act=GELU_ERF):
    """The same network applied to consecutive row blocks of ``block`` rows."""
    x = _as64(x)
    return np.concatenate([ffn_fwd(x[r:r + block], w1, b1, w2, b2, act)
                           for r in range(0, x.shape[0], block)], axis=0)


def ffn_bwd(x, w1, b1, w2, dy, act=GELU_ERF):
    """Returns (dx, dw1, db1, dw2, db2)."""
    x, w1, b1, w2, dy = map(_as64, (x, w1, b1, w2, dy))
    h = x @ w1
    if b1 is not None:
        h = h + b1
    a = act_fwd(h, act)
    da = dy @ w2.T
    dh = da * act_grad(h, act)
    return dh @ w1.T, x.T @ dh, dh.sum(axis=0), a.T @ dy, dy.sum(axis=0)


def linear_fwd(x, w, residual=None):
    """y = x W (+ residual)."""
    y = _as64(x) @ _as64(w)
    if residual is not None:
        y = y + _as64(residual)
    return y


def linear_bwd(x, w, dy):
    """Returns (dx, dw) for y = x W."""
    x, w, dy = map(_as64, (x, w, dy))
    return dy @ w.T, x.T @ dy
