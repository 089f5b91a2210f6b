"""Pins for the FFN / projection / layer oracles (CPU only).

The activation and the network are checked against torch's fp64 CPU routines and
autograd (a library special case), the blockwise form against the whole-sequence
form, and the backward passes against central finite differences.
"""
import numpy as np
import pytest
import torch

from oracle import ffn as F
from oracle import layer as L


def _rand(seed, *shape, std=1.0):
    return np.random.default_rng(seed).standard_normal(shape) * std


_TORCH_ACT = {
    F.GELU_ERF: lambda h: torch.nn.functional.gelu(h),
    F.RELU: torch.relu,
    F.GELU_TANH: lambda h: torch.nn.functional.gelu(h, approximate="tanh"),
}


@pytest.mark.parametrize("act", [F.GELU_ERF, F.RELU, F.GELU_TANH])
def test_activation_and_derivative_match_torch(act):
    h = np.linspace(-6, 6, 1001)
    th = torch.from_numpy(h).requires_grad_()
    y = _TORCH_ACT[act](th)
    y.sum().backward()
    np.testing.assert_allclose(F.act_fwd(h, act), y.detach().numpy(), atol=1e-15)
    mask = np.abs(h) > 1e-9  # ReLU's derivative at 0 is a convention
    np.testing.assert_allclose(F.act_grad(h, act)[mask], th.grad.numpy()[mask], atol=1e-14)


@pytest.mark.parametrize("bias", [False, True])
@pytest.mark.parametrize("act", [F.GELU_ERF, F.RELU, F.GELU_TANH])
def test_ffn_forward_backward_match_torch_autograd(act, bias):
    T, dm, dff = 24, 16, 40
    x, w1, w2, dy = _rand(1, T, dm), _rand(2, dm, dff, std=0.3), _rand(3, dff, dm, std=0.3), _rand(4, T, dm)
    b1 = _rand(5, dff, std=0.3) if bias else None
    b2 = _rand(6, dm, std=0.3) if bias else None
    y = F.ffn_fwd(x, w1, b1, w2, b2, act)
    tx, tw1, tw2 = (torch.from_numpy(a).requires_grad_() for a in (x, w1, w2))
    tb1 = torch.from_numpy(b1).requires_grad_() if bias else None
    tb2 = torch.from_numpy(b2).requires_grad_() if bias else None
    h = tx @ tw1 + (tb1 if bias else 0)
    ty = _TORCH_ACT[act](h) @ tw2 + (tb2 if bias else 0)
    np.testing.assert_allclose(y, ty.detach().numpy(), atol=1e-12)
    ty.backward(torch.from_numpy(dy))
    dx, dw1, db1, dw2, db2 = F.ffn_bwd(x, w1, b1, w2, dy, act)
    np.testing.assert_allclose(dx, tx.grad.numpy(), atol=1e-12)
    np.testing.assert_allclose(dw1, tw1.grad.numpy(), atol=1e-12)
    np.testing.assert_allclose(dw2, tw2.grad.numpy(), atol=1e-12)
    if bias:
        np.testing.assert_allclose(db1, tb1.grad.numpy(), atol=1e-12)
        np.testing.assert_allclose(db2, tb2.grad.numpy(), atol=1e-12)


def test_blockwise_ffn_equals_full():
    x, w1, w2 = _rand(7, 64, 8), _rand(8, 8, 32), _rand(9, 32, 8)
    b1, b2 = _rand(10, 32), _rand(11, 8)
    full = F.ffn_fwd(x, w1, b1, w2, b2)
    for block in (1, 7, 16, 64):
        np.testing.assert_allclose(F.ffn_blockwise_fwd(x, w1, b1, w2, b2, block), full, atol=1e-13)


def test_ffn_backward_finite_differences():
    x, w1, w2, dy = _rand(12, 3, 4), _rand(13, 4, 6), _rand(14, 6, 4), _rand(15, 3, 4)
    b1 = _rand(16, 6)
    dx, dw1, db1, dw2, db2 = F.ffn_bwd(x, w1, b1, w2, dy)
    loss = lambda x_, w1_, b1_, w2_: float((F.ffn_fwd(x_, w1_, b1_, w2_, None) * dy).sum())
    eps = 1e-6
    for idx, grad in enumerate((dx, dw1, db1, dw2)):
        args = [x, w1, b1, w2]
        num = np.zeros_like(args[idx])
        for pos in np.ndindex(num.shape):
            ap, am = [a.copy() for a in args], [a.copy() for a in args]
            ap[idx][pos] += eps
            am[idx][pos] -= eps
            num[pos] = (loss(*ap) - loss(*am)) / (2 * eps)
        np.testing.assert_allclose(grad, num, atol=1e-8)
    np.testing.assert_allclose(db2, dy.sum(axis=0), atol=1e-14)


def test_linear_forward_backward():
    x, w, r, dy = _rand(17, 10, 6), _rand(18, 6, 5), _rand(19, 10, 5), _rand(20, 10, 5)
    np.testing.assert_allclose(F.linear_fwd(x, w, r), np.einsum("td,de->te", x, w) + r, atol=1e-13)
    tx, tw = torch.from_numpy(x).requires_grad_(), torch.from_numpy(w).requires_grad_()
    (tx @ tw).backward(torch.from_numpy(dy))
    dx, dw = F.linear_bwd(x, w, dy)
    np.testing.assert_allclose(dx, tx.grad.numpy(), atol=1e-13)
    np.testing.assert_allclose(dw, tw.grad.numpy(), atol=1e-13)


def _torch_layer(x, wq, wk, wv, wo, w1, w2, H):
    S, dm = x.shape
    D = dm // H
    heads = lambda t: t.reshape(1, S, H, D).permute(0, 2, 1, 3)
    a = torch.nn.functional.scaled_dot_product_attention(heads(x @ wq), heads(x @ wk), heads(x @ wv), is_causal=True)
    y = x + a.permute(0, 2, 1, 3).reshape(S, dm) @ wo
    return y + torch.nn.functional.gelu(y @ w1) @ w2


def test_layer_matches_torch_composition():
    S, dm, H, dff = 20, 16, 4, 24
    ws = [_rand(30 + i, *shape, std=0.3) for i, shape in
          enumerate([(dm, dm)] * 4 + [(dm, dff), (dff, dm)])]
    x, dz = _rand(21, S, dm), _rand(22, S, dm)
    z = L.layer_fwd(x, *ws, n_heads=H)
    tx = torch.from_numpy(x).requires_grad_()
    tws = [torch.from_numpy(w).requires_grad_() for w in ws]
    tz = _torch_layer(tx, *tws, H)
    np.testing.assert_allclose(z, tz.detach().numpy(), atol=1e-12)
    tz.backward(torch.from_numpy(dz))
    grads = L.layer_bwd(x, *ws, dz, n_heads=H)
    for g, t in zip(grads, [tx] + tws):
        np.testing.assert_allclose(g, t.grad.numpy(), atol=1e-11)


def test_layer_backward_finite_differences():
    S, dm, H, dff = 4, 4, 2, 6
    ws = [_rand(40 + i, *shape, std=0.5) for i, shape in
          enumerate([(dm, dm)] * 4 + [(dm, dff), (dff, dm)])]
    x, dz = _rand(23, S, dm), _rand(24, S, dm)
    grads = L.layer_bwd(x, *ws, dz, n_heads=H)
    loss = lambda args: float((L.layer_fwd(*args, n_heads=H) * dz).sum())
    eps = 1e-6
    base = [x] + ws
    for idx in (0, 1, 4, 6):  # x, wq, wo, w2
        num = np.zeros_like(base[idx])
        for pos in np.ndindex(num.shape):
            ap, am = [a.copy() for a in base], [a.copy() for a in base]
            ap[idx][pos] += eps
            am[idx][pos] -= eps
            num[pos] = (loss(ap) - loss(am)) / (2 * eps)
        np.testing.assert_allclose(grads[idx], num, atol=1e-7)


def test_layer_uniform_attention_closed_form():
    """With Wq = Wk = 0 every score is 0, so causal attention is the running mean of the
    value rows: A = P (X Wv) with P the lower-triangular averaging matrix, and the layer
    is Z = Y + GeLU(Y W1) W2 with Y = X + A Wo, written here with numpy and scipy's erf
    alone (no oracle code)."""
    from scipy.special import erf
    S, dm, H, dff = 24, 16, 4, 20
    x = _rand(50, S, dm)
    wv, wo, w1, w2 = (_rand(51 + i, *shape, std=0.4) for i, shape in
                      enumerate([(dm, dm), (dm, dm), (dm, dff), (dff, dm)]))
    zero = np.zeros((dm, dm))
    z = L.layer_fwd(x, zero, zero, wv, wo, w1, w2, n_heads=H)
    P = np.tril(np.ones((S, S))) / np.arange(1, S + 1)[:, None]
    y = x + (P @ (x @ wv)) @ wo
    h = y @ w1
    np.testing.assert_allclose(z, y + (0.5 * h * (1.0 + erf(h / np.sqrt(2.0)))) @ w2, atol=1e-12)
    # without causal masking the mean runs over every row
    z_full = L.layer_fwd(x, zero, zero, wv, wo, w1, w2, n_heads=H, causal=False)
    y_full = x + np.mean(x @ wv, axis=0, keepdims=True) @ wo
    h_full = y_full @ w1
    np.testing.assert_allclose(z_full, y_full + (0.5 * h_full * (1.0 + erf(h_full / np.sqrt(2.0)))) @ w2,
                               atol=1e-12)

