"""Pins for the LLaMA-style layer oracle (CPU only).

RMSNorm against torch's rms_norm and autograd; RoPE against complex multiplication by
e^{i angle} (torch.polar on interleaved pairs), the identity at position 0, norm
preservation, the relative-position property <R_m q, R_n k> = <R_{m-n} q, k> and its
inverse; SwiGLU's activation against torch.nn.functional.silu and autograd; the layer and
the stack backward against central finite differences.
"""
import numpy as np
import pytest
import torch

from oracle import llama as L


def _rand(seed, *shape, scale=1.0):
    return np.random.default_rng(seed).standard_normal(shape) * scale


def test_rmsnorm_matches_torch_and_autograd():
    x, g, dy = _rand(1, 7, 16), _rand(2, 16), _rand(3, 7, 16)
    y, rstd = L.rmsnorm_fwd(x, g)
    tx = torch.from_numpy(x).requires_grad_()
    tg = torch.from_numpy(g).requires_grad_()
    ty = torch.nn.functional.rms_norm(tx, (16,), weight=tg, eps=L.EPS)
    np.testing.assert_allclose(y, ty.detach().numpy(), atol=1e-13)
    np.testing.assert_allclose(rstd, 1.0 / np.sqrt((x * x).mean(1) + L.EPS), atol=1e-13)
    ty.backward(torch.from_numpy(dy))
    dx, dg = L.rmsnorm_bwd(x, g, dy)
    np.testing.assert_allclose(dx, tx.grad.numpy(), atol=1e-12)
    np.testing.assert_allclose(dg, tg.grad.numpy(), atol=1e-12)


def test_rope_is_complex_rotation():
    x = _rand(4, 5, 3, 8)
    pos = np.array([0, 1, 7, 100, 65535])
    y = L.rope(x, pos)
    xc = torch.view_as_complex(torch.from_numpy(x).reshape(5, 3, 4, 2).contiguous())
    ang = torch.from_numpy(L.rope_angles(pos, 8))[:, None, :]
    rot = torch.polar(torch.ones_like(ang), ang)
    ref = torch.view_as_real(xc * rot).reshape(5, 3, 8).numpy()
    np.testing.assert_allclose(y, ref, atol=1e-12)
    np.testing.assert_allclose(L.rope_angles([1], 2)[0, 0], 1.0)  # theta_0 = base^0


def test_rope_properties():
    q, k = _rand(5, 1, 2, 16), _rand(6, 1, 2, 16)
    np.testing.assert_allclose(L.rope(q, [0]), q, atol=0)  # identity at position 0
    y = L.rope(q, [12345])
    pair_norm = lambda t: t[..., 0::2] ** 2 + t[..., 1::2] ** 2
    np.testing.assert_allclose(pair_norm(y), pair_norm(q), atol=1e-12)
    # relative position: <R_m q, R_n k> = <R_{m-n} q, k>
    for m, n in ((9, 4), (300, 299), (5, 40)):
        lhs = (L.rope(q, [m]) * L.rope(k, [n])).sum(-1)
        rhs = (L.rope(q, [m - n]) * k).sum(-1)
        np.testing.assert_allclose(lhs, rhs, atol=1e-11)
    np.testing.assert_allclose(L.rope(y, [12345], inverse=True), q, atol=1e-12)


def test_silu_matches_torch():
    u = np.linspace(-12, 12, 97)
    tu = torch.from_numpy(u).requires_grad_()
    ts = torch.nn.functional.silu(tu)
    np.testing.assert_allclose(L.silu(u), ts.detach().numpy(), atol=1e-14)
    ts.sum().backward()
    np.testing.assert_allclose(L.silu_grad(u), tu.grad.numpy(), atol=1e-14)


def test_swiglu_backward_matches_autograd():
    x, w1, w3, w2, dy = _rand(7, 5, 8), _rand(8, 8, 12), _rand(9, 8, 12), _rand(10, 12, 8), _rand(11, 5, 8)
    ts = [torch.from_numpy(t).requires_grad_() for t in (x, w1, w3, w2)]
    out = (torch.nn.functional.silu(ts[0] @ ts[1]) * (ts[0] @ ts[2])) @ ts[3]
    np.testing.assert_allclose(L.swiglu_fwd(x, w1, w3, w2), out.detach().numpy(), atol=1e-12)
    out.backward(torch.from_numpy(dy))
    for mine, t in zip(L.swiglu_bwd(x, w1, w3, w2, dy), ts):
        np.testing.assert_allclose(mine, t.grad.numpy(), atol=1e-11)


def _tiny_layer(seed, S=6, d=8, dff=6):
    r = np.random.default_rng(seed)
    w = lambda *s: r.standard_normal(s) * 0.3
    return (r.standard_normal((S, d)), 1.0 + 0.1 * r.standard_normal(d), w(d, d), w(d, d), w(d, d), w(d, d),
            1.0 + 0.1 * r.standard_normal(d), w(d, dff), w(d, dff), w(dff, d)), r.standard_normal((S, d))


def _fd(loss, arrays, idx, eps=1e-6):
    a = arrays[idx]
    num = np.zeros_like(a)
    for pos in np.ndindex(a.shape):
        old = a[pos]
        a[pos] = old + eps
        lp = loss()
        a[pos] = old - eps
        lm = loss()
        a[pos] = old
        num[pos] = (lp - lm) / (2 * eps)
    return num


@pytest.mark.parametrize("causal", [True, False])
def test_layer_backward_finite_differences(causal):
    params, dz = _tiny_layer(12)
    arrays = [p.copy() for p in params]
    H = 2
    loss = lambda: float((L.layer_fwd(*arrays, H, causal) * dz).sum())
    grads = L.layer_bwd(*arrays, dz, H, causal)
    for idx in range(len(arrays)):  # x, g1, wq, wk, wv, wo, g2, w1, w3, w2
        np.testing.assert_allclose(grads[idx], _fd(loss, arrays, idx), atol=2e-7, rtol=1e-6)


def test_stack_backward_finite_differences():
    p1, dz = _tiny_layer(13)
    p2, _ = _tiny_layer(14)
    x = p1[0].copy()
    layers = [list(p1[1:]), list(p2[1:])]
    loss = lambda: float((L.stack_fwd(x, layers, 2) * dz).sum())
    dx, grads = L.stack_bwd(x, layers, dz, 2)
    np.testing.assert_allclose(dx, _fd(loss, [x], 0), atol=2e-7, rtol=1e-6)
    for li in range(2):
        for pi in (0, 3, 6, 8):  # g1, wv, w1, w2 of each layer
            num = _fd(loss, layers[li], pi)
            np.testing.assert_allclose(grads[li][pi], num, atol=2e-7, rtol=1e-6)
    # one layer: the stack is the layer
    dx1, g1 = L.stack_bwd(x, layers[:1], dz, 2)
    ref = L.layer_bwd(x, *layers[0], dz, 2)
    np.testing.assert_allclose(dx1, ref[0], atol=1e-13)


def _torch_llama_layer(x, g1, wq, wk, wv, wo, g2, w1, w3, w2, H, causal=True):
    """The same pre-norm layer written with torch fp64 library routines: rms_norm, rotary
    embedding as complex multiplication (torch.polar on interleaved pairs), scaled dot-product
    attention with its own causal mask, silu."""
    F = torch.nn.functional
    S, d = x.shape
    D = d // H
    rms = lambda t, g: F.rms_norm(t, (d,), weight=g, eps=L.EPS)
    inv = L.ROPE_BASE ** (-torch.arange(0, D, 2, dtype=torch.float64) / D)
    ang = torch.arange(S, dtype=torch.float64)[:, None] * inv[None, :]
    rot = torch.polar(torch.ones_like(ang), ang)[:, None, :]  # [S, 1, D/2]

    def rope(t):
        tc = torch.view_as_complex(t.reshape(S, H, D // 2, 2))
        return torch.view_as_real(tc * rot).reshape(S, d)

    heads = lambda t: t.reshape(S, H, D).transpose(0, 1)
    n1 = rms(x, g1)
    a = F.scaled_dot_product_attention(heads(rope(n1 @ wq)), heads(rope(n1 @ wk)), heads(n1 @ wv), is_causal=causal)
    h = x + a.transpose(0, 1).reshape(S, d) @ wo
    n2 = rms(h, g2)
    return h + (F.silu(n2 @ w1) * (n2 @ w3)) @ w2


@pytest.mark.parametrize("causal", [True, False])
def test_layer_matches_torch_composition(causal):
    """The layer and its every gradient against the torch restatement and autograd."""
    params, dz = _tiny_layer(15, S=10, d=16, dff=12)
    H = 2
    z = L.layer_fwd(*params, H, causal)
    ts = [torch.from_numpy(p.copy()).requires_grad_() for p in params]
    tz = _torch_llama_layer(*ts, H, causal)
    np.testing.assert_allclose(z, tz.detach().numpy(), atol=1e-12)
    tz.backward(torch.from_numpy(dz))
    grads = L.layer_bwd(*params, dz, H, causal)
    for g, t in zip(grads, ts):  # x, g1, wq, wk, wv, wo, g2, w1, w3, w2
        np.testing.assert_allclose(g, t.grad.numpy(), atol=1e-11)


def test_stack_matches_torch_composition():
    """A 2-layer stack and its full-recomputation training step against autograd through
    the torch restatement applied twice."""
    p1, dz = _tiny_layer(16, S=10, d=16, dff=12)
    p2, _ = _tiny_layer(17, S=10, d=16, dff=12)
    x = p1[0]
    layers = [list(p1[1:]), list(p2[1:])]
    H = 2
    tx = torch.from_numpy(x.copy()).requires_grad_()
    tl = [[torch.from_numpy(p.copy()).requires_grad_() for p in ly] for ly in layers]
    tz = _torch_llama_layer(_torch_llama_layer(tx, *tl[0], H), *tl[1], H)
    np.testing.assert_allclose(L.stack_fwd(x, layers, H), tz.detach().numpy(), atol=1e-12)
    tz.backward(torch.from_numpy(dz))
    dx, grads = L.stack_bwd(x, layers, dz, H)
    np.testing.assert_allclose(dx, tx.grad.numpy(), atol=1e-11)
    for li in range(2):
        for g, t in zip(grads[li], tl[li]):
            np.testing.assert_allclose(g, t.grad.numpy(), atol=1e-11)


def test_layer_zero_query_key_closed_form():
    """With zero query and key weights every score is 0 (rotary embedding of zero is zero),
    so causal attention is the running mean of the value rows; the layer is then written
    out with numpy alone: n1 = x g1 / rms(x), h = x + P (n1 Wv) Wo with P the lower-triangular
    averaging matrix, z = h + (silu(n2 W1) * (n2 W3)) W2 with n2 = h g2 / rms(h)."""
    S, d, H, dff = 24, 16, 4, 20
    x = _rand(70, S, d)
    g1, g2 = 1.0 + 0.1 * _rand(71, d), 1.0 + 0.1 * _rand(72, d)
    wv, wo = _rand(73, d, d, scale=0.4), _rand(74, d, d, scale=0.4)
    w1, w3, w2 = _rand(75, d, dff, scale=0.4), _rand(76, d, dff, scale=0.4), _rand(77, dff, d, scale=0.4)
    zero = np.zeros((d, d))
    z = L.layer_fwd(x, g1, zero, zero, wv, wo, g2, w1, w3, w2, H)
    rms = lambda t: np.sqrt((t * t).mean(axis=1, keepdims=True) + L.EPS)
    n1 = x / rms(x) * g1
    P = np.tril(np.ones((S, S))) / np.arange(1, S + 1)[:, None]
    h = x + (P @ (n1 @ wv)) @ wo
    n2 = h / rms(h) * g2
    u = n2 @ w1
    np.testing.assert_allclose(z, h + ((u / (1.0 + np.exp(-u))) * (n2 @ w3)) @ w2, atol=1e-12)

