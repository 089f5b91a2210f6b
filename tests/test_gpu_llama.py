"""GPU parity of the LLaMA-style entry points (RMSNorm, RoPE, SwiGLU, the layer and a
two-layer training step) against the fp64 oracle (oracle/llama.py).

Tolerances (bf16 storage of every activation, float32 arithmetic):
  * RMSNorm / RoPE outputs: |gpu - ref| <= 1e-2 * max(1, |ref|); RMSNorm dg (float32 sums
    over rows): <= 1e-2 * max(1, rms(ref)).
  * SwiGLU, layer and stack at small widths: outputs 2e-2, input gradients 5e-2, scaled as
    above; weight and gain gradients max |err| <= 5e-2 * max(1, rms(ref)) (as the
    Algorithm 1 layer tests).
"""
import numpy as np
import pytest
import torch

import paper_2310_01889_amd as ra
from paper_2310_01889_amd import synth
from oracle import llama as OL
from tests.gpu_util import dev, log, np64

pytestmark = pytest.mark.gpu


def _scaled_err(got, ref):
    g, r = np64(got), np.asarray(ref)
    return float((np.abs(g - r) / np.maximum(1.0, np.abs(r))).max())


def _grad_ok(got, ref, tol=5e-2, name=""):
    g, r = np64(got), np.asarray(ref)
    bound = tol * max(1.0, float(np.sqrt(np.mean(r * r))))
    err = float(np.abs(g - r).max())
    log("   %s grad err %.3e bound %.3e" % (name, err, bound))
    return err <= bound


@pytest.mark.parametrize("T,d", [(512, 256), (256, 4096), (96, 1024)])
def test_rmsnorm(T, d):
    gen = torch.Generator().manual_seed(200 + d)
    x = (torch.randn(T, d, generator=gen) * 3).to(torch.bfloat16)
    g = (1 + 0.1 * torch.randn(d, generator=gen)).to(torch.bfloat16)
    dy = torch.randn(T, d, generator=gen)
    dres = torch.randn(T, d, generator=gen).to(torch.bfloat16)
    xd, gd = dev(x, g)
    y = torch.empty_like(xd)
    rstd = torch.empty(T, device="cuda")
    ra.rms_norm_fwd(xd, gd, y, rstd)
    y_ref, r_ref = OL.rmsnorm_fwd(np64(x), np64(g))
    ey = _scaled_err(y, y_ref)
    er = float(np.abs(np64(rstd) - r_ref).max() / r_ref.max())
    log("rmsnorm T=%d d=%d: y %.3e rstd(rel) %.3e" % (T, d, ey, er))
    assert ey <= 1e-2 and er <= 1e-5
    dx_ref, dg_ref = OL.rmsnorm_bwd(np64(x), np64(g), dy.numpy())
    for res in (None, dres):
        dx = torch.empty_like(xd)
        dg = torch.empty(d, device="cuda")
        ra.rms_norm_bwd(xd, gd, dev(dy), None if res is None else dev(res), dx, dg)
        ref = dx_ref if res is None else dx_ref + np64(res)
        edx = _scaled_err(dx, ref)
        log("   dx %.3e" % edx)
        assert edx <= 1e-2
        assert _grad_ok(dg, dg_ref, 1e-2, "dg")


@pytest.mark.parametrize("pos0", [0, 60000])
@pytest.mark.parametrize("D", [64, 128])
def test_rope(pos0, D):
    S, H = 256, 3
    gen = torch.Generator().manual_seed(300 + D)
    x = torch.randn(S, H, D, generator=gen).to(torch.bfloat16)
    y = dev(x).clone()
    ra.rope_apply(y, pos0)
    pos = np.arange(pos0, pos0 + S)
    ref = OL.rope(np64(x), pos)
    e = _scaled_err(y, ref)
    ra.rope_apply(y, pos0, inverse=True)
    e_inv = _scaled_err(y, np64(x))
    log("rope D=%d pos0=%d: fwd %.3e, fwd+inverse vs x %.3e" % (D, pos0, e, e_inv))
    assert e <= 1e-2 and e_inv <= 2e-2
    y0 = dev(x).clone()
    ra.rope_apply(y0, 0)
    assert torch.equal(y0[0].cpu(), x[0])  # position 0 is the identity


def test_swiglu_forward_backward():
    T, dm, dff, blk = 512, 256, 512, 256
    x, layers, dy = synth.llama_layer_inputs(400, T, dm, dff)
    w1, w3, w2 = layers[0][6], layers[0][7], layers[0][8]
    args = dev(x, w1, w3, w2)
    y = torch.empty((T, dm), dtype=torch.bfloat16, device="cuda")
    ra.swiglu_ffn(*args, None, y, blk)
    y_ref = OL.swiglu_fwd(*(np64(t) for t in (x, w1, w3, w2)))
    ey = _scaled_err(y, y_ref)
    log("swiglu y %.3e" % ey)
    assert ey <= 2e-2
    dx = torch.empty_like(args[0])
    f = lambda *s: torch.empty(*s, dtype=torch.float32, device="cuda")
    dw1, dw3, dw2 = f(dm, dff), f(dm, dff), f(dff, dm)
    ra.swiglu_ffn_bwd(*args, dev(dy), dx, dw1, dw3, dw2, blk)
    ref = OL.swiglu_bwd(*(np64(t) for t in (x, w1, w3, w2, dy)))
    edx = _scaled_err(dx, ref[0])
    log("   dx %.3e" % edx)
    assert edx <= 5e-2
    for got, r, n in zip((dw1, dw3, dw2), ref[1:], ("w1", "w3", "w2")):
        assert _grad_ok(got, r, name=n)


def _run_layer(seed, S, dm, H, dff, N, n_layers=1):
    x, layers, dz = synth.llama_layer_inputs(seed, S, dm, dff, n_layers)
    xd, dzd = dev(x), dev(dz)
    pd = [[t.cuda() for t in p] for p in layers]
    return x, layers, dz, xd, pd, dzd


@pytest.mark.parametrize("N", [1, 4])
def test_llama_layer_small(N):
    S, dm, H, dff = 1024, 256, 2, 512
    log("llama layer small N=%d" % N)
    x, layers, dz, xd, pd, dzd = _run_layer(410 + N, S, dm, H, dff, N)
    z = torch.empty_like(xd)
    ra.llama_layer_fwd(xd, pd[0], z, H, N)
    p64 = [np64(t) for t in layers[0]]
    z_ref = OL.layer_fwd(np64(x), *p64, H)
    ez = _scaled_err(z, z_ref)
    log("   z %.3e" % ez)
    assert ez <= 2e-2
    dx = torch.empty_like(xd)
    f = lambda t: torch.empty(t.shape, dtype=torch.float32, device="cuda")
    grads = [f(t) for t in pd[0]]
    ra.llama_layer_bwd(xd, pd[0], dzd, dx, grads, H, N)
    torch.cuda.synchronize()
    ref = OL.layer_bwd(np64(x), *p64, np64(dz), H)
    edx = _scaled_err(dx, ref[0])
    log("   dx %.3e" % edx)
    assert edx <= 5e-2
    names = ("g1", "wq", "wk", "wv", "wo", "g2", "w1", "w3", "w2")
    for g, r, n in zip(grads, ref[1:], names):
        assert _grad_ok(g, r, name=n)


def test_llama_stack_two_layers():
    S, dm, H, dff, N = 512, 256, 2, 512, 2
    x, layers, dz, xd, pd, dzd = _run_layer(420, S, dm, H, dff, N, n_layers=2)
    z, dx = torch.empty_like(xd), torch.empty_like(xd)
    grads = [[torch.empty(t.shape, dtype=torch.float32, device="cuda") for t in p] for p in pd]
    ra.llama_stack_train_step(xd, pd, dzd, z, dx, grads, H, N)
    torch.cuda.synchronize()
    p64 = [[np64(t) for t in p] for p in layers]
    z_ref = OL.stack_fwd(np64(x), p64, H)
    dx_ref, g_ref = OL.stack_bwd(np64(x), p64, np64(dz), H)
    ez, edx = _scaled_err(z, z_ref), _scaled_err(dx, dx_ref)
    log("stack z %.3e dx %.3e" % (ez, edx))
    assert ez <= 2e-2 and edx <= 5e-2
    for li in range(2):
        for g, r in zip(grads[li], g_ref[li]):
            assert _grad_ok(g, r, name="layer%d" % li)
    # the step's forward output is the layer forward applied twice
    z1 = torch.empty_like(xd)
    z2 = torch.empty_like(xd)
    ra.llama_layer_fwd(xd, pd[0], z1, H, N)
    ra.llama_layer_fwd(z1, pd[1], z2, H, N)
    assert torch.equal(z2, z)


def _rel_rms(got, ref):
    g, r = np64(got), np.asarray(ref)
    return float(np.sqrt(np.mean((g - r) ** 2)) / max(1e-30, np.sqrt(np.mean(r * r))))


@pytest.mark.slow
def test_llama_layer_model_width_short_sequence():
    """LLaMA-7B widths (d_model 4096 = 32 heads x 128, d_ff 11008) on a 2048-token sequence
    in 8 host blocks of 256, forward and backward in full.  At these widths bf16 storage of
    the intermediates sets the floor (tests/bf16_error_model.py at this shape: max scaled
    error 6.6e-2 for z and 1.9e-1 for dx -- 2.3e-1 at 512 tokens --, query/key weight
    gradients max |err| = 5.5e-2 * rms, relative RMS < 1e-2 everywhere).  Bounds, about 1.7x
    the floor: z relative RMS <= 2e-2 and max scaled <= 1.2e-1; dx relative RMS <= 5e-2 and max
    scaled <= 4e-1; weight and gain gradients relative RMS <= 2e-2 and
    max |err| <= 8e-2 * max(1, rms(ref))."""
    S, dm, H, dff, N = 2048, 4096, 32, 11008, 8
    x, layers, dz, xd, pd, dzd = _run_layer(430, S, dm, H, dff, N)
    z, dx = torch.empty_like(xd), torch.empty_like(xd)
    ra.llama_layer_fwd(xd, pd[0], z, H, N)
    grads = [torch.empty(t.shape, dtype=torch.float32, device="cuda") for t in pd[0]]
    ra.llama_layer_bwd(xd, pd[0], dzd, dx, grads, H, N)
    torch.cuda.synchronize()
    p64 = [np64(t) for t in layers[0]]
    z_ref = OL.layer_fwd(np64(x), *p64, H)
    ez, rz = _scaled_err(z, z_ref), _rel_rms(z, z_ref)
    log("   z scaled err %.3e rel rms %.3e" % (ez, rz))
    ref = OL.layer_bwd(np64(x), *p64, np64(dz), H)
    edx, rdx = _scaled_err(dx, ref[0]), _rel_rms(dx, ref[0])
    log("   dx scaled err %.3e rel rms %.3e" % (edx, rdx))
    assert rz <= 2e-2 and ez <= 1.2e-1
    assert rdx <= 5e-2 and edx <= 4e-1
    for g, r, n in zip(grads, ref[1:], ("g1", "wq", "wk", "wv", "wo", "g2", "w1", "w3", "w2")):
        rr = _rel_rms(g, r)
        log("   %s rel rms %.3e" % (n, rr))
        assert rr <= 2e-2 and _grad_ok(g, r, 8e-2, name=n)


@pytest.mark.slow
def test_llama_layer_full_size_forward_sampled_rows():
    """The benchmarked size (S = 65536 in 8 host blocks of 8192, d_model 4096 = 32 heads x 128,
    d_ff 11008): rows of z in the first host block and at the start of the second, against
    the oracle layer on the prefix x[:8200] -- a causal row depends only on the rows before
    it, and the prefix keeps the positions (RoPE) of the full sequence.  Bounds as the
    model-width test: relative RMS <= 2e-2, max scaled <= 1.2e-1."""
    S, dm, H, dff, N = 65536, 4096, 32, 11008, 8
    x, layers, _, xd, pd, _ = _run_layer(440, S, dm, H, dff, N)
    z = torch.empty_like(xd)
    ra.llama_layer_fwd(xd, pd[0], z, H, N)
    torch.cuda.synchronize()
    rows = np.array([0, 1, 777, 4095, 8191, 8192, 8199])
    rmax = int(rows.max()) + 1
    p64 = [np64(t) for t in layers[0]]
    z_ref = OL.layer_fwd(np64(x[:rmax]), *p64, H)[rows]
    zs = z[torch.from_numpy(rows).cuda()]
    ez, rz = _scaled_err(zs, z_ref), _rel_rms(zs, z_ref)
    log("   sampled z scaled err %.3e rel rms %.3e" % (ez, rz))
    assert rz <= 2e-2 and ez <= 1.2e-1
