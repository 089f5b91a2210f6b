"""GPU parity of the blockwise FFN and projection entry points against the fp64 oracle.

Tolerance (magnitude-scaled, because products of many bf16 terms grow with the
reduction length): |gpu - ref| <= tol * max(1, |ref|) elementwise, tol = 2e-2 for
outputs and 5e-2 for gradients; weight gradients (float32 sums over every row) use
max |gpu - ref| <= 5e-2 * max(1, rms(ref)).
"""
import numpy as np
import pytest
import torch

import paper_2310_01889_amd as ra
from paper_2310_01889_amd import synth
from oracle import ffn as OF
from tests.gpu_util import dev, log, np64

pytestmark = pytest.mark.gpu


def _scaled_ok(got, ref, tol):
    g, r = np64(got), np.asarray(ref)
    err = np.abs(g - r) / np.maximum(1.0, np.abs(r))
    log("   scaled err %.3e (max|ref| %.3e)" % (err.max(), np.abs(r).max()))
    return float(err.max()) <= tol


def _wgrad_ok(got, ref, tol=5e-2):
    g, r = np64(got), np.asarray(ref)
    bound = tol * max(1.0, float(np.sqrt(np.mean(r * r))))
    log("   wgrad err %.3e bound %.3e" % (np.abs(g - r).max(), bound))
    return float(np.abs(g - r).max()) <= bound


@pytest.mark.parametrize("act", [ra.ACT_GELU_ERF, ra.ACT_RELU, ra.ACT_GELU_TANH])
@pytest.mark.parametrize("bias", [False, True])
def test_blockwise_ffn_forward(act, bias):
    T, dm, dff, blk = 768, 256, 512, 256
    log("ffn fwd act=%d bias=%d" % (act, bias))
    x, w1, b1, w2, b2, _ = synth.ffn_inputs(20 + act, T, dm, dff, with_bias=bias)
    y = torch.empty((T, dm), dtype=torch.bfloat16, device="cuda")
    ra.blockwise_ffn(dev(x), dev(w1), dev(b1) if bias else None, dev(w2), dev(b2) if bias else None, y, blk, act)
    torch.cuda.synchronize()
    ref = OF.ffn_fwd(np64(x), np64(w1), np64(b1) if bias else None, np64(w2), np64(b2) if bias else None, act)
    assert _scaled_ok(y, ref, 2e-2)


@pytest.mark.parametrize("act", [ra.ACT_GELU_ERF, ra.ACT_RELU, ra.ACT_GELU_TANH])
def test_blockwise_ffn_backward(act):
    T, dm, dff, blk = 768, 256, 512, 256
    log("ffn bwd act=%d" % act)
    x, w1, b1, w2, b2, dy = synth.ffn_inputs(30 + act, T, dm, dff, with_bias=True, with_grad=True)
    xd, w1d, b1d, w2d, dyd = dev(x, w1, b1, w2, dy)
    dx = torch.empty_like(xd)
    dw1 = torch.empty((dm, dff), dtype=torch.float32, device="cuda")
    db1 = torch.empty((dff,), dtype=torch.float32, device="cuda")
    dw2 = torch.empty((dff, dm), dtype=torch.float32, device="cuda")
    db2 = torch.empty((dm,), dtype=torch.float32, device="cuda")
    ra.blockwise_ffn_bwd(xd, w1d, b1d, w2d, dyd, dx, dw1, db1, dw2, db2, blk, act)
    torch.cuda.synchronize()
    rdx, rdw1, rdb1, rdw2, rdb2 = OF.ffn_bwd(np64(x), np64(w1), np64(b1), np64(w2), np64(dy), act)
    assert _scaled_ok(dx, rdx, 5e-2)
    for g, r in ((dw1, rdw1), (db1, rdb1), (dw2, rdw2), (db2, rdb2)):
        assert _wgrad_ok(g, r)


def test_blockwise_ffn_block_size_invariance():
    """One block of all rows and 256-row blocks give bit-identical outputs (rows are
    independent and each row's arithmetic is the same)."""
    T, dm, dff = 1024, 256, 512
    x, w1, b1, w2, b2, _ = synth.ffn_inputs(40, T, dm, dff, with_bias=True)
    args = dev(x, w1, b1, w2, b2)
    y1 = torch.empty((T, dm), dtype=torch.bfloat16, device="cuda")
    y2 = torch.empty_like(y1)
    ra.blockwise_ffn(*args, y1, T)
    ra.blockwise_ffn(*args, y2, 256)
    torch.cuda.synchronize()
    assert torch.equal(y1, y2)


# The GEMM walks K in steps of 32 through a five-stage ring, in groups of five steps plus a
# remainder of 0..4 steps: K = 512 (16 steps), 768 (24), 1280 (40) and 256 (8) cover
# remainders 1, 4, 0 and 3 across the forward (K = d_in), dX (K = d_out) and dW (K = block)
# products.
@pytest.mark.parametrize("T,di,do,blk", [(512, 512, 256, 256), (512, 768, 1280, 256), (768, 1280, 768, 768)])
def test_blockwise_linear_forward_backward(T, di, do, blk):
    log("linear T=%d d_in=%d d_out=%d block=%d" % (T, di, do, blk))
    g = torch.Generator().manual_seed(50 + di)
    x = torch.randn(T, di, generator=g).to(torch.bfloat16)
    w = (torch.randn(di, do, generator=g) * 0.02).to(torch.bfloat16)
    r = torch.randn(T, do, generator=g).to(torch.bfloat16)
    dy = torch.randn(T, do, generator=g).to(torch.bfloat16)
    xd, wd, rd, dyd = dev(x, w, r, dy)
    y = torch.empty((T, do), dtype=torch.bfloat16, device="cuda")
    ra.blockwise_linear(xd, wd, rd, y, blk)
    dx = torch.empty_like(xd)
    dw = torch.empty((di, do), dtype=torch.float32, device="cuda")
    ra.blockwise_linear_bwd(xd, wd, dyd, dx, dw, blk)
    torch.cuda.synchronize()
    assert _scaled_ok(y, OF.linear_fwd(np64(x), np64(w), np64(r)), 2e-2)
    rdx, rdw = OF.linear_bwd(np64(x), np64(w), np64(dy))
    assert _scaled_ok(dx, rdx, 5e-2)
    assert _wgrad_ok(dw, rdw)


def test_ffn_rejects_unsupported_shapes():
    x = torch.zeros((300, 256), dtype=torch.bfloat16, device="cuda")
    w1 = torch.zeros((256, 512), dtype=torch.bfloat16, device="cuda")
    w2 = torch.zeros((512, 256), dtype=torch.bfloat16, device="cuda")
    y = torch.full((300, 256), 3.0, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(ra.RingAttnError) as e:
        ra.blockwise_ffn(x, w1, None, w2, None, y, 300)
    assert e.value.code == 2
    torch.cuda.synchronize()
    assert bool((y == 3.0).all())
