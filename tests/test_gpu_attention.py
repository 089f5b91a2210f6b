"""GPU parity of the ring-attention entry points against the fp64 CPU oracle.

Every case draws seeded inputs (paper_2310_01889_amd.synth), runs the HIP library through
its C ABI, and compares element by element with oracle/ on the same values.
Tolerances: float32 path max |err| <= 1e-5; bf16 path <= 2e-2 on o and lse, <= 5e-2 on
dq, dk, dv (absolute, against the fp64 oracle).
"""
import itertools

import numpy as np
import pytest
import torch

import paper_2310_01889_amd as ra
from paper_2310_01889_amd import synth
from oracle import attention as OA
from oracle import ring as OR
from tests.gpu_util import dev, log, max_err, np64

pytestmark = pytest.mark.gpu

TOL_F32 = 1e-5
TOL_O = 2e-2
TOL_G = 5e-2


def _fwd_case(seed, B, S, H, D, N, causal, dtype=torch.bfloat16):
    log("fwd case seed=%d B=%d S=%d H=%d D=%d N=%d causal=%d %s" % (seed, B, S, H, D, N, causal, dtype))
    q, k, v = synth.attention_inputs(seed, B, S, H, D, dtype)
    o, lse = ra.attention_fwd(*dev(q, k, v), N, causal)
    torch.cuda.synchronize()
    o_ref, lse_ref = OA.attention_fwd(np64(q), np64(k), np64(v), bool(causal))
    return o, lse, o_ref, lse_ref, (q, k, v)


def test_tiny_causal_fp32_config():
    """B=1, H=1, S=1024, D=64, float32, ring of 4 hosts with 256-token blocks."""
    o, lse, o_ref, lse_ref, _ = _fwd_case(1, 1, 1024, 1, 64, 4, 1, torch.float32)
    assert max_err(o, o_ref) <= TOL_F32
    assert max_err(lse, lse_ref) <= TOL_F32


@pytest.mark.parametrize("N", [1, 2, 4])
@pytest.mark.parametrize("causal", [0, 1])
def test_fp32_forward_hosts(N, causal):
    o, lse, o_ref, lse_ref, _ = _fwd_case(2, 2, 512, 3, 64, N, causal, torch.float32)
    assert max_err(o, o_ref) <= TOL_F32
    assert max_err(lse, lse_ref) <= TOL_F32


def test_fp32_forward_d128():
    o, lse, o_ref, lse_ref, _ = _fwd_case(3, 1, 256, 2, 128, 2, 1, torch.float32)
    assert max_err(o, o_ref) <= TOL_F32
    assert max_err(lse, lse_ref) <= TOL_F32


@pytest.mark.parametrize("D", [64, 128])
@pytest.mark.parametrize("N", [1, 2, 4, 8])
@pytest.mark.parametrize("causal", [0, 1])
def test_bf16_forward_hosts(D, N, causal):
    o, lse, o_ref, lse_ref, _ = _fwd_case(4, 2, 1024, 3, D, N, causal)
    eo, el = max_err(o, o_ref), max_err(lse, lse_ref)
    log("  max|o err| %.3e  max|lse err| %.3e" % (eo, el))
    assert eo <= TOL_O and el <= TOL_O


def test_bf16_forward_zero_query_prefix_mean_and_first_token():
    """Q = 0: causal row r is the mean of V_0..V_r and lse = ln(r+1); row 0 is V_0 exactly."""
    B, S, H, D = 1, 1024, 2, 128
    _, k, v = synth.attention_inputs(5, B, S, H, D)
    q = torch.zeros_like(v)
    o, lse = ra.attention_fwd(*dev(q, k, v), 4, True)
    torch.cuda.synchronize()
    prefix = np.cumsum(np64(v), axis=1) / np.arange(1, S + 1)[None, :, None, None]
    assert max_err(o, prefix) <= TOL_O
    assert max_err(lse, np.broadcast_to(np.log(np.arange(1, S + 1)), (B, H, S))) <= TOL_O
    assert torch.equal(o[:, 0].cpu(), v[:, 0])


def test_bf16_forward_invariant_to_block_order():
    B, S, H, D, N = 1, 1024, 2, 128, 4
    q, k, v = synth.attention_inputs(6, B, S, H, D)
    qd, kd, vd = dev(q, k, v)
    o_ref, lse_ref = OA.attention_fwd(np64(q), np64(k), np64(v), True)
    rng = np.random.default_rng(0)
    orders = [[list(rng.permutation(N)) for _ in range(N)] for _ in range(3)]
    orders.append([[(i - t) % N for t in range(N)] for i in range(N)])
    for order in orders:
        log("order %s" % order)
        o = torch.empty_like(qd)
        lse = torch.empty((B, H, S), dtype=torch.float32, device="cuda")
        ra.ring_attn_fwd_ordered(qd, kd, vd, o, lse, N, True, order)
        torch.cuda.synchronize()
        assert max_err(o, o_ref) <= TOL_O
        assert max_err(lse, lse_ref) <= TOL_O


@pytest.mark.parametrize("S,N,causal,full,B,D", [(16384, 1, 1, True, 1, 128), (32768, 2, 1, False, 1, 128),
                                                 (32768, 2, 0, False, 1, 128), (32768, 2, 1, False, 2, 128),
                                                 (16384, 1, 1, True, 1, 64), (32768, 2, 1, False, 1, 64)])
def test_bf16_forward_long_blocks(S, N, causal, full, B, D):
    """Blocks of 16384 keys or more: with D = 128 they run the eight-wave kernel (256 queries
    per workgroup), with D = 64 the four-wave kernel over as many key tiles.  A whole head in
    full on the first case of each (diagonal tiles of every workgroup), otherwise one sampled
    row of every 32-row wave tile of both heads (of every batch) plus the block edges."""
    H = 2
    q, k, v = synth.attention_inputs(13, B, S, H, D)
    o, lse = ra.attention_fwd(*dev(q, k, v), N, causal)
    torch.cuda.synchronize()
    o, lse = o.cpu(), lse.cpu()
    c = S // N
    worst = [0.0, 0.0]
    for h in range(H):
        hs = slice(h, h + 1)
        if full and h == 0:
            o_ref, lse_ref = OA.attention_fwd(np64(q[:, :, hs]), np64(k[:, :, hs]), np64(v[:, :, hs]), bool(causal))
            worst[0] = max(worst[0], max_err(o[:, :, hs], o_ref))
            worst[1] = max(worst[1], max_err(lse[:, hs], lse_ref))
            continue
        rng = np.random.default_rng(300 + h)
        rows = np.arange(0, S, 32) + rng.integers(0, 32, size=S // 32)
        rows = np.array(sorted(r for r in set(rows.tolist()) | {0, 255, 256, c - 1, c, S - 1} if r < S))
        o_ref, lse_ref = OA.attention_rows(q[:, :, hs], k[:, :, hs], v[:, :, hs], rows, bool(causal))
        worst[0] = max(worst[0], max_err(o[:, rows, hs], o_ref))
        worst[1] = max(worst[1], max_err(lse[:, hs][:, :, rows], lse_ref))
    log("  S=%d N=%d causal=%d D=%d: o %.3e lse %.3e" % (S, N, causal, D, worst[0], worst[1]))
    assert worst[0] <= TOL_O and worst[1] <= TOL_O


def test_bf16_one_host_share_long_block():
    """One host's share with 16384-key blocks (eight-wave kernel, side-stream copies into
    the receive slots): host 1 of 2, sampled rows of both heads."""
    B, H, D, N, host = 1, 2, 128, 2, 1
    S = 32768
    c = S // N
    q, k, v = synth.attention_inputs(14, B, S, H, D)
    qb = q[:, host * c:(host + 1) * c].contiguous()
    o = torch.empty(qb.shape, dtype=torch.bfloat16, device="cuda")
    lse = torch.empty((B, H, c), dtype=torch.float32, device="cuda")
    ra.ring_attn_fwd_host(dev(qb), *dev(k, v), o, lse, N, host, True)
    torch.cuda.synchronize()
    o, lse = o.cpu(), lse.cpu()
    rng = np.random.default_rng(400)
    rows = np.array(sorted(set((np.arange(0, c, 32) + rng.integers(0, 32, size=c // 32)).tolist()) | {0, c - 1}))
    worst = [0.0, 0.0]
    for h in range(H):
        hs = slice(h, h + 1)
        o_ref, lse_ref = OA.attention_rows(q[:, :, hs], k[:, :, hs], v[:, :, hs], rows + host * c, True)
        worst[0] = max(worst[0], max_err(o[:, rows, hs], o_ref))
        worst[1] = max(worst[1], max_err(lse[:, hs][:, :, rows], lse_ref))
    log("  host share c=%d: o %.3e lse %.3e" % (c, worst[0], worst[1]))
    assert worst[0] <= TOL_O and worst[1] <= TOL_O


@pytest.mark.parametrize("host", [0, 3, 7])
def test_bf16_one_host_share(host):
    B, H, D, N, c = 1, 2, 128, 8, 256
    S = N * c
    q, k, v = synth.attention_inputs(7, B, S, H, D)
    qb = q[:, host * c:(host + 1) * c].contiguous()
    o = torch.empty(qb.shape, dtype=torch.bfloat16, device="cuda")
    lse = torch.empty((B, H, c), dtype=torch.float32, device="cuda")
    ra.ring_attn_fwd_host(dev(qb), *dev(k, v), o, lse, N, host, True)
    torch.cuda.synchronize()
    o_ref, lse_ref = OR.ring_host_fwd(np64(qb), np64(k), np64(v), N, host, True)
    assert max_err(o, o_ref) <= TOL_O
    assert max_err(lse, lse_ref) <= TOL_O


@pytest.mark.parametrize("causal", [0, 1])
@pytest.mark.parametrize("env", ["RINGATTN_SERIAL_COPY", "RINGATTN_POISON"])
def test_bf16_copy_modes_match(env, causal, monkeypatch):
    """The key/value blocks reach every host's receive slot by side-stream copies (forward)
    or by the backward step kernels forwarding the block they hold to the next host.
    Receive slots poisoned with NaN before they are to be filled, or copies serialised on
    the caller stream (which also replaces the backward's forwarding by copies), give
    bit-identical forward and backward results to the default."""
    B, S, H, D, N = 1, 2048, 2, 128, 8
    q, k, v, do = dev(*synth.attention_inputs(8, B, S, H, D, with_grad=True))
    o0, l0 = ra.attention_fwd(q, k, v, N, causal)
    g0 = ra.attention_bwd(q, k, v, o0, l0, do, N, causal)
    monkeypatch.setenv(env, "1")
    o1, l1 = ra.attention_fwd(q, k, v, N, causal)
    g1 = ra.attention_bwd(q, k, v, o0, l0, do, N, causal)
    torch.cuda.synchronize()
    assert torch.equal(o0, o1) and torch.equal(l0, l1)
    for a, b in zip(g0, g1):
        assert torch.equal(a, b)
        assert not torch.isnan(a.float()).any()


@pytest.mark.parametrize("N", [1, 2, 8])
@pytest.mark.parametrize("causal", [0, 1])
def test_bf16_backward(N, causal):
    B, S, H, D = 1, 1024, 2, 128
    log("bwd case N=%d causal=%d" % (N, causal))
    q, k, v, do = synth.attention_inputs(9, B, S, H, D, with_grad=True)
    qd, kd, vd, dod = dev(q, k, v, do)
    o, lse = ra.attention_fwd(qd, kd, vd, N, causal)
    dq, dk, dv = ra.attention_bwd(qd, kd, vd, o, lse, dod, N, causal)
    torch.cuda.synchronize()
    ref = OA.attention_bwd(np64(q), np64(k), np64(v), np64(do), bool(causal))
    errs = [max_err(g, r) for g, r in zip((dq, dk, dv), ref)]
    log("  max|dq,dk,dv err| %s" % errs)
    assert max(errs) <= TOL_G


@pytest.mark.parametrize("S,N,D", [(1, 1, 128), (300, 8, 128), (1000, 3, 64), (1000, 3, 128),
                                   (2500, 4, 128), (1024, 4, 128)])
def test_bf16_varlen_causal_forward_backward(S, N, D):
    """Ragged causal lengths (ring_attn_*_varlen): the trailing host blocks are short or empty
    (S = 300 over 8 hosts of 128 leaves five hosts with padding only).  Forward and backward
    against the oracle on the real rows; when S already fills the blocks the call is the
    plain ring, bit for bit."""
    B, H = 2, 2
    log("varlen case S=%d N=%d D=%d" % (S, N, D))
    q, k, v, do = synth.attention_inputs(12, B, S, H, D, with_grad=True)
    qd, kd, vd, dod = dev(q, k, v, do)
    o = torch.empty_like(qd)
    lse = torch.empty((B, H, S), dtype=torch.float32, device="cuda")
    ra.ring_attn_fwd_varlen(qd, kd, vd, o, lse, N)
    dq, dk, dv = (torch.empty_like(qd) for _ in range(3))
    ra.ring_attn_bwd_varlen(qd, kd, vd, o, lse, dod, dq, dk, dv, N)
    torch.cuda.synchronize()
    o_ref, lse_ref = OA.attention_fwd(np64(q), np64(k), np64(v), True)
    ref = OA.attention_bwd(np64(q), np64(k), np64(v), np64(do), True)
    eo, el = max_err(o, o_ref), max_err(lse, lse_ref)
    eg = [max_err(g, r) for g, r in zip((dq, dk, dv), ref)]
    log("  max|o|,|lse| err %.3e %.3e  dq,dk,dv %s" % (eo, el, eg))
    assert eo <= TOL_O and el <= TOL_O
    assert max(eg) <= TOL_G
    # the high-level wrappers: for a ragged S the same entry points, else the plain ring,
    # which the padded path must then match bit for bit
    o2, lse2 = ra.attention_fwd(qd, kd, vd, N, True)
    g2 = ra.attention_bwd(qd, kd, vd, o2, lse2, dod, N, True)
    torch.cuda.synchronize()
    assert torch.equal(o, o2) and torch.equal(lse, lse2)
    assert all(torch.equal(a, b) for a, b in zip((dq, dk, dv), g2))


@pytest.mark.parametrize("D", [64, 128])
def test_bf16_backward_long_blocks(D):
    """Whole-ring backward over two hosts of 16384 keys (S = 32768, one head): dq, dk, dv
    compared in full; D = 64 runs the one-wave dK/dV kernel, D = 128 the split one."""
    B, S, H, N = 1, 32768, 1, 2
    log("bwd long-block case S=%d N=%d D=%d" % (S, N, D))
    q, k, v, do = synth.attention_inputs(15, B, S, H, D, with_grad=True)
    qd, kd, vd, dod = dev(q, k, v, do)
    o, lse = ra.attention_fwd(qd, kd, vd, N, True)
    dq, dk, dv = ra.attention_bwd(qd, kd, vd, o, lse, dod, N, True)
    torch.cuda.synchronize()
    ref = OA.attention_bwd(np64(q), np64(k), np64(v), np64(do), True)
    errs = [max_err(g, r) for g, r in zip((dq, dk, dv), ref)]
    log("  max|dq,dk,dv err| %s" % ["%.3e" % e for e in errs])
    assert max(errs) <= TOL_G


def test_bf16_backward_d64_batch2():
    B, S, H, D, N = 2, 512, 3, 64, 4
    q, k, v, do = synth.attention_inputs(10, B, S, H, D, with_grad=True)
    qd, kd, vd, dod = dev(q, k, v, do)
    o, lse = ra.attention_fwd(qd, kd, vd, N, True)
    grads = ra.attention_bwd(qd, kd, vd, o, lse, dod, N, True)
    torch.cuda.synchronize()
    ref = OA.attention_bwd(np64(q), np64(k), np64(v), np64(do), True)
    assert max(max_err(g, r) for g, r in zip(grads, ref)) <= TOL_G


def test_bf16_backward_gradient_invariants():
    """sum_s dK_s = 0 and sum_s dV_s = sum_r dO_r for every (batch, head)."""
    B, S, H, D, N = 1, 1024, 2, 128, 4
    q, k, v, do = dev(*synth.attention_inputs(11, B, S, H, D, with_grad=True))
    o, lse = ra.attention_fwd(q, k, v, N, True)
    dq, dk, dv = ra.attention_bwd(q, k, v, o, lse, do, N, True)
    torch.cuda.synchronize()
    assert np.max(np.abs(np64(dk).sum(axis=1))) <= TOL_G * 8
    assert np.max(np.abs(np64(dv).sum(axis=1) - np64(do).sum(axis=1))) <= TOL_G * 8
    # first causal token: dQ_0 = 0
    assert np.max(np.abs(np64(dq)[:, 0])) <= 1e-6


@pytest.mark.parametrize("N", [1, 4])
def test_fp32_backward(N):
    B, S, H, D = 1, 256, 2, 64
    q, k, v, do = synth.attention_inputs(12, B, S, H, D, torch.float32, with_grad=True)
    qd, kd, vd, dod = dev(q, k, v, do)
    o, lse = ra.attention_fwd(qd, kd, vd, N, True)
    grads = ra.attention_bwd(qd, kd, vd, o, lse, dod, N, True)
    torch.cuda.synchronize()
    ref = OA.attention_bwd(np64(q), np64(k), np64(v), np64(do), True)
    errs = [max_err(g, r) for g, r in zip(grads, ref)]
    log("  fp32 bwd errs %s" % errs)
    assert max(errs) <= TOL_F32


def test_errors_leave_outputs_untouched():
    q, k, v = dev(*synth.attention_inputs(13, 1, 512, 1, 128))
    o = torch.full_like(q, 7.0)
    lse = torch.full((1, 1, 512), 7.0, device="cuda")
    with pytest.raises(ra.RingAttnError) as e:
        ra.ring_attn_fwd(q, k, v, o, lse, 3, True)  # 512 % 3 != 0
    assert e.value.code == 2
    with pytest.raises(ra.RingAttnError) as e:
        ra.ring_attn_fwd(q, k, v, o, lse, 8, True)  # block 64 is not a multiple of 128
    assert e.value.code == 2
    torch.cuda.synchronize()
    assert bool((o == 7.0).all()) and bool((lse == 7.0).all())


@pytest.mark.parametrize("n_hosts", [8, 1])
def test_launch_timing_counts_and_bounds(n_hosts):
    """ring_attn_timing_*: one timed entry per ring step (consecutive steps share their
    boundary event), durations positive and together within the call's own duration."""
    log("timing case n_hosts=%d" % n_hosts)
    q, k, v = dev(*synth.attention_inputs(5, 1, 2048, 2, 128, torch.bfloat16))
    o, lse = ra.attention_fwd(q, k, v, n_hosts, True)  # warm-up
    dO = torch.ones_like(q)
    torch.cuda.synchronize()
    for kind in (ra.KERNEL_ATTN_FWD, ra.KERNEL_ATTN_BWD):
        ra.timing_read(kind)
    ra.timing_enable(True)
    try:
        e = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        e[0].record()
        o, lse = ra.attention_fwd(q, k, v, n_hosts, True)
        e[1].record()
        ra.attention_bwd(q, k, v, o, lse, dO, n_hosts, True)
        e[2].record()
        torch.cuda.synchronize()
    finally:
        ra.timing_enable(False)
    for kind, i in ((ra.KERNEL_ATTN_FWD, 0), (ra.KERNEL_ATTN_BWD, 1)):
        ms, n = ra.timing_read(kind)
        assert n == n_hosts
        assert 0 < ms <= e[i].elapsed_time(e[i + 1]) * 1.01 + 0.01
        assert ra.timing_read(kind) == (0.0, 0)


@pytest.mark.parametrize("D", [64, 128])
@pytest.mark.parametrize("amp", [4.0, 8.0])
def test_bf16_forward_large_logits(amp, D):
    """Queries scaled by 4 and 8 (exact in bf16): scores of standard deviation 4 and 8, the
    range of trained models' attention logits.  The products q.k are exact in float32 and
    the 1/sqrt(D) scale is applied in float32 (the paper's float32 logits), so the error
    stays at the bf16 rounding of P and o, independent of the logit scale."""
    B, S, H, N = 1, 1024, 2, 4
    q, k, v = synth.attention_inputs(12, B, S, H, D)
    q = q * amp
    o, lse = ra.attention_fwd(*dev(q, k, v), N, True)
    torch.cuda.synchronize()
    o_ref, lse_ref = OA.attention_fwd(np64(q), np64(k), np64(v), True)
    eo, el = max_err(o, o_ref), max_err(lse, lse_ref)
    log("  amp %.0f D %d: max|o err| %.3e  max|lse err| %.3e" % (amp, D, eo, el))
    assert eo <= TOL_O and el <= TOL_O


@pytest.mark.parametrize("D", [64, 128])
def test_bf16_backward_large_logits(D):
    """Backward with scores of standard deviation 4 (queries scaled by 4): the recomputed
    probabilities use float32 scores.  The gradients grow with the scale (|dK| up to ~14
    here), and bf16 storage alone -- o as the entry point receives it (it enters
    Delta = rowsum(dO * o)), P and dS as product operands, the outputs -- leaves a dK error
    above the plain 5e-2 bound: the CPU emulation of exactly that storage
    (tests/bf16_error_model.py attention_rounding_errors, checked on its own in
    tests/test_tolerance_model.py) gives the floor on these same inputs, and each gradient's
    magnitude-scaled error is bounded by max(5e-2, 1.25 x its floor), its relative RMS by
    1e-2."""
    from tests.test_tolerance_model import large_logit_floor
    B, S, H, N = 1, 1024, 2, 4
    q, k, v, do = synth.attention_inputs(13, B, S, H, D, with_grad=True)
    q = q * 4.0
    qd, kd, vd, dod = dev(q, k, v, do)
    o, lse = ra.attention_fwd(qd, kd, vd, N, True)
    dq, dk, dv = ra.attention_bwd(qd, kd, vd, o, lse, dod, N, True)
    torch.cuda.synchronize()
    floor = large_logit_floor(D)
    ref = OA.attention_bwd(np64(q), np64(k), np64(v), np64(do), True)
    for name, g, r in zip(("dq", "dk", "dv"), (dq, dk, dv), ref):
        e = np.abs(np64(g) - r)
        scaled = float((e / np.maximum(1.0, np.abs(r))).max())
        rms = float(np.sqrt((e ** 2).mean() / (r ** 2).mean()))
        bound = max(5e-2, 1.25 * floor[name][1])
        log("  %s: max|err| %.3e  scaled %.3e (floor %.3e, bound %.3e)  rel rms %.2e  max|ref| %.2f"
            % (name, e.max(), scaled, floor[name][1], bound, rms, np.abs(r).max()))
        assert scaled <= bound and rms <= 1e-2


def test_release_workspace_between_calls():
    """The library pool's cached workspace can be returned to the driver between calls; the
    next call allocates afresh and gives the same result."""
    q, k, v = dev(*synth.attention_inputs(14, 1, 1024, 2, 128))
    o1, l1 = ra.attention_fwd(q, k, v, 4, True)
    torch.cuda.synchronize()
    ra.release_workspace()
    o2, l2 = ra.attention_fwd(q, k, v, 4, True)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(l1, l2)
