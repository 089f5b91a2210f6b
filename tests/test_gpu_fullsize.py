"""GPU parity at the full sizes of the benchmark workloads, in the launch configuration
bench.py times, on outputs the fp64 oracle can compute one by one (each query row of a
causal attention depends only on its own query row, its upstream gradient and the keys
and values), or on whole heads (heads are independent), plus invariants that hold at any
size.  Tolerances as in test_gpu_attention.py."""
import numpy as np
import pytest
import torch

import paper_2310_01889_amd as ra
from paper_2310_01889_amd import synth
from oracle import attention as OA
from tests.gpu_util import dev, log, max_err, np64

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

TOL_O, TOL_G = 2e-2, 5e-2


def f32(t):
    """float32 NumPy view of a bf16 tensor (exact); the oracle upcasts one head at a time."""
    return t.float().numpy()


def _sample_rows(n, c, extra):
    rng = np.random.default_rng(n)
    rows = set(extra) | set(rng.integers(0, c, size=n).tolist())
    return np.array(sorted(rows))


def test_causal_forward_S32768_H32_hosts8():
    B, S, H, D, N = 1, 32768, 32, 128, 8
    q, k, v = synth.attention_inputs(2, B, S, H, D)
    o, lse = ra.attention_fwd(*dev(q, k, v), N, True)
    torch.cuda.synchronize()
    c = S // N
    rows = _sample_rows(48, S, [0, 1, c - 1, c, 3 * c + 17, S - c, S - 1])
    o_ref, lse_ref = OA.attention_rows(f32(q), f32(k), f32(v), rows, True)
    idx = torch.from_numpy(rows).cuda()
    eo, el = max_err(o[:, idx], o_ref), max_err(lse[:, :, idx], lse_ref)
    log("   C2 sampled rows: o %.3e lse %.3e" % (eo, el))
    assert eo <= TOL_O and el <= TOL_O


def _host_inputs(seed, B, c, H, D, N, host):
    q, k, v, do = synth.attention_inputs(seed, B, c, H, D, with_grad=True, kv_len=N * c)
    return q, k, v, do


def test_one_host_share_forward_backward_c32768_hosts8():
    """Host 7 of 8: a 32768-token query block against 262144 keys, forward, then the
    backward with dK/dV travelling through the double buffer."""
    B, c, H, D, N, host = 1, 32768, 32, 128, 8, 7
    S = N * c
    q, k, v, do = _host_inputs(5, B, c, H, D, N, host)
    qd, kd, vd, dod = dev(q, k, v, do)
    o = torch.empty_like(qd)
    lse = torch.empty((B, H, c), dtype=torch.float32, device="cuda")
    ra.ring_attn_fwd_host(qd, kd, vd, o, lse, N, host, True)
    dq = torch.empty_like(qd)
    dk_acc = torch.zeros((B, S, H, D), dtype=torch.float32, device="cuda")
    dv_acc = torch.zeros_like(dk_acc)
    ra.ring_attn_bwd_host(qd, kd, vd, o, lse, dod, dq, dk_acc, dv_acc, N, host, True)
    torch.cuda.synchronize()
    rows = _sample_rows(24, c, [0, 1, 4095, c - 1])
    idx = torch.from_numpy(rows).cuda()
    qf, kf, vf, dof = f32(q), f32(k), f32(v), f32(do)
    o_ref, lse_ref = OA.attention_rows(qf, kf, vf, rows, True, q_offset=host * c)
    eo, el = max_err(o[:, idx], o_ref), max_err(lse[:, :, idx], lse_ref)
    dq_ref = OA.attention_bwd_rows(qf, kf, vf, dof, rows, True, q_offset=host * c)
    eq = max_err(dq[:, idx], dq_ref)
    log("   host 7 sampled rows: o %.3e lse %.3e dq %.3e" % (eo, el, eq))
    assert eo <= TOL_O and el <= TOL_O and eq <= TOL_G
    # the contributions of one host's queries to dK sum to zero over the keys and those
    # to dV sum to the host's upstream gradient (rows of dS sum to zero; rows of P to one)
    sk = dk_acc.sum(dim=1).double().cpu().numpy()
    sv = dv_acc.sum(dim=1).double().cpu().numpy()
    ref_sv = np64(do).sum(axis=1)
    log("   sum dK %.3e  sum dV - sum dO %.3e (scale %.1f)" % (np.abs(sk).max(), np.abs(sv - ref_sv).max(),
                                                            np.abs(ref_sv).max()))
    assert np.abs(sk).max() <= 1.0 and np.abs(sv - ref_sv).max() <= 1.0


@pytest.mark.parametrize("host", [0, 3, 7])
def test_one_host_share_backward_small(host):
    """The same path at c = 256 in full: dq and this host's dK/dV contributions, added on
    top of nonzero carried gradients."""
    B, c, H, D, N = 1, 256, 2, 128, 8
    S = N * c
    q, k, v, do = _host_inputs(70 + host, B, c, H, D, N, host)
    qd, kd, vd, dod = dev(q, k, v, do)
    o = torch.empty_like(qd)
    lse = torch.empty((B, H, c), dtype=torch.float32, device="cuda")
    ra.ring_attn_fwd_host(qd, kd, vd, o, lse, N, host, True)
    g = torch.Generator().manual_seed(host)
    carried_k = torch.randn((B, S, H, D), generator=g)
    carried_v = torch.randn((B, S, H, D), generator=g)
    dk_acc, dv_acc = dev(carried_k.clone(), carried_v.clone())
    dq = torch.empty_like(qd)
    ra.ring_attn_bwd_host(qd, kd, vd, o, lse, dod, dq, dk_acc, dv_acc, N, host, True)
    torch.cuda.synchronize()
    dq_ref, dk_ref, dv_ref = OA.attention_bwd(np64(q), np64(k), np64(v), np64(do), True, q_offset=host * c)
    e = (max_err(dq, dq_ref), max_err(dk_acc.cpu() - carried_k, dk_ref), max_err(dv_acc.cpu() - carried_v, dv_ref))
    log("   host %d: dq %.3e dk %.3e dv %.3e" % ((host,) + e))
    assert max(e) <= TOL_G


def test_causal_forward_backward_S16384_H16_hosts8():
    """Full forward and backward; the oracle runs on heads 0 and 15 (heads are independent)."""
    B, S, H, D, N = 1, 16384, 16, 128, 8
    q, k, v, do = synth.attention_inputs(3, B, S, H, D, with_grad=True)
    qd, kd, vd, dod = dev(q, k, v, do)
    o, lse = ra.attention_fwd(qd, kd, vd, N, True)
    dq, dk, dv = ra.attention_bwd(qd, kd, vd, o, lse, dod, N, True)
    torch.cuda.synchronize()
    for h in (0, 15):
        sl = lambda t: np64(t[:, :, h:h + 1])
        o_ref, lse_ref = OA.attention_fwd(sl(q), sl(k), sl(v), True)
        g_ref = OA.attention_bwd(sl(q), sl(k), sl(v), sl(do), True)
        eo, el = max_err(o[:, :, h:h + 1], o_ref), max_err(lse[:, h:h + 1], lse_ref)
        eg = [max_err(t[:, :, h:h + 1], r) for t, r in zip((dq, dk, dv), g_ref)]
        log("   head %d: o %.3e lse %.3e dq/dk/dv %s" % (h, eo, el, ["%.3e" % x for x in eg]))
        assert eo <= TOL_O and el <= TOL_O and max(eg) <= TOL_G


def test_blockwise_ffn_full_size_sampled():
    """Blockwise FFN at the benchmarked size (T = 65536 in 8 blocks of 8192, d_model 4096,
    d_ff 16384, GeLU, no bias), forward and backward.  The FFN acts row by row, so rows of
    y and dx come from the oracle on those rows alone; a column j of dW1 (and row j of dW2,
    entry j of db1) depends only on column j of W1 and row j of W2, so the oracle on a
    narrow FFN made of sampled hidden units gives them exactly.  Tolerances as in
    test_gpu_ffn.py: |err| <= 2e-2 (y) / 5e-2 (dx) times max(1, |ref|); weight gradients
    max |err| <= 5e-2 * max(1, rms(ref))."""
    from oracle import ffn as OF
    T, dm, dff, blk, act = 65536, 4096, 16384, 8192, ra.ACT_GELU_ERF
    x, w1, _, w2, _, dy = synth.ffn_inputs(61, T, dm, dff, with_grad=True)
    xd, w1d, w2d, dyd = dev(x, w1, w2, dy)
    y = torch.empty((T, dm), dtype=torch.bfloat16, device="cuda")
    ra.blockwise_ffn(xd, w1d, None, w2d, None, y, blk, act)
    dx = torch.empty_like(xd)
    dw1 = torch.empty((dm, dff), dtype=torch.float32, device="cuda")
    db1 = torch.empty((dff,), dtype=torch.float32, device="cuda")
    dw2 = torch.empty((dff, dm), dtype=torch.float32, device="cuda")
    db2 = torch.empty((dm,), dtype=torch.float32, device="cuda")
    ra.blockwise_ffn_bwd(xd, w1d, None, w2d, dyd, dx, dw1, db1, dw2, db2, blk, act)
    torch.cuda.synchronize()

    rows = _sample_rows(12, T, [0, blk - 1, blk, T - 1])
    log("ffn full size: rows %s" % rows.tolist())
    y_ref = OF.ffn_fwd(np64(x[rows]), np64(w1), None, np64(w2), None, act)
    dx_ref = OF.ffn_bwd(np64(x[rows]), np64(w1), None, np64(w2), np64(dy[rows]), act)[0]
    ey = np.abs(np64(y[rows].cpu()) - y_ref) / np.maximum(1.0, np.abs(y_ref))
    ex = np.abs(np64(dx[rows].cpu()) - dx_ref) / np.maximum(1.0, np.abs(dx_ref))
    log("  y scaled err %.3e  dx scaled err %.3e" % (ey.max(), ex.max()))
    assert ey.max() <= 2e-2 and ex.max() <= 5e-2

    cols = np.array(sorted(set([0, dff - 1]) | set(np.random.default_rng(5).integers(0, dff, 4).tolist())))
    _, rdw1, rdb1, rdw2, rdb2 = OF.ffn_bwd(np64(x), np64(w1[:, cols]), None, np64(w2[cols, :]), np64(dy), act)
    for name, got, ref in (("dW1 cols", dw1[:, cols], rdw1), ("db1", db1[cols], rdb1), ("dW2 rows", dw2[cols, :], rdw2)):
        g, r = np64(got.cpu()), np.asarray(ref)
        bound = 5e-2 * max(1.0, float(np.sqrt(np.mean(r * r))))
        log("  %s: max|err| %.3e bound %.3e" % (name, np.abs(g - r).max(), bound))
        assert np.abs(g - r).max() <= bound
    # db2 = column sums of dy (no hidden unit involved)
    e2 = np.abs(np64(db2.cpu()) - rdb2).max()
    log("  db2: max|err| %.3e" % e2)
    assert e2 <= 5e-2 * max(1.0, float(np.sqrt(np.mean(rdb2 * rdb2))))
