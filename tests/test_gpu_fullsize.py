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


def _sample_rows(n, c, extra):
    rng = np.random.default_rng(n)
    rows = set(extra) | set(rng.integers(0, c, size=n).tolist())
    return np.array(sorted(rows))


def _tile_rows(n_rows, tile, seed, extra=()):
    """One row per tile of ``tile`` rows (a random offset in each), plus ``extra`` rows."""
    rng = np.random.default_rng(seed)
    rows = np.arange(0, n_rows, tile) + rng.integers(0, tile, size=n_rows // tile)
    return np.array(sorted(set(rows.tolist()) | set(extra)))


def test_causal_forward_S32768_H32_hosts8():
    """The forward's work items are (host, head, 128-row query tile): one sampled row of every
    query tile of every head is compared (8192 rows), plus the block edges."""
    B, S, H, D, N = 1, 32768, 32, 128, 8
    q, k, v = synth.attention_inputs(2, B, S, H, D)
    o, lse = ra.attention_fwd(*dev(q, k, v), N, True)
    torch.cuda.synchronize()
    o, lse = o.cpu(), lse.cpu()
    c = S // N
    worst = [0.0, 0.0]
    for h in range(H):
        rows = _tile_rows(S, 128, 200 + h, [0, 1, c - 1, c, 3 * c + 17, S - c, S - 1])
        hs = slice(h, h + 1)
        o_ref, lse_ref = OA.attention_rows(q[:, :, hs], k[:, :, hs], v[:, :, hs], rows, True)
        worst[0] = max(worst[0], max_err(o[:, rows, hs], o_ref))
        worst[1] = max(worst[1], max_err(lse[:, hs][:, :, rows], lse_ref))
    log("   C2, one row per query tile of every head: o %.3e lse %.3e" % tuple(worst))
    assert worst[0] <= TOL_O and worst[1] <= TOL_O


def test_causal_backward_S65536_H2_hosts8_c8192():
    """The attention of the Algorithm 1 layer at its ring shape (S = 65536 in 8 blocks of
    8192), forward and backward through ring_attn_fwd / ring_attn_bwd: head 0 compared in
    full (o, lse, dq, dk, dv), head 1 on one sampled query row per tile (o, lse, dq)."""
    B, S, H, D, N = 1, 65536, 2, 128, 8
    q, k, v, do = synth.attention_inputs(44, B, S, H, D, with_grad=True)
    qd, kd, vd, dod = dev(q, k, v, do)
    o, lse = ra.attention_fwd(qd, kd, vd, N, True)
    dq, dk, dv = ra.attention_bwd(qd, kd, vd, o, lse, dod, N, True)
    torch.cuda.synchronize()
    o, lse, dq, dk, dv = (t.cpu() for t in (o, lse, dq, dk, dv))
    del qd, kd, vd, dod
    h0 = slice(0, 1)
    o_ref, lse_ref = OA.attention_fwd(q[:, :, h0], k[:, :, h0], v[:, :, h0], True)
    eo, el = max_err(o[:, :, h0], o_ref), max_err(lse[:, h0], lse_ref)
    log("   head 0 forward: o %.3e lse %.3e" % (eo, el))
    g_ref = OA.attention_bwd(q[:, :, h0], k[:, :, h0], v[:, :, h0], do[:, :, h0], True)
    eg = [max_err(t[:, :, h0], r) for t, r in zip((dq, dk, dv), g_ref)]
    log("   head 0 backward: dq %.3e dk %.3e dv %.3e" % tuple(eg))
    assert eo <= TOL_O and el <= TOL_O and max(eg) <= TOL_G
    h1 = slice(1, 2)
    rows = _tile_rows(S, 128, 45, [0, S // N - 1, S // N, S - 1])
    o_ref, lse_ref = OA.attention_rows(q[:, :, h1], k[:, :, h1], v[:, :, h1], rows, True)
    dq_ref = OA.attention_bwd_rows(q[:, :, h1], k[:, :, h1], v[:, :, h1], do[:, :, h1], rows, True)
    e1 = (max_err(o[:, rows, h1], o_ref), max_err(lse[:, h1][:, :, rows], lse_ref), max_err(dq[:, rows, h1], dq_ref))
    log("   head 1 sampled rows: o %.3e lse %.3e dq %.3e" % e1)
    assert e1[0] <= TOL_O and e1[1] <= TOL_O and e1[2] <= TOL_G


def _host_inputs(seed, B, c, H, D, N, host):
    q, k, v, do = synth.attention_inputs(seed, B, c, H, D, with_grad=True, kv_len=N * c)
    return q, k, v, do


@pytest.fixture(scope="module")
def host7():
    """Host 7 of 8: a 32768-token query block against 262144 keys, forward, then the
    backward with dK/dV travelling through the double buffer (accumulators start at zero,
    so they hold this host's contributions).  Results are copied to the host; dK/dV of
    head 0 only, plus their sums over the keys for every head."""
    B, c, H, D, N, host = 1, 32768, 32, 128, 8, 7
    S = N * c
    log("host-share case: B=%d c=%d H=%d D=%d n_hosts=%d host=%d" % (B, c, H, D, N, host))
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
    out = dict(q=q, k=k, v=v, do=do, o=o.cpu(), lse=lse.cpu(), dq=dq.cpu(),
               dk0=dk_acc[:, :, 0:1].cpu(), dv0=dv_acc[:, :, 0:1].cpu(),
               sk=dk_acc.sum(dim=1).double().cpu().numpy(), sv=dv_acc.sum(dim=1).double().cpu().numpy(),
               c=c, H=H, N=N, host=host)
    del qd, kd, vd, dod, dk_acc, dv_acc
    torch.cuda.empty_cache()
    return out


def test_host_share_forward_rows_c32768_hosts8(host7):
    """One sampled query row of each of the 256 query tiles, in every head, plus rows 0 and
    c - 1: o and lse against the oracle on those rows (global positions 7c + r)."""
    t = host7
    c, off = t["c"], t["host"] * t["c"]
    worst = [0.0, 0.0, 0.0]
    for h in range(t["H"]):
        rows = _tile_rows(c, 128, 300 + h, [0, 1, c - 1])
        hs = slice(h, h + 1)
        o_ref, lse_ref = OA.attention_rows(t["q"][:, :, hs], t["k"][:, :, hs], t["v"][:, :, hs], rows, True,
                                           q_offset=off)
        eo = max_err(t["o"][:, rows, hs], o_ref)
        worst[0] = max(worst[0], eo)
        worst[1] = max(worst[1], max_err(t["lse"][:, hs][:, :, rows], lse_ref))
        worst[2] = max(worst[2], eo / np.abs(o_ref).max())
    log("   host 7, one row per query tile of every head: o %.3e (%.3e of max |o|) lse %.3e"
        % (worst[0], worst[2], worst[1]))
    # rows averaging ~245K values are small (|o| ~ 1e-2): the error is bounded relative to
    # their magnitude as well, at the tolerance of the plain bound
    assert worst[0] <= TOL_O and worst[1] <= TOL_O and worst[2] <= TOL_O


def test_host_share_dq_rows_c32768_hosts8(host7):
    """dq on one sampled query row of each query tile, in every head, plus rows 0, c - 1."""
    t = host7
    c, off = t["c"], t["host"] * t["c"]
    worst, rel = 0.0, 0.0
    for h in range(t["H"]):
        rows = _tile_rows(c, 128, 400 + h, [0, 1, c - 1])
        hs = slice(h, h + 1)
        dq_ref = OA.attention_bwd_rows(t["q"][:, :, hs], t["k"][:, :, hs], t["v"][:, :, hs], t["do"][:, :, hs],
                                       rows, True, q_offset=off)
        e = max_err(t["dq"][:, rows, hs], dq_ref)
        worst, rel = max(worst, e), max(rel, e / np.abs(dq_ref).max())
    log("   host 7, one dq row per query tile of every head: %.3e (%.3e of max |dq|)" % (worst, rel))
    assert worst <= TOL_G and rel <= TOL_G


def test_host_share_dkdv_key_rows_c32768_hosts8(host7):
    """This host's contributions to dK and dV, element by element, on 32 sampled key rows of
    each of the 8 blocks (edges included) of head 0: the oracle evaluates the host's 32768
    query rows in full to get every row's probabilities and Delta."""
    t = host7
    c, N, off = t["c"], t["N"], t["host"] * t["c"]
    rng = np.random.default_rng(7)
    rows = sorted(set(j * c + r for j in range(N)
                      for r in [0, 1, c // 2, c - 1] + rng.integers(0, c, size=28).tolist()))
    rows = np.array(rows)
    h0 = slice(0, 1)
    # the contributions are sums over query rows: evaluated in slices of 4096 query rows
    dk_ref, dv_ref = 0.0, 0.0
    for r0 in range(0, c, 4096):
        qs = slice(r0, r0 + 4096)
        dk_s, dv_s = OA.attention_bwd_key_rows(t["q"][:, qs, h0], t["k"][:, :, h0], t["v"][:, :, h0],
                                               t["do"][:, qs, h0], rows, True, q_offset=off + r0)
        dk_ref, dv_ref = dk_ref + dk_s, dv_ref + dv_s
        log("     query rows %d..%d done" % (r0, r0 + 4095))
    ek, ev = max_err(t["dk0"][:, rows], dk_ref), max_err(t["dv0"][:, rows], dv_ref)
    rk, rv = ek / np.abs(dk_ref).max(), ev / np.abs(dv_ref).max()
    log("   host 7, %d key rows of head 0: dk %.3e dv %.3e (%.3e / %.3e of max |ref|)" % (len(rows), ek, ev, rk, rv))
    # one host's contributions are small (|dK|, |dV| ~ 1e-2 here): bounded relative to their
    # magnitude as well, at the tolerance of the plain gradient bound
    assert ek <= TOL_G and ev <= TOL_G and rk <= TOL_G and rv <= TOL_G


def test_host_share_gradient_sums_c32768_hosts8(host7):
    """The contributions of one host's queries to dK sum to zero over the keys and those to
    dV sum to the host's upstream gradient (rows of dS sum to zero; rows of P to one), in
    every head."""
    t = host7
    ref_sv = np64(t["do"]).sum(axis=1)
    ek, ev = np.abs(t["sk"]).max(), np.abs(t["sv"] - ref_sv).max()
    log("   sum dK %.3e  sum dV - sum dO %.3e (scale %.1f)" % (ek, ev, np.abs(ref_sv).max()))
    assert ek <= 1.0 and ev <= 1.0


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
