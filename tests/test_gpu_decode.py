"""GPU parity of ring_attn_decode against the fp64 oracle (oracle/decode.py).

Seeded bf16 inputs (synth.attention_inputs with the queries as a short block and the
cache as the key/value length) go through the C ABI; o and lse are compared element by
element with the oracle on the same values.  Tolerance 2e-2 absolute on o and lse (the
bf16 attention bound).  Small cases span several chunks and tiles, every host count,
both head dims, 1..32 queries and the queries-equal-cache edge; the full-size cases
(cache of 262144 tokens over 8 hosts, 32 heads of 128) compare every output of sampled
heads.
"""
import numpy as np
import pytest
import torch

import paper_2310_01889_amd as ra
from paper_2310_01889_amd import synth
from oracle import attention as OA
from oracle import decode as OD
from tests.gpu_util import dev, log, max_err, np64

pytestmark = pytest.mark.gpu

TOL = 2e-2


def _case(seed, B, S, H, D, Tq, N, causal, amp=1.0):
    log("decode case seed=%d B=%d S=%d H=%d D=%d Tq=%d N=%d causal=%d amp=%g" % (seed, B, S, H, D, Tq, N, causal, amp))
    q, k, v = synth.attention_inputs(seed, B, Tq, H, D, kv_len=S)
    q = q * amp  # a power of two: exact in bf16
    o, lse = ra.attention_decode(*dev(q, k, v), N, causal)
    torch.cuda.synchronize()
    o_ref, lse_ref = OD.ring_decode_fwd(np64(q), np64(k), np64(v), N, bool(causal))
    eo, el = max_err(o, o_ref), max_err(lse, lse_ref)
    log("   max|o err| %.3e  max|lse err| %.3e" % (eo, el))
    return eo, el, (q, k, v, o, lse)


@pytest.mark.parametrize("D", [64, 128])
@pytest.mark.parametrize("Tq", [1, 5, 32])
@pytest.mark.parametrize("causal", [0, 1])
def test_decode_small(D, Tq, causal):
    eo, el, _ = _case(70 + Tq, 2, 2048, 3, D, Tq, 4, causal)
    assert eo <= TOL and el <= TOL


@pytest.mark.parametrize("N", [1, 2, 8, 64])
def test_decode_host_counts(N):
    eo, el, _ = _case(80 + N, 1, 2048, 2, 128, 7, N, 1)
    assert eo <= TOL and el <= TOL


def test_decode_single_tile_blocks_and_full_window():
    """Blocks of one 32-key tile, and Tq = S (every cache row is a query: full causal
    attention of 32 tokens, compared with the plain definition as well)."""
    eo, el, _ = _case(90, 1, 256, 2, 128, 3, 8, 1)
    assert eo <= TOL and el <= TOL
    eo, el, (q, k, v, o, lse) = _case(91, 1, 32, 2, 64, 32, 1, 1)
    assert eo <= TOL and el <= TOL
    o_ref, lse_ref = OA.attention_fwd(np64(q), np64(k), np64(v), True)
    assert max_err(o, o_ref) <= TOL and max_err(lse, lse_ref) <= TOL


def test_decode_first_row_exact():
    """Causal Tq = S = 32: query 0 sees only key 0, so o_0 = V_0 exactly (bf16 in, bf16 out)."""
    q, k, v = synth.attention_inputs(93, 1, 32, 1, 128, kv_len=32)
    o, _ = ra.attention_decode(*dev(q, k, v), 1, True)
    assert torch.equal(o[0, 0].cpu(), v[0, 0])


def test_decode_repeated_calls_agree():
    """The partial / merge launches are deterministic: two calls give identical bits."""
    q, k, v = dev(*synth.attention_inputs(94, 1, 4, 4, 128, kv_len=8192))
    o1, l1 = ra.attention_decode(q, k, v, 8, True)
    o2, l2 = ra.attention_decode(q, k, v, 8, True)
    assert torch.equal(o1, o2) and torch.equal(l1, l2)


@pytest.mark.parametrize("Tq", [1, 8])
def test_decode_full_size_sampled_heads(Tq):
    """Cache of 262144 tokens (8 hosts x 32768), 32 heads of 128: every output of heads
    0, 13 and 31 against the oracle (heads are independent)."""
    B, S, H, D, N = 1, 262144, 32, 128, 8
    log("decode full size Tq=%d" % Tq)
    q, k, v = synth.attention_inputs(95 + Tq, B, Tq, H, D, kv_len=S)
    o, lse = ra.attention_decode(*dev(q, k, v), N, True)
    torch.cuda.synchronize()
    for h in (0, 13, 31):
        sl = slice(h, h + 1)
        o_ref, lse_ref = OD.ring_decode_fwd(np64(q[:, :, sl]), np64(k[:, :, sl]), np64(v[:, :, sl]), N, True)
        eo, el = max_err(o[:, :, sl], o_ref), max_err(lse[:, sl], lse_ref)
        log("   head %d: max|o err| %.3e  max|lse err| %.3e" % (h, eo, el))
        assert eo <= TOL and el <= TOL


@pytest.mark.parametrize("amp", [4.0, 8.0])
def test_decode_large_logits(amp):
    """Scores of standard deviation 4 and 8: the products are exact in float32 and the scale
    is applied in float32, so the error does not grow with the logit scale."""
    eo, el, _ = _case(90, 1, 4096, 2, 128, 8, 4, 1, amp)
    assert eo <= TOL and el <= TOL
