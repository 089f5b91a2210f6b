"""ring_attn_decode_noalloc (decode without any allocation, partial states in the library's
fixed device scratch) against ring_attn_decode through the C ABI: two calls in a row, the
second smaller, each bit-identical to the allocating entry point (same kernels, same chunking)
and within the decode tolerance of the fp64 oracle on sampled heads."""
import numpy as np
import pytest
import torch

import paper_2310_01889_amd as ra
from paper_2310_01889_amd import synth
from oracle import decode as OD
from tests.gpu_util import dev, log, max_err, np64

pytestmark = pytest.mark.gpu


def _decode(fn, q, kc, vc, n_hosts, causal):
    B, Tq, H, D = q.shape
    o = torch.full_like(q, 7.0)
    lse = torch.full((B, H, Tq), 7.0, dtype=torch.float32, device=q.device)
    fn(q, kc, vc, o, lse, n_hosts, causal)
    return o, lse


@pytest.mark.parametrize("order", ["noalloc_first", "alloc_first"])
def test_decode_noalloc_matches_decode(order):
    cases = [  # (seed, B, Tq, H, D, S, n_hosts, causal): the second call is smaller
        (81, 1, 12, 32, 128, 65536, 8, True),
        (82, 1, 3, 2, 64, 4096, 4, False),
    ]
    for seed, B, Tq, H, D, S, N, causal in cases:
        log("decode noalloc case: seed=%d B=%d Tq=%d H=%d D=%d S=%d n_hosts=%d causal=%d (%s)"
            % (seed, B, Tq, H, D, S, N, causal, order))
        q, kc, vc = synth.attention_inputs(seed, B, Tq, H, D, kv_len=S)
        qd, kd, vd = dev(q, kc, vc)
        if order == "noalloc_first":
            o1, l1 = _decode(ra.ring_attn_decode_noalloc, qd, kd, vd, N, causal)
            o0, l0 = _decode(ra.ring_attn_decode, qd, kd, vd, N, causal)
        else:
            o0, l0 = _decode(ra.ring_attn_decode, qd, kd, vd, N, causal)
            o1, l1 = _decode(ra.ring_attn_decode_noalloc, qd, kd, vd, N, causal)
        torch.cuda.synchronize()
        assert torch.equal(o1, o0) and torch.equal(l1, l0)
        for h in (0, H - 1):
            hs = slice(h, h + 1)
            o_ref, l_ref = OD.ring_decode_fwd(np64(q[:, :, hs]), np64(kc[:, :, hs]), np64(vc[:, :, hs]), N, causal)
            eo, el = max_err(o1[:, :, hs], o_ref), max_err(l1[:, hs], l_ref)
            log("   head %d: o %.3e lse %.3e" % (h, eo, el))
            assert eo <= 2e-2 and el <= 2e-2
        del qd, kd, vd


def test_decode_noalloc_rejects_more_than_the_scratch():
    """Tq = 32 over a 262144-token cache of 32 heads needs 17 M floats of partial state."""
    B, Tq, H, D, S = 1, 32, 32, 128, 262144
    q = torch.zeros((B, Tq, H, D), dtype=torch.bfloat16, device="cuda")
    kc = torch.zeros((B, S, H, D), dtype=torch.bfloat16, device="cuda")
    o = torch.full_like(q, 7.0)
    lse = torch.full((B, H, Tq), 7.0, dtype=torch.float32, device="cuda")
    with pytest.raises(ra.RingAttnError) as e:
        ra.ring_attn_decode_noalloc(q, kc, kc, o, lse, 8, True)
    assert e.value.code == 2 and "scratch" in str(e.value)
    torch.cuda.synchronize()
    assert bool((o == 7.0).all()) and bool((lse == 7.0).all())
