"""The reading behind the ragged-length causal entry points, checked on the oracle alone:
a causal sequence padded at its end with zero rows (q = k = v = dO = 0) gives, on its real
rows, the same o, lse, dQ, dK and dV as the unpadded sequence, because no real query sees
a padded key and a padded query row has dO = 0, hence dP = 0 and dS = 0.  The same check
without the causal mask must fail (padded keys then enter every real row's softmax)."""
import numpy as np
import pytest

from oracle import attention as OA


def _pad(x, Sp):
    out = np.zeros((x.shape[0], Sp) + x.shape[2:], dtype=x.dtype)
    out[:, : x.shape[1]] = x
    return out


@pytest.mark.parametrize("S,Sp", [(1, 4), (5, 8), (13, 32)])
def test_causal_zero_padding_leaves_real_rows_unchanged(S, Sp):
    rng = np.random.default_rng(S)
    B, H, D = 2, 2, 8
    q, k, v, do = (rng.standard_normal((B, S, H, D)) for _ in range(4))
    o, lse = OA.attention_fwd(q, k, v, True)
    op, lsep = OA.attention_fwd(_pad(q, Sp), _pad(k, Sp), _pad(v, Sp), True)
    np.testing.assert_allclose(op[:, :S], o, rtol=0, atol=1e-13)
    np.testing.assert_allclose(lsep[:, :, :S], lse, rtol=0, atol=1e-13)
    g = OA.attention_bwd(q, k, v, do, True)
    gp = OA.attention_bwd(_pad(q, Sp), _pad(k, Sp), _pad(v, Sp), _pad(do, Sp), True)
    for a, b in zip(gp, g):
        np.testing.assert_allclose(a[:, :S], b, rtol=0, atol=1e-12)
    # padded keys get no value gradient: every query that sees them has dO = 0
    assert np.all(gp[2][:, S:] == 0)


def test_non_causal_zero_padding_changes_real_rows():
    rng = np.random.default_rng(7)
    q, k, v = (rng.standard_normal((1, 5, 1, 8)) for _ in range(3))
    o, _ = OA.attention_fwd(q, k, v, False)
    op, _ = OA.attention_fwd(_pad(q, 8), _pad(k, 8), _pad(v, 8), False)
    assert np.max(np.abs(op[:, :5] - o)) > 1e-3
