"""Planted mistakes in the oracle must be caught by its pins (CPU only).

Each case patches one plausible slip into a copy of an oracle function (a dropped
scale, an off-by-one mask, a missing rescale, a wrong sign, a dropped derivative
term, a transposed operand) and re-runs the pin that should catch it.
"""
import numpy as np
import pytest

from oracle import attention as A
from oracle import ffn as F
from oracle import ring as R
import tests.test_oracle_attention as TA
import tests.test_oracle_ffn as TF
import tests.test_oracle_ring as TR


def _fails(check, *args):
    with pytest.raises(AssertionError):
        check(*args)


def test_dropped_scale_is_caught(monkeypatch):
    orig = A._masked_scores
    monkeypatch.setattr(A, "_masked_scores", lambda qh, kh, scale, c, p, r: orig(qh, kh, 1.0, c, p, r))
    _fails(TA.test_naive_matches_brute_force, 5, 3, True)
    _fails(TA.test_naive_matches_torch_sdpa_fp64, True)


def test_off_by_one_causal_mask_is_caught(monkeypatch):
    import torch

    def masked(qh, kh, scale, causal, q_pos0, r0):
        s = (qh @ kh.T) * scale
        qpos = q_pos0 + r0 + torch.arange(qh.shape[0])[:, None]
        kpos = torch.arange(kh.shape[0])[None, :]
        return s.masked_fill(kpos > qpos + 1, float("-inf")) if causal else s
    monkeypatch.setattr(A, "_masked_scores", masked)
    _fails(TA.test_first_causal_token)
    _fails(TA.test_zero_query_gives_prefix_mean)


def test_missing_numerator_rescale_is_caught(monkeypatch):
    import torch

    def fold(state, q, kb, vb, qp, kp, causal, scale, qc, kc):
        # fold every tile with the max of its own tile only: correction dropped
        mx, num, den = state
        for q0 in range(0, q.shape[1], qc):
            q1 = min(q.shape[1], q0 + qc)
            for k0 in range(0, kb.shape[1], kc):
                k1 = min(kb.shape[1], k0 + kc)
                vis = R._visible(qp + torch.arange(q0, q1), kp + torch.arange(k0, k1), causal)
                if not bool(vis.any()):
                    continue
                s = R._scores(q[:, q0:q1], kb[:, k0:k1], scale).masked_fill(~vis[None, None], float("-inf"))
                m_new = torch.maximum(mx[:, :, q0:q1], s.amax(dim=3))
                p = torch.exp(s - m_new[..., None])
                den[:, :, q0:q1] = den[:, :, q0:q1] + p.sum(dim=3)
                num[:, q0:q1] = num[:, q0:q1] + torch.einsum("bhqk,bkhd->bqhd", p, vb[:, k0:k1])
                mx[:, :, q0:q1] = m_new
    monkeypatch.setattr(R, "_fold_block_fwd", fold)
    _fails(TR.test_ring_forward_equals_naive, 4, True)


def test_wrong_sign_in_softmax_gradient_is_caught(monkeypatch):
    def bwd(q, k, v, do, causal, scale=None, q_offset=0, row_chunk=1024):
        dq, dk, dv = orig(q, k, v, do, causal, scale, q_offset, row_chunk)
        return -dq, -dk, dv
    orig = A.attention_bwd
    monkeypatch.setattr(A, "attention_bwd", bwd)
    _fails(TA.test_backward_finite_differences, True)


def test_dropped_gelu_derivative_term_is_caught(monkeypatch):
    orig = F.act_grad
    monkeypatch.setattr(F, "act_grad", lambda h, act: 0.5 * (1 + np.tanh(h)) if act == F.GELU_ERF else orig(h, act))
    _fails(TF.test_ffn_backward_finite_differences)


def test_transposed_weight_gradient_is_caught(monkeypatch):
    orig = F.linear_bwd
    monkeypatch.setattr(F, "linear_bwd", lambda x, w, dy: (orig(x, w, dy)[0], (np.asarray(dy).T @ np.asarray(x)).T[::-1]))
    _fails(TF.test_linear_forward_backward)


def _mutated_decode(old, new):
    """A copy of oracle.decode.ring_decode_fwd with one source fragment replaced."""
    import inspect
    from oracle import decode as D
    src = inspect.getsource(D.ring_decode_fwd)
    assert old in src
    ns = dict(vars(D))
    exec(src.replace(old, new), ns)
    return ns["ring_decode_fwd"]


def test_decode_queries_at_the_start_are_caught(monkeypatch):
    from oracle import decode as D
    import tests.test_oracle_decode as TD
    monkeypatch.setattr(D, "ring_decode_fwd", _mutated_decode("np.arange(S - Tq, S)", "np.arange(0, Tq)"))
    _fails(TD.test_single_query_sees_its_own_key_last)
    _fails(TD.test_zero_query_gives_visible_mean)


def test_decode_missing_rescale_is_caught(monkeypatch):
    from oracle import decode as D
    import tests.test_oracle_decode as TD
    monkeypatch.setattr(D, "ring_decode_fwd", _mutated_decode("num = num * corr[..., None] +", "num = num +"))
    _fails(TD.test_matches_torch_sdpa_fp64, 64, 4, 5, True)


def _mutated(module, fname, old, new):
    """A copy of module.fname with one source fragment replaced."""
    import inspect
    src = inspect.getsource(getattr(module, fname))
    assert old in src
    ns = dict(vars(module))
    exec(src.replace(old, new), ns)
    return ns[fname]


def test_llama_rope_half_split_pairing_is_caught(monkeypatch):
    from oracle import llama as LL
    import tests.test_oracle_llama as TL
    bad = _mutated(LL, "rope", "x0, x1 = x[..., 0::2], x[..., 1::2]", "x0, x1 = x[..., :D // 2], x[..., D // 2:]")
    monkeypatch.setattr(LL, "rope", bad)
    _fails(TL.test_rope_is_complex_rotation)


def test_llama_rmsnorm_dropped_term_is_caught(monkeypatch):
    from oracle import llama as LL
    import tests.test_oracle_llama as TL
    monkeypatch.setattr(LL, "rmsnorm_bwd", _mutated(LL, "rmsnorm_bwd", "gdy * rstd[:, None] - x *", "gdy * rstd[:, None] - 0 * x *"))
    _fails(TL.test_rmsnorm_matches_torch_and_autograd)


def test_llama_swiglu_wrong_derivative_is_caught(monkeypatch):
    from oracle import llama as LL
    import tests.test_oracle_llama as TL
    monkeypatch.setattr(LL, "swiglu_bwd", _mutated(LL, "swiglu_bwd", "w * silu_grad(u)", "w * silu(u)"))
    _fails(TL.test_swiglu_backward_matches_autograd)


def test_key_rows_dropped_delta_is_caught(monkeypatch):
    monkeypatch.setattr(A, "attention_bwd_key_rows",
                        _mutated(A, "attention_bwd_key_rows", "(doh @ vs.T - delta[:, None])", "(doh @ vs.T)"))
    _fails(TA.test_key_row_gradients_match_torch_autograd, True, 24, 7)


def test_causal_key_limit_one_short_is_caught(monkeypatch):
    monkeypatch.setattr(A, "_key_end", lambda n, causal, off, r1: n if not causal else max(0, min(n, off + r1 - 1)))
    _fails(TA.test_naive_matches_torch_sdpa_fp64, True)
    _fails(TA.test_backward_matches_torch_autograd_fp64, True)


def test_llama_composition_slip_in_forward_and_backward_is_caught(monkeypatch):
    """A wrong rotary base in both the forward and the backward of the layer: the two stay
    consistent with each other (finite differences pass), so only the torch restatement of
    the composition can catch it."""
    from oracle import llama as LL
    import tests.test_oracle_llama as TL
    slip = ("eps=EPS, base=ROPE_BASE", "eps=EPS, base=500.0")
    monkeypatch.setattr(LL, "layer_fwd", _mutated(LL, "layer_fwd", *slip))
    monkeypatch.setattr(LL, "layer_bwd", _mutated(LL, "layer_bwd", *slip))
    TL.test_layer_backward_finite_differences(True)  # still self-consistent
    _fails(TL.test_layer_matches_torch_composition, True)
    _fails(TL.test_stack_matches_torch_composition)


def test_llama_post_norm_residual_is_caught(monkeypatch):
    """The first residual taken from the normalised input instead of x."""
    from oracle import llama as LL
    import tests.test_oracle_llama as TL
    monkeypatch.setattr(LL, "layer_fwd", _mutated(LL, "layer_fwd", "h = x + a @", "h = n1 + a @"))
    _fails(TL.test_layer_matches_torch_composition, True)
    _fails(TL.test_layer_zero_query_key_closed_form)


def test_llama_second_norm_on_the_input_is_caught(monkeypatch):
    """The feed-forward branch normalising x instead of h."""
    from oracle import llama as LL
    import tests.test_oracle_llama as TL
    monkeypatch.setattr(LL, "layer_fwd", _mutated(LL, "layer_fwd", "n2, _ = rmsnorm_fwd(h,", "n2, _ = rmsnorm_fwd(x,"))
    _fails(TL.test_layer_zero_query_key_closed_form)
    _fails(TL.test_layer_matches_torch_composition, True)


def test_layer_ffn_on_the_wrong_input_is_caught(monkeypatch):
    """The feed-forward network applied to the layer input X instead of Y = X + A Wo."""
    from oracle import layer as L
    monkeypatch.setattr(L, "layer_fwd", _mutated(L, "layer_fwd", "_ffn.ffn_fwd(y,", "_ffn.ffn_fwd(x,"))
    _fails(TF.test_layer_uniform_attention_closed_form)
    _fails(TF.test_layer_matches_torch_composition)


def test_layer_dropped_attention_residual_is_caught(monkeypatch):
    """Y = A Wo without the residual X."""
    from oracle import layer as L
    monkeypatch.setattr(L, "layer_fwd", _mutated(L, "layer_fwd", "y = x + a.reshape", "y = 0 * x + a.reshape"))
    _fails(TF.test_layer_uniform_attention_closed_form)
    _fails(TF.test_layer_matches_torch_composition)

