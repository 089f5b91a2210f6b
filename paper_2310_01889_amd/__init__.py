"""Python binding of libringattn.so, the MI355X (gfx950) ring-attention library.

Argument marshalling only: every step of the computation runs in the library's HIP
kernels.  torch supplies device memory and the current HIP stream.  Each function has
the name of the C entry point it calls (see include/ringattn.h for layouts, ownership
and error behaviour) and takes torch tensors that live on the current GPU; shapes are
read from the tensors.  Convenience wrappers that allocate their outputs are provided
for tests and benchmarks (``attention_fwd``, ``attention_bwd``, ``ffn_fwd``...).

The library is loaded on first use.  If it has not been built, or no GPU is present,
calls raise: there is no fallback path.
"""
import ctypes
import os

import torch

__all__ = [
    "RingAttnError", "library_path", "load", "exported_symbols",
    "ring_attn_fwd", "ring_attn_bwd", "ring_attn_fwd_f32", "ring_attn_bwd_f32",
    "ring_attn_fwd_host", "ring_attn_bwd_host", "ring_attn_fwd_ordered", "ring_attn_decode",
    "ring_attn_decode_noalloc",
    "blockwise_ffn", "blockwise_ffn_bwd",
    "blockwise_linear", "blockwise_linear_bwd", "ring_layer_fwd", "ring_layer_bwd",
    "rms_norm_fwd", "rms_norm_bwd", "rope_apply", "swiglu_ffn", "swiglu_ffn_bwd",
    "llama_layer_fwd", "llama_layer_bwd", "llama_stack_train_step",
    "attention_fwd", "attention_bwd", "attention_decode",
    "ACT_GELU_ERF", "ACT_RELU", "ACT_GELU_TANH",
]

ACT_GELU_ERF, ACT_RELU, ACT_GELU_TANH = 0, 1, 2
_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB = None

_P = ctypes.c_void_p
_I = ctypes.c_int
_SIGS = {
    "ring_attn_mfma_probe": [ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p],
    "ring_attn_release_workspace": [],
    "ring_attn_fwd": [_P] * 5 + [_I] * 6 + [_P],
    "ring_attn_fwd_f32": [_P] * 5 + [_I] * 6 + [_P],
    "ring_attn_bwd": [_P] * 9 + [_I] * 6 + [_P],
    "ring_attn_bwd_f32": [_P] * 9 + [_I] * 6 + [_P],
    "ring_attn_fwd_varlen": [_P] * 5 + [_I] * 5 + [_P],
    "ring_attn_bwd_varlen": [_P] * 9 + [_I] * 5 + [_P],
    "ring_attn_fwd_host": [_P] * 5 + [_I] * 7 + [_P],
    "ring_attn_bwd_host": [_P] * 9 + [_I] * 7 + [_P],
    "ring_attn_fwd_ordered": [_P] * 5 + [_I] * 6 + [_P, _P],
    "ring_attn_decode": [_P] * 5 + [_I] * 7 + [_P],
    "ring_attn_decode_noalloc": [_P] * 5 + [_I] * 7 + [_P],
    "blockwise_ffn": [_P] * 6 + [_I] * 5 + [_P],
    "blockwise_ffn_bwd": [_P] * 10 + [_I] * 5 + [_P],
    "blockwise_linear": [_P] * 4 + [_I] * 4 + [_P],
    "blockwise_linear_bwd": [_P] * 5 + [_I] * 4 + [_P],
    "ring_layer_fwd": [_P] * 8 + [_I] * 7 + [_P],
    "ring_layer_bwd": [_P] * 15 + [_I] * 7 + [_P],
    "rms_norm_fwd": [_P] * 4 + [_I] * 2 + [_P],
    "rms_norm_bwd": [_P] * 6 + [_I] * 2 + [_P],
    "rope_apply": [_P] + [_I] * 5 + [_P],
    "swiglu_ffn": [_P] * 6 + [_I] * 4 + [_P],
    "swiglu_ffn_bwd": [_P] * 9 + [_I] * 4 + [_P],
    "llama_layer_fwd": [_P] * 3 + [_I] * 6 + [_P],
    "llama_layer_bwd": [_P] * 5 + [_I] * 6 + [_P],
    "llama_stack_train_step": [_P] * 6 + [_I] * 7 + [_P],
}


class RingAttnError(RuntimeError):
    """A library call returned a non-zero ra_status."""

    def __init__(self, name, code, msg):
        super().__init__("%s failed (status %d): %s" % (name, code, msg))
        self.code = code


def library_path():
    return os.path.join(_HERE, "libringattn.so")


def load():
    """Load the shared library (once).  Raises if it is missing."""
    global _LIB
    if _LIB is None:
        path = library_path()
        if not os.path.exists(path):
            raise RuntimeError("%s is not built; run __graft_entry__.build() or "
                               "python -m paper_2310_01889_amd.build" % path)
        lib = ctypes.CDLL(path)
        for name, args in _SIGS.items():
            fn = getattr(lib, name, None)
            if fn is None:  # checked by the symbol test; calling it raises AttributeError
                continue
            fn.argtypes = args
            fn.restype = ctypes.c_int
        lib.ring_attn_last_error.argtypes = []
        lib.ring_attn_last_error.restype = ctypes.c_char_p
        lib.ring_attn_timing_enable.argtypes = [ctypes.c_int]
        lib.ring_attn_timing_enable.restype = None
        lib.ring_attn_timing_read.argtypes = [ctypes.c_int, ctypes.POINTER(ctypes.c_double),
                                              ctypes.POINTER(ctypes.c_int)]
        lib.ring_attn_timing_read.restype = ctypes.c_int
        _LIB = lib
    return _LIB


def exported_symbols():
    """Names of the C entry points the binding expects the library to export."""
    return sorted(list(_SIGS) + ["ring_attn_last_error", "ring_attn_timing_enable",
                                 "ring_attn_timing_read"])


KERNEL_ATTN_FWD, KERNEL_ATTN_BWD, KERNEL_GEMM, KERNEL_DECODE = 0, 1, 2, 3


def timing_enable(on=True):
    """Bracket every later hot-kernel launch with timing events (ring_attn_timing_enable)."""
    load().ring_attn_timing_enable(1 if on else 0)


def timing_read(kind):
    """(total milliseconds, launches) of the timed launches of ``kind`` since the last read."""
    ms, n = ctypes.c_double(0.0), ctypes.c_int(0)
    lib = load()
    rc = lib.ring_attn_timing_read(int(kind), ctypes.byref(ms), ctypes.byref(n))
    if rc != 0:
        raise RingAttnError("ring_attn_timing_read", rc, lib.ring_attn_last_error().decode())
    return ms.value, n.value


def release_workspace():
    """Return the library's cached workspace on the current device to the driver."""
    _call("ring_attn_release_workspace")


MFMA_PROBE_WAVES = 2048


def mfma_probe(iters, random_operands=False, stream=None):
    """Launch the matrix-core calibration kernel (ring_attn_mfma_probe) on the current
    stream, with fixed or random operands; returns the flops it performs.  Time it with
    events around the call."""
    import torch
    sink = torch.empty(MFMA_PROBE_WAVES, dtype=torch.float32, device="cuda")
    _call("ring_attn_mfma_probe", int(iters), 1 if random_operands else 0, sink.data_ptr(), _stream(stream))
    return float(MFMA_PROBE_WAVES) * iters * 32 * 32768


def _call(name, *args):
    lib = load()
    rc = getattr(lib, name)(*args)
    if rc != 0:
        raise RingAttnError(name, rc, lib.ring_attn_last_error().decode())


def _ptr(t, dtype=None, name="tensor"):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("%s must be a GPU tensor" % name)
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    if dtype is not None and t.dtype != dtype:
        raise TypeError("%s must be %s, got %s" % (name, dtype, t.dtype))
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _bshd(q):
    if q.dim() != 4:
        raise ValueError("expected a [B, S, H, D] tensor")
    return tuple(int(x) for x in q.shape)


# ----------------------------------------------------------------------------------
# C entry points (outputs passed in)
# ----------------------------------------------------------------------------------
def ring_attn_fwd(q, k, v, o, lse, n_hosts, causal, stream=None):
    B, S, H, D = _bshd(q)
    bf = torch.bfloat16
    _call("ring_attn_fwd", _ptr(q, bf, "q"), _ptr(k, bf, "k"), _ptr(v, bf, "v"), _ptr(o, bf, "o"),
          _ptr(lse, torch.float32, "lse"), B, H, S, D, int(n_hosts), int(causal), _stream(stream))


def ring_attn_fwd_f32(q, k, v, o, lse, n_hosts, causal, stream=None):
    B, S, H, D = _bshd(q)
    f = torch.float32
    _call("ring_attn_fwd_f32", _ptr(q, f, "q"), _ptr(k, f, "k"), _ptr(v, f, "v"), _ptr(o, f, "o"),
          _ptr(lse, f, "lse"), B, H, S, D, int(n_hosts), int(causal), _stream(stream))


def ring_attn_bwd(q, k, v, o, lse, dO, dq, dk, dv, n_hosts, causal, stream=None):
    B, S, H, D = _bshd(q)
    bf = torch.bfloat16
    _call("ring_attn_bwd", _ptr(q, bf, "q"), _ptr(k, bf, "k"), _ptr(v, bf, "v"), _ptr(o, bf, "o"),
          _ptr(lse, torch.float32, "lse"), _ptr(dO, bf, "dO"), _ptr(dq, bf, "dq"), _ptr(dk, bf, "dk"),
          _ptr(dv, bf, "dv"), B, H, S, D, int(n_hosts), int(causal), _stream(stream))


def ring_attn_bwd_f32(q, k, v, o, lse, dO, dq, dk, dv, n_hosts, causal, stream=None):
    B, S, H, D = _bshd(q)
    f = torch.float32
    _call("ring_attn_bwd_f32", _ptr(q, f, "q"), _ptr(k, f, "k"), _ptr(v, f, "v"), _ptr(o, f, "o"),
          _ptr(lse, f, "lse"), _ptr(dO, f, "dO"), _ptr(dq, f, "dq"), _ptr(dk, f, "dk"), _ptr(dv, f, "dv"),
          B, H, S, D, int(n_hosts), int(causal), _stream(stream))


def ring_attn_fwd_varlen(q, k, v, o, lse, n_hosts, stream=None):
    B, S, H, D = _bshd(q)
    bf = torch.bfloat16
    _call("ring_attn_fwd_varlen", _ptr(q, bf, "q"), _ptr(k, bf, "k"), _ptr(v, bf, "v"), _ptr(o, bf, "o"),
          _ptr(lse, torch.float32, "lse"), B, H, S, D, int(n_hosts), _stream(stream))


def ring_attn_bwd_varlen(q, k, v, o, lse, dO, dq, dk, dv, n_hosts, stream=None):
    B, S, H, D = _bshd(q)
    bf = torch.bfloat16
    _call("ring_attn_bwd_varlen", _ptr(q, bf, "q"), _ptr(k, bf, "k"), _ptr(v, bf, "v"), _ptr(o, bf, "o"),
          _ptr(lse, torch.float32, "lse"), _ptr(dO, bf, "dO"), _ptr(dq, bf, "dq"), _ptr(dk, bf, "dk"),
          _ptr(dv, bf, "dv"), B, H, S, D, int(n_hosts), _stream(stream))


def ring_attn_fwd_host(q_blk, k_all, v_all, o_blk, lse_blk, n_hosts, host_idx, causal, stream=None):
    B, c, H, D = _bshd(q_blk)
    S = int(k_all.shape[1])
    bf = torch.bfloat16
    _call("ring_attn_fwd_host", _ptr(q_blk, bf, "q_blk"), _ptr(k_all, bf, "k_all"), _ptr(v_all, bf, "v_all"),
          _ptr(o_blk, bf, "o_blk"), _ptr(lse_blk, torch.float32, "lse_blk"), B, H, S, D, int(n_hosts),
          int(host_idx), int(causal), _stream(stream))


def ring_attn_bwd_host(q_blk, k_all, v_all, o_blk, lse_blk, dO_blk, dq_blk, dk_acc, dv_acc, n_hosts, host_idx, causal,
                       stream=None):
    B, c, H, D = _bshd(q_blk)
    S = int(k_all.shape[1])
    bf, f = torch.bfloat16, torch.float32
    _call("ring_attn_bwd_host", _ptr(q_blk, bf, "q_blk"), _ptr(k_all, bf, "k_all"), _ptr(v_all, bf, "v_all"),
          _ptr(o_blk, bf, "o_blk"), _ptr(lse_blk, f, "lse_blk"), _ptr(dO_blk, bf, "dO_blk"), _ptr(dq_blk, bf, "dq_blk"),
          _ptr(dk_acc, f, "dk_acc"), _ptr(dv_acc, f, "dv_acc"), B, H, S, D, int(n_hosts), int(host_idx), int(causal),
          _stream(stream))


def ring_attn_fwd_ordered(q, k, v, o, lse, n_hosts, causal, kv_order, stream=None):
    B, S, H, D = _bshd(q)
    bf = torch.bfloat16
    flat = [int(x) for row in kv_order for x in row]
    arr = (ctypes.c_int * len(flat))(*flat)
    _call("ring_attn_fwd_ordered", _ptr(q, bf, "q"), _ptr(k, bf, "k"), _ptr(v, bf, "v"), _ptr(o, bf, "o"),
          _ptr(lse, torch.float32, "lse"), B, H, S, D, int(n_hosts), int(causal),
          ctypes.cast(arr, ctypes.c_void_p), _stream(stream))


def ring_attn_decode(q, k_cache, v_cache, o, lse, n_hosts, causal=True, stream=None):
    B, Tq, H, D = _bshd(q)
    S = int(k_cache.shape[1])
    bf = torch.bfloat16
    _call("ring_attn_decode", _ptr(q, bf, "q"), _ptr(k_cache, bf, "k_cache"), _ptr(v_cache, bf, "v_cache"),
          _ptr(o, bf, "o"), _ptr(lse, torch.float32, "lse"), B, H, S, D, Tq, int(n_hosts), int(causal),
          _stream(stream))


def ring_attn_decode_noalloc(q, k_cache, v_cache, o, lse, n_hosts, causal=True, stream=None):
    B, Tq, H, D = _bshd(q)
    S = int(k_cache.shape[1])
    bf = torch.bfloat16
    _call("ring_attn_decode_noalloc", _ptr(q, bf, "q"), _ptr(k_cache, bf, "k_cache"), _ptr(v_cache, bf, "v_cache"),
          _ptr(o, bf, "o"), _ptr(lse, torch.float32, "lse"), B, H, S, D, Tq, int(n_hosts), int(causal),
          _stream(stream))


def blockwise_ffn(x, w1, b1, w2, b2, y, block, act=ACT_GELU_ERF, stream=None):
    T, dm = (int(s) for s in x.shape)
    dff = int(w1.shape[1])
    bf = torch.bfloat16
    _call("blockwise_ffn", _ptr(x, bf, "x"), _ptr(w1, bf, "w1"), _ptr(b1, bf, "b1"), _ptr(w2, bf, "w2"),
          _ptr(b2, bf, "b2"), _ptr(y, bf, "y"), T, dm, dff, int(block), int(act), _stream(stream))


def blockwise_ffn_bwd(x, w1, b1, w2, dy, dx, dw1, db1, dw2, db2, block, act=ACT_GELU_ERF, stream=None):
    T, dm = (int(s) for s in x.shape)
    dff = int(w1.shape[1])
    bf, f = torch.bfloat16, torch.float32
    _call("blockwise_ffn_bwd", _ptr(x, bf, "x"), _ptr(w1, bf, "w1"), _ptr(b1, bf, "b1"), _ptr(w2, bf, "w2"),
          _ptr(dy, bf, "dy"), _ptr(dx, bf, "dx"), _ptr(dw1, f, "dw1"), _ptr(db1, f, "db1"), _ptr(dw2, f, "dw2"),
          _ptr(db2, f, "db2"), T, dm, dff, int(block), int(act), _stream(stream))


def blockwise_linear(x, w, residual, y, block, stream=None):
    T, di = (int(s) for s in x.shape)
    do = int(w.shape[1])
    bf = torch.bfloat16
    _call("blockwise_linear", _ptr(x, bf, "x"), _ptr(w, bf, "w"), _ptr(residual, bf, "residual"),
          _ptr(y, bf, "y"), T, di, do, int(block), _stream(stream))


def blockwise_linear_bwd(x, w, dy, dx, dw, block, stream=None):
    T, di = (int(s) for s in x.shape)
    do = int(w.shape[1])
    bf = torch.bfloat16
    _call("blockwise_linear_bwd", _ptr(x, bf, "x"), _ptr(w, bf, "w"), _ptr(dy, bf, "dy"), _ptr(dx, bf, "dx"),
          _ptr(dw, torch.float32, "dw"), T, di, do, int(block), _stream(stream))


def ring_layer_fwd(x, wq, wk, wv, wo, w1, w2, z, n_heads, n_hosts, causal=True, act=ACT_GELU_ERF, stream=None):
    S, dm = (int(s) for s in x.shape)
    dff = int(w1.shape[1])
    bf = torch.bfloat16
    _call("ring_layer_fwd", _ptr(x, bf, "x"), _ptr(wq, bf, "wq"), _ptr(wk, bf, "wk"), _ptr(wv, bf, "wv"),
          _ptr(wo, bf, "wo"), _ptr(w1, bf, "w1"), _ptr(w2, bf, "w2"), _ptr(z, bf, "z"), S, dm, int(n_heads), dff,
          int(n_hosts), int(causal), int(act), _stream(stream))


def ring_layer_bwd(x, wq, wk, wv, wo, w1, w2, dz, dx, dwq, dwk, dwv, dwo, dw1, dw2, n_heads, n_hosts, causal=True,
                   act=ACT_GELU_ERF, stream=None):
    S, dm = (int(s) for s in x.shape)
    dff = int(w1.shape[1])
    bf, f = torch.bfloat16, torch.float32
    _call("ring_layer_bwd", _ptr(x, bf, "x"), _ptr(wq, bf, "wq"), _ptr(wk, bf, "wk"), _ptr(wv, bf, "wv"),
          _ptr(wo, bf, "wo"), _ptr(w1, bf, "w1"), _ptr(w2, bf, "w2"), _ptr(dz, bf, "dz"), _ptr(dx, bf, "dx"),
          _ptr(dwq, f, "dwq"), _ptr(dwk, f, "dwk"), _ptr(dwv, f, "dwv"), _ptr(dwo, f, "dwo"), _ptr(dw1, f, "dw1"),
          _ptr(dw2, f, "dw2"), S, dm, int(n_heads), dff, int(n_hosts), int(causal), int(act), _stream(stream))


def rms_norm_fwd(x, g, y, rstd=None, stream=None):
    T, d = (int(s) for s in x.shape)
    bf = torch.bfloat16
    _call("rms_norm_fwd", _ptr(x, bf, "x"), _ptr(g, bf, "g"), _ptr(y, bf, "y"), _ptr(rstd, torch.float32, "rstd"),
          T, d, _stream(stream))


def rms_norm_bwd(x, g, dy, dres, dx, dg, stream=None):
    T, d = (int(s) for s in x.shape)
    bf, f = torch.bfloat16, torch.float32
    _call("rms_norm_bwd", _ptr(x, bf, "x"), _ptr(g, bf, "g"), _ptr(dy, f, "dy"), _ptr(dres, bf, "dres"),
          _ptr(dx, bf, "dx"), _ptr(dg, f, "dg"), T, d, _stream(stream))


def rope_apply(x, pos0=0, inverse=False, stream=None):
    """In place on a bf16 [S, H, D] tensor."""
    S, H, D = (int(s) for s in x.shape)
    _call("rope_apply", _ptr(x, torch.bfloat16, "x"), S, H, D, int(pos0), int(bool(inverse)), _stream(stream))


def swiglu_ffn(x, w1, w3, w2, residual, y, block, stream=None):
    T, dm = (int(s) for s in x.shape)
    dff = int(w1.shape[1])
    bf = torch.bfloat16
    _call("swiglu_ffn", _ptr(x, bf, "x"), _ptr(w1, bf, "w1"), _ptr(w3, bf, "w3"), _ptr(w2, bf, "w2"),
          _ptr(residual, bf, "residual"), _ptr(y, bf, "y"), T, dm, dff, int(block), _stream(stream))


def swiglu_ffn_bwd(x, w1, w3, w2, dy, dx, dw1, dw3, dw2, block, stream=None):
    T, dm = (int(s) for s in x.shape)
    dff = int(w1.shape[1])
    bf, f = torch.bfloat16, torch.float32
    _call("swiglu_ffn_bwd", _ptr(x, bf, "x"), _ptr(w1, bf, "w1"), _ptr(w3, bf, "w3"), _ptr(w2, bf, "w2"),
          _ptr(dy, bf, "dy"), _ptr(dx, bf, "dx"), _ptr(dw1, f, "dw1"), _ptr(dw3, f, "dw3"), _ptr(dw2, f, "dw2"),
          T, dm, dff, int(block), _stream(stream))


def _ptr_array(ts, dtype, name):
    arr = (ctypes.c_void_p * len(ts))(*[_ptr(t, dtype, name).value for t in ts])
    return arr, ctypes.cast(arr, ctypes.c_void_p)


def llama_layer_fwd(x, params, z, n_heads, n_hosts, causal=True, stream=None):
    """params: [g1, wq, wk, wv, wo, g2, w1, w3, w2] (bf16 tensors)."""
    S, dm = (int(s) for s in x.shape)
    dff = int(params[6].shape[1])
    keep, parr = _ptr_array(params, torch.bfloat16, "params")
    _call("llama_layer_fwd", _ptr(x, torch.bfloat16, "x"), parr, _ptr(z, torch.bfloat16, "z"), S, dm, int(n_heads),
          dff, int(n_hosts), int(causal), _stream(stream))


def llama_layer_bwd(x, params, dz, dx, grads, n_heads, n_hosts, causal=True, stream=None):
    """grads: [dg1, dwq, dwk, dwv, dwo, dg2, dw1, dw3, dw2] (float32 tensors, overwritten)."""
    S, dm = (int(s) for s in x.shape)
    dff = int(params[6].shape[1])
    bf = torch.bfloat16
    keep_p, parr = _ptr_array(params, bf, "params")
    keep_g, garr = _ptr_array(grads, torch.float32, "grads")
    _call("llama_layer_bwd", _ptr(x, bf, "x"), parr, _ptr(dz, bf, "dz"), _ptr(dx, bf, "dx"), garr, S, dm,
          int(n_heads), dff, int(n_hosts), int(causal), _stream(stream))


def llama_stack_train_step(x, layer_params, dz, z, dx, layer_grads, n_heads, n_hosts, causal=True, stream=None):
    """layer_params / layer_grads: one 9-element list per layer (as llama_layer_fwd / _bwd)."""
    S, dm = (int(s) for s in x.shape)
    dff = int(layer_params[0][6].shape[1])
    bf = torch.bfloat16
    keep_p, parr = _ptr_array([t for p in layer_params for t in p], bf, "params")
    keep_g, garr = _ptr_array([t for g in layer_grads for t in g], torch.float32, "grads")
    _call("llama_stack_train_step", _ptr(x, bf, "x"), parr, _ptr(dz, bf, "dz"), _ptr(z, bf, "z"), _ptr(dx, bf, "dx"),
          garr, len(layer_params), S, dm, int(n_heads), dff, int(n_hosts), int(causal), _stream(stream))


# ----------------------------------------------------------------------------------
# Allocating wrappers
# ----------------------------------------------------------------------------------
def attention_fwd(q, k, v, n_hosts, causal=True):
    """Returns (o, lse) for bf16 or float32 q, k, v of shape [B, S, H, D].  A bf16 causal
    sequence whose length does not fill n_hosts blocks of a multiple of 128 tokens goes
    through ring_attn_fwd_varlen (short or empty last blocks)."""
    B, S, H, D = _bshd(q)
    o = torch.empty_like(q)
    lse = torch.empty((B, H, S), dtype=torch.float32, device=q.device)
    if _ragged(q, S, n_hosts, causal):
        ring_attn_fwd_varlen(q, k, v, o, lse, n_hosts)
        return o, lse
    fn = ring_attn_fwd if q.dtype == torch.bfloat16 else ring_attn_fwd_f32
    fn(q, k, v, o, lse, n_hosts, causal)
    return o, lse


def _ragged(q, S, n_hosts, causal):
    return bool(causal) and q.dtype == torch.bfloat16 and int(n_hosts) > 0 and S % (128 * int(n_hosts)) != 0


def attention_bwd(q, k, v, o, lse, dO, n_hosts, causal=True):
    """Returns (dq, dk, dv); ragged bf16 causal lengths as in attention_fwd."""
    dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    if _ragged(q, int(q.shape[1]), n_hosts, causal):
        ring_attn_bwd_varlen(q, k, v, o, lse, dO, dq, dk, dv, n_hosts)
        return dq, dk, dv
    fn = ring_attn_bwd if q.dtype == torch.bfloat16 else ring_attn_bwd_f32
    fn(q, k, v, o, lse, dO, dq, dk, dv, n_hosts, causal)
    return dq, dk, dv


def attention_decode(q, k_cache, v_cache, n_hosts, causal=True):
    """Returns (o [B, Tq, H, D] bf16, lse [B, H, Tq] f32) of ring_attn_decode."""
    B, Tq, H, D = _bshd(q)
    o = torch.empty_like(q)
    lse = torch.empty((B, H, Tq), dtype=torch.float32, device=q.device)
    ring_attn_decode(q, k_cache, v_cache, o, lse, n_hosts, causal)
    return o, lse
