"""C-ABI checks that need no GPU: the library loads, exports every entry point its
header declares, and rejects invalid arguments with the documented status codes before
touching the device (pointer arguments here are never dereferenced)."""
import ctypes
import os
import re

import pytest

import paper_2310_01889_amd as ra

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ringattn.h")

RA_OK, RA_EINVAL, RA_EUNSUPPORTED = 0, 1, 2
FAKE = ctypes.c_void_p(0x1000)  # never dereferenced: validation fails first
NULL = ctypes.c_void_p(0)


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?(?:int|void|char)\s*\*?\s*(\w+)\s*\(", text, flags=re.M)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(ra.library_path()):
        pytest.skip("library not built")
    return ra.load()


def test_header_declares_what_the_binding_expects():
    assert header_functions() == ra.exported_symbols()


def test_library_exports_every_header_symbol(lib):
    for name in header_functions():
        assert hasattr(lib, name), name


def _fwd(lib, *, q=FAKE, B=1, H=1, S=1024, D=128, N=4, causal=1):
    return lib.ring_attn_fwd(q, FAKE, FAKE, FAKE, FAKE, B, H, S, D, N, causal, NULL)


def test_attention_argument_validation(lib):
    assert _fwd(lib, q=NULL) == RA_EINVAL
    assert b"null" in lib.ring_attn_last_error()
    assert _fwd(lib, B=0) == RA_EINVAL
    assert _fwd(lib, N=0) == RA_EINVAL
    assert _fwd(lib, causal=2) == RA_EINVAL
    assert _fwd(lib, D=96) == RA_EUNSUPPORTED
    assert _fwd(lib, N=3) == RA_EUNSUPPORTED          # S % n_hosts
    assert _fwd(lib, S=1024, N=16) == RA_EUNSUPPORTED  # block 64 not a multiple of 128
    assert _fwd(lib, N=65, S=65 * 128) == RA_EUNSUPPORTED
    assert _fwd(lib, B=1 << 10, H=64, S=1 << 16) == RA_EUNSUPPORTED  # > 2^31 elements
    assert b"2^31" in lib.ring_attn_last_error()
    # float32 variant accepts 64-token blocks but not 32
    assert lib.ring_attn_fwd_f32(FAKE, FAKE, FAKE, FAKE, FAKE, 1, 1, 1024, 64, 32, 1, NULL) == RA_EUNSUPPORTED
    assert lib.ring_attn_fwd_host(FAKE, FAKE, FAKE, FAKE, FAKE, 1, 1, 1024, 128, 4, 4, 1, NULL) == RA_EINVAL
    bad = (ctypes.c_int * 4)(0, 0, 1, 0)  # row 0 repeats block 0
    assert lib.ring_attn_fwd_ordered(FAKE, FAKE, FAKE, FAKE, FAKE, 1, 1, 512, 128, 2, 1,
                                     ctypes.cast(bad, ctypes.c_void_p), NULL) == RA_EINVAL
    assert b"permutation" in lib.ring_attn_last_error()
    assert lib.ring_attn_bwd(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, NULL,
                             1, 1, 1024, 128, 4, 1, NULL) == RA_EINVAL


def test_varlen_argument_validation(lib):
    """Ragged-length causal entry points: any S >= 1 is accepted in principle; these calls
    all fail validation, so nothing is allocated or enqueued."""
    def fwd(*, q=FAKE, B=1, H=1, S=1000, D=128, N=3):
        return lib.ring_attn_fwd_varlen(q, FAKE, FAKE, FAKE, FAKE, B, H, S, D, N, NULL)
    assert fwd(q=NULL) == RA_EINVAL
    assert fwd(S=0) == RA_EINVAL
    assert fwd(N=0) == RA_EINVAL
    assert fwd(B=0) == RA_EINVAL
    assert fwd(D=96) == RA_EUNSUPPORTED
    assert fwd(N=65) == RA_EUNSUPPORTED
    assert fwd(S=(1 << 31) - 1, N=64) == RA_EUNSUPPORTED  # padded length above 2^31 - 1
    assert b"padded length" in lib.ring_attn_last_error()
    assert fwd(B=1 << 10, H=64, S=(1 << 16) - 5) == RA_EUNSUPPORTED  # padded tensor > 2^31 elements
    assert lib.ring_attn_bwd_varlen(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, NULL,
                                    1, 1, 1000, 128, 3, NULL) == RA_EINVAL
    assert lib.ring_attn_bwd_varlen(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
                                    1, 1, 1000, 96, 3, NULL) == RA_EUNSUPPORTED


def test_decode_argument_validation(lib):
    def dec(*, q=FAKE, B=1, H=2, S=4096, D=128, Tq=1, N=8, causal=1):
        return lib.ring_attn_decode(q, FAKE, FAKE, FAKE, FAKE, B, H, S, D, Tq, N, causal, NULL)
    assert dec(q=NULL) == RA_EINVAL
    assert dec(Tq=0) == RA_EINVAL
    assert dec(S=16, N=1, Tq=17) == RA_EINVAL            # more queries than cache
    assert dec(causal=-1) == RA_EINVAL
    assert dec(Tq=33) == RA_EUNSUPPORTED                 # at most 32 query tokens
    assert b"32" in lib.ring_attn_last_error()
    assert dec(D=80) == RA_EUNSUPPORTED
    assert dec(S=4096, N=3) == RA_EUNSUPPORTED           # S % n_hosts
    assert dec(S=4096 + 16 * 8, N=8) == RA_EUNSUPPORTED  # block 528 not a multiple of 32
    assert dec(N=65, S=65 * 64) == RA_EUNSUPPORTED
    assert dec(B=1 << 10, H=64, S=1 << 16, N=8) == RA_EUNSUPPORTED


def test_llama_argument_validation(lib):
    P9 = (ctypes.c_void_p * 9)(*([0x1000] * 9))
    pp = ctypes.cast(P9, ctypes.c_void_p)
    f = lib.llama_layer_fwd
    assert f(NULL, pp, FAKE, 1024, 256, 2, 512, 4, 1, NULL) == RA_EINVAL
    assert f(FAKE, pp, FAKE, 1024, 256, 3, 512, 4, 1, NULL) == RA_EUNSUPPORTED   # d_model % n_heads
    assert f(FAKE, pp, FAKE, 1024, 384, 4, 512, 4, 1, NULL) == RA_EUNSUPPORTED   # head dim 96
    assert f(FAKE, pp, FAKE, 1024, 256, 2, 500, 4, 1, NULL) == RA_EUNSUPPORTED   # d_ff % 256
    assert f(FAKE, pp, FAKE, 1024, 256, 2, 512, 8, 1, NULL) == RA_EUNSUPPORTED   # block 128 < 256
    assert f(FAKE, pp, FAKE, 1024, 16384, 128, 512, 4, 1, NULL) == RA_EUNSUPPORTED  # d_model > 8192
    bad = (ctypes.c_void_p * 9)(*([0x1000] * 8 + [0]))
    assert f(FAKE, ctypes.cast(bad, ctypes.c_void_p), FAKE, 1024, 256, 2, 512, 4, 1, NULL) == RA_EINVAL
    assert lib.llama_stack_train_step(FAKE, pp, FAKE, FAKE, FAKE, pp, 0, 1024, 256, 2, 512, 4, 1, NULL) == RA_EINVAL
    assert lib.rms_norm_fwd(FAKE, FAKE, FAKE, NULL, 16, 12, NULL) == RA_EUNSUPPORTED  # d % 8
    assert lib.rms_norm_fwd(FAKE, FAKE, FAKE, NULL, 16, 16384, NULL) == RA_EUNSUPPORTED
    assert lib.rms_norm_bwd(FAKE, FAKE, FAKE, NULL, FAKE, NULL, 16, 256, NULL) == RA_EINVAL
    assert lib.rope_apply(FAKE, 16, 2, 6, 0, 0, NULL) == RA_EUNSUPPORTED  # D % 4
    assert lib.rope_apply(FAKE, 16, 2, 8, -1, 0, NULL) == RA_EINVAL
    assert lib.rope_apply(FAKE, 16, 2, 8, 0, 2, NULL) == RA_EINVAL
    assert lib.swiglu_ffn(FAKE, FAKE, FAKE, FAKE, NULL, FAKE, 512, 256, 300, 256, NULL) == RA_EUNSUPPORTED
    assert lib.swiglu_ffn_bwd(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, NULL, FAKE, 512, 256, 512, 256,
                              NULL) == RA_EINVAL


def test_ffn_argument_validation(lib):
    f = lib.blockwise_ffn
    assert f(FAKE, FAKE, NULL, FAKE, NULL, FAKE, 512, 256, 512, 256, 5, NULL) == RA_EINVAL
    assert f(FAKE, FAKE, NULL, FAKE, NULL, FAKE, 500, 256, 512, 250, 0, NULL) == RA_EUNSUPPORTED
    assert f(FAKE, FAKE, NULL, FAKE, NULL, FAKE, 512, 256, 500, 256, 0, NULL) == RA_EUNSUPPORTED
    assert f(NULL, FAKE, NULL, FAKE, NULL, FAKE, 512, 256, 512, 256, 0, NULL) == RA_EINVAL
    assert lib.blockwise_linear(FAKE, FAKE, NULL, FAKE, 512, 256, 300, 256, NULL) == RA_EUNSUPPORTED
    assert lib.blockwise_linear_bwd(FAKE, FAKE, FAKE, NULL, NULL, 512, 256, 256, 256, NULL) == RA_EINVAL
    assert lib.blockwise_ffn_bwd(FAKE, FAKE, NULL, FAKE, FAKE, FAKE, FAKE, NULL, FAKE, NULL,
                                 512, 256, 512, 256, 3, NULL) == RA_EINVAL


def test_misaligned_pointers_are_rejected(lib):
    """Row tensors are accessed with 16-byte vector loads and stores from their start, so
    they must begin on a 16-byte boundary; lse needs 4 bytes.  Either is rejected with
    RA_EINVAL before any device work."""
    MIS16, MIS4 = ctypes.c_void_p(0x1008), ctypes.c_void_p(0x1002)
    assert lib.ring_attn_fwd(MIS16, FAKE, FAKE, FAKE, FAKE, 1, 1, 1024, 128, 4, 1, NULL) == RA_EINVAL
    assert b"16-byte" in lib.ring_attn_last_error()
    assert lib.ring_attn_fwd(FAKE, FAKE, FAKE, FAKE, MIS4, 1, 1, 1024, 128, 4, 1, NULL) == RA_EINVAL
    assert b"4-byte" in lib.ring_attn_last_error()
    assert lib.ring_attn_bwd(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, MIS16, FAKE,
                             1, 1, 1024, 128, 4, 1, NULL) == RA_EINVAL
    assert lib.ring_attn_bwd_host(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, MIS16,
                                  1, 1, 1024, 128, 4, 1, 1, NULL) == RA_EINVAL
    assert lib.ring_attn_decode(FAKE, FAKE, FAKE, MIS16, FAKE, 1, 2, 4096, 128, 1, 8, 1, NULL) == RA_EINVAL
    assert lib.ring_attn_decode_noalloc(FAKE, MIS16, FAKE, FAKE, FAKE, 1, 2, 4096, 128, 1, 8, 1, NULL) == RA_EINVAL
    assert lib.blockwise_ffn(FAKE, FAKE, MIS16, FAKE, NULL, FAKE, 512, 256, 512, 256, 0, NULL) == RA_EINVAL
    assert lib.blockwise_linear(FAKE, FAKE, NULL, MIS16, 512, 256, 256, 256, NULL) == RA_EINVAL
    P9 = (ctypes.c_void_p * 9)(*([0x1000] * 8 + [0x1008]))
    assert lib.llama_layer_fwd(FAKE, ctypes.cast(P9, ctypes.c_void_p), FAKE, 1024, 256, 2, 512, 4, 1,
                               NULL) == RA_EINVAL
    assert lib.rope_apply(MIS16, 16, 2, 8, 0, 0, NULL) == RA_EINVAL


def test_product_path_does_not_use_the_oracle():
    """The package never imports the CPU oracle (it would be a silent CPU fallback)."""
    pkg = os.path.join(ROOT, "paper_2310_01889_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".h", ".cpp")):
                text = open(os.path.join(dirpath, f)).read()
                assert not re.search(r"^\s*(from|import)\s+oracle\b", text, flags=re.M), f


def test_mfma_probe_argument_validation(lib):
    assert lib.ring_attn_mfma_probe(1, 0, NULL, NULL) == RA_EINVAL
    assert lib.ring_attn_mfma_probe(0, 0, FAKE, NULL) == RA_EINVAL
    assert lib.ring_attn_mfma_probe((1 << 20) + 1, 1, FAKE, NULL) == RA_EINVAL
    assert b"iters" in lib.ring_attn_last_error()
    assert lib.ring_attn_mfma_probe(1, 2, FAKE, NULL) == RA_EINVAL
    assert b"random_operands" in lib.ring_attn_last_error()
