// C ABI of one transformer layer composed as Algorithm 1 lays it out (batch 1):
// per-host query/key/value projections of each input block, ring attention over the
// hosts, output projection with residual, then the blockwise feed-forward network on
// each host's block with residual.  The paper fixes neither normalisation, positional
// encoding nor biases for this layer; the composition implemented (and checked against
// the CPU oracle) is
//     Q, K, V = X Wq, X Wk, X Wv;  A = RingAttention(Q, K, V);  Y = X + A Wo;
//     Z = Y + act(Y W1) W2.
// The backward pass recomputes every activation from X (full gradient checkpointing,
// as in the paper's training setup) and returns float32 weight gradients.
#include "ra_gemm.h"
#include "ra_ops.h"
#include "ra_runtime.h"
#include "ringattn.h"

namespace ra {

static int check_layer(int S, int dm, int H, int dff, int N, int causal, int act) {
  if (S <= 0 || dm <= 0 || H <= 0 || dff <= 0 || N <= 0)
    return set_err(RA_EINVAL, "sizes must be positive");
  if (causal != 0 && causal != 1) return set_err(RA_EINVAL, "causal must be 0 or 1");
  if (act < 0 || act > 2) return set_err(RA_EINVAL, "act=%d is not an ra_act value", act);
  if (dm % H) return set_err(RA_EUNSUPPORTED, "d_model=%d is not a multiple of n_heads=%d", dm, H);
  const int D = dm / H;
  if (D != 64 && D != 128) return set_err(RA_EUNSUPPORTED, "head dim %d not supported (64 or 128)", D);
  if (S % N) return set_err(RA_EUNSUPPORTED, "S=%d is not a multiple of n_hosts=%d", S, N);
  const int c = S / N;
  int rc = check_gemm_dims(S, dm, dff, c);  // host block = projection / FFN block
  if (rc) return rc;
  if (c % 128) return set_err(RA_EUNSUPPORTED, "block S/n_hosts=%d is not a multiple of 128", c);
  return RA_OK;
}

// Forward activations shared by forward and backward: Q, K, V, O (bf16 [S, dm]), lse, Y.
struct LayerActs {
  char *q, *k, *v, *o, *y;
  float* lse;
  static size_t bytes(int S, int dm, int H) { return 5 * (size_t)S * dm * 2 + (size_t)H * S * 4; }
  void carve(void* base, int S, int dm) {
    const size_t t = (size_t)S * dm * 2;
    q = (char*)base;
    k = q + t;
    v = k + t;
    o = v + t;
    y = o + t;
    lse = (float*)(y + t);
  }
};

static int layer_acts(const void* x, const void* wq, const void* wk, const void* wv, const void* wo, LayerActs& a,
                      int S, int dm, int H, int N, int causal, hipStream_t st) {
  const int c = S / N;
  int rc;
  if ((rc = proj(x, wq, nullptr, a.q, S, dm, dm, c, st))) return rc;
  if ((rc = proj(x, wk, nullptr, a.k, S, dm, dm, c, st))) return rc;
  if ((rc = proj(x, wv, nullptr, a.v, S, dm, dm, c, st))) return rc;
  if ((rc = ring_attn_fwd(a.q, a.k, a.v, a.o, a.lse, 1, H, S, dm / H, N, causal, st))) return rc;
  return proj(a.o, wo, x, a.y, S, dm, dm, c, st);  // Y = X + A Wo
}

}  // namespace ra

using namespace ra;

extern "C" {

int ring_layer_fwd(const void* x, const void* wq, const void* wk, const void* wv, const void* wo, const void* w1,
                   const void* w2, void* z, int S, int d_model, int n_heads, int d_ff, int n_hosts, int causal,
                   int act, hipStream_t stream) {
  g_err.clear();
  if (!x || !wq || !wk || !wv || !wo || !w1 || !w2 || !z) return set_err(RA_EINVAL, "null pointer argument");
  if (int e = check_aligned({x, wq, wk, wv, wo, w1, w2, z})) return e;
  int rc = check_layer(S, d_model, n_heads, d_ff, n_hosts, causal, act);
  if (rc) return rc;
  CallResources R(stream);
  if ((rc = R.alloc(LayerActs::bytes(S, d_model, n_heads)))) return rc;
  LayerActs a;
  a.carve(R.ws, S, d_model);
  if ((rc = layer_acts(x, wq, wk, wv, wo, a, S, d_model, n_heads, n_hosts, causal, stream))) return rc;
  // Z = Y + FFN(Y), block = host block
  return ffn_forward(a.y, w1, nullptr, w2, nullptr, a.y, z, S, d_model, d_ff, S / n_hosts, act, stream);
}

int ring_layer_bwd(const void* x, const void* wq, const void* wk, const void* wv, const void* wo, const void* w1,
                   const void* w2, const void* dz, void* dx, float* dwq, float* dwk, float* dwv, float* dwo,
                   float* dw1, float* dw2, int S, int d_model, int n_heads, int d_ff, int n_hosts, int causal,
                   int act, hipStream_t stream) {
  g_err.clear();
  if (!x || !wq || !wk || !wv || !wo || !w1 || !w2 || !dz || !dx || !dwq || !dwk || !dwv || !dwo || !dw1 || !dw2)
    return set_err(RA_EINVAL, "null pointer argument");
  if (int e = check_aligned({x, wq, wk, wv, wo, w1, w2, dz, dx, dwq, dwk, dwv, dwo, dw1, dw2})) return e;
  int rc = check_layer(S, d_model, n_heads, d_ff, n_hosts, causal, act);
  if (rc) return rc;
  const int c = S / n_hosts, H = n_heads, dm = d_model;
  const size_t t = (size_t)S * dm;
  CallResources R(stream);
  // activations, then dY, dO, dQ, dK, dV (bf16) and dX accumulated in float32
  if ((rc = R.alloc(LayerActs::bytes(S, dm, H) + 5 * t * 2 + t * 4))) return rc;
  LayerActs a;
  a.carve(R.ws, S, dm);
  char* dy = (char*)R.ws + LayerActs::bytes(S, dm, H);
  char* dO = dy + t * 2;
  char* dq = dO + t * 2;
  char* dk = dq + t * 2;
  char* dv = dk + t * 2;
  float* dx32 = (float*)(dv + t * 2);
  if ((rc = layer_acts(x, wq, wk, wv, wo, a, S, dm, H, n_hosts, causal, stream))) return rc;
  // Z = Y + FFN(Y):  dY = dZ + FFN'(Y)^T dZ
  if ((rc = ffn_backward(a.y, w1, nullptr, w2, dz, dz, dy, dw1, nullptr, dw2, nullptr, S, dm, d_ff, c, act, stream)))
    return rc;
  // Y = X + A Wo:  dWo = A^T dY,  dA = dY Wo^T
  if ((rc = wgrad(a.o, dy, dwo, S, dm, dm, c, stream))) return rc;
  for (int r0 = 0; r0 < S; r0 += c) {
    GemmArgs g{};
    g.A = dy + (size_t)r0 * dm * 2;
    g.B = wo;
    g.C = dO + (size_t)r0 * dm * 2;
    g.lda = dm;
    g.ldb = dm;
    g.ldc = dm;
    g.M = c;
    g.N = dm;
    g.K = dm;
    if ((rc = gemm(g, false, true, EPI_BF16, stream))) return rc;
  }
  // ring attention backward
  if ((rc = ring_attn_bwd(a.q, a.k, a.v, a.o, a.lse, dO, dq, dk, dv, 1, H, S, dm / H, n_hosts, causal, stream)))
    return rc;
  // projections: dW* = X^T d*, dX = dY + dQ Wq^T + dK Wk^T + dV Wv^T (float32 sum, one rounding)
  if ((rc = wgrad(x, dq, dwq, S, dm, dm, c, stream))) return rc;
  if ((rc = wgrad(x, dk, dwk, S, dm, dm, c, stream))) return rc;
  if ((rc = wgrad(x, dv, dwv, S, dm, dm, c, stream))) return rc;
  if ((rc = dgrad32(dq, wq, dx32, 0, S, dm, dm, c, stream))) return rc;
  if ((rc = dgrad32(dk, wk, dx32, 1, S, dm, dm, c, stream))) return rc;
  if ((rc = dgrad32(dv, wv, dx32, 1, S, dm, dm, c, stream))) return rc;
  RA_HIP(launch_add_cast_bf16(dx32, dy, dx, (long long)t, stream));
  return RA_OK;
}

}  // extern "C"
