// C ABI of the blockwise feed-forward network and the per-block projections.
//
// The feed-forward network of Section 2 is applied to `block` rows at a time
// (Blockwise Parallel Transformers, Section 2; the feed-forward step of Algorithm 1),
// so the [rows, d_ff] intermediate exists for one block only.  Every product runs in
// the bf16 matrix-core GEMM; bias, activation, residual and activation-derivative are
// fused into its epilogue.  The backward pass recomputes each block's pre-activation
// (gradient checkpointing) and accumulates weight gradients in float32.
#include "ra_gemm.h"
#include "ra_ops.h"
#include "ra_runtime.h"
#include "ringattn.h"

namespace ra {

int check_gemm_dims(int T, int d_in, int d_out, int block) {
  if (!(T > 0 && d_in > 0 && d_out > 0 && block > 0))
    return set_err(RA_EINVAL, "sizes must be positive (T=%d d_in=%d d_out=%d block=%d)", T, d_in, d_out, block);
  if (T % block) return set_err(RA_EUNSUPPORTED, "T=%d is not a multiple of block=%d", T, block);
  if (block % 256 || d_in % 256 || d_out % 256)
    return set_err(RA_EUNSUPPORTED, "block=%d, d_in=%d and d_out=%d must be multiples of 256", block, d_in, d_out);
  if ((long long)T * d_in >= (1ll << 31) || (long long)T * d_out >= (1ll << 31) ||
      (long long)block * d_in >= (1ll << 31) || (long long)d_in * d_out >= (1ll << 31))
    return set_err(RA_EUNSUPPORTED, "tensor sizes exceed 2^31-1 elements");
  return RA_OK;
}

int gemm(const GemmArgs& g, bool ta, bool tb, int epi, hipStream_t st) {
  RA_HIP(timed_launch(RA_KERNEL_GEMM, st, [&] { return launch_gemm(g, ta, tb, epi, st); }));
  return RA_OK;
}

// y (bf16) = x w (+ residual), row blocks of `block`
int proj(const void* x, const void* w, const void* residual, void* y, int T, int din, int dout, int block,
                hipStream_t st) {
  for (int r0 = 0; r0 < T; r0 += block) {
    GemmArgs g{};
    g.A = (const char*)x + (size_t)r0 * din * 2;
    g.B = w;
    g.C = (char*)y + (size_t)r0 * dout * 2;
    g.residual = residual ? (const char*)residual + (size_t)r0 * dout * 2 : nullptr;
    g.lda = din;
    g.ldb = dout;
    g.ldc = dout;
    g.M = block;
    g.N = dout;
    g.K = din;
    int rc = gemm(g, false, false, EPI_BF16, st);
    if (rc) return rc;
  }
  return RA_OK;
}

// dW (f32, overwritten) = x^T dy, accumulated over row blocks
int wgrad(const void* x, const void* dy, float* dw, int T, int din, int dout, int block, hipStream_t st) {
  for (int bi = 0, r0 = 0; r0 < T; ++bi, r0 += block) {
    GemmArgs g{};
    g.A = (const char*)x + (size_t)r0 * din * 2;
    g.B = (const char*)dy + (size_t)r0 * dout * 2;
    g.C = dw;
    g.lda = din;
    g.ldb = dout;
    g.ldc = dout;
    g.M = din;
    g.N = dout;
    g.K = block;
    g.accumulate = bi > 0;
    int rc = gemm(g, true, false, EPI_F32, st);
    if (rc) return rc;
  }
  return RA_OK;
}

// dx32 (f32) (+)= dy w^T, row blocks
int dgrad32(const void* dy, const void* w, float* dx32, int accumulate, int T, int din, int dout, int block,
                   hipStream_t st) {
  for (int r0 = 0; r0 < T; r0 += block) {
    GemmArgs g{};
    g.A = (const char*)dy + (size_t)r0 * dout * 2;
    g.B = w;
    g.C = dx32 + (size_t)r0 * din;
    g.lda = dout;
    g.ldb = dout;
    g.ldc = din;
    g.M = block;
    g.N = din;
    g.K = dout;
    g.accumulate = accumulate;
    int rc = gemm(g, false, true, EPI_F32, st);
    if (rc) return rc;
  }
  return RA_OK;
}

int ffn_forward(const void* x, const void* w1, const void* b1, const void* w2, const void* b2, const void* residual,
                void* y, int T, int d_model, int d_ff, int block, int act, hipStream_t stream) {
  int rc;
  CallResources R(stream);
  rc = R.alloc((size_t)block * d_ff * 2);
  if (rc) return rc;
  void* a = R.ws;  // activation of one block, bf16 [block, d_ff]
  for (int r0 = 0; r0 < T; r0 += block) {
    GemmArgs up{};
    up.A = (const char*)x + (size_t)r0 * d_model * 2;
    up.B = w1;
    up.C = a;
    up.bias = b1;
    up.lda = d_model;
    up.ldb = d_ff;
    up.ldc = d_ff;
    up.M = block;
    up.N = d_ff;
    up.K = d_model;
    up.act = act;
    rc = gemm(up, false, false, EPI_ACT_BF16, stream);
    if (rc) return rc;
    GemmArgs dn{};
    dn.A = a;
    dn.B = w2;
    dn.C = (char*)y + (size_t)r0 * d_model * 2;
    dn.bias = b2;
    dn.residual = residual ? (const char*)residual + (size_t)r0 * d_model * 2 : nullptr;
    dn.lda = d_ff;
    dn.ldb = d_model;
    dn.ldc = d_model;
    dn.M = block;
    dn.N = d_model;
    dn.K = d_ff;
    rc = gemm(dn, false, false, EPI_BF16, stream);
    if (rc) return rc;
  }
  return RA_OK;
}

int ffn_backward(const void* x, const void* w1, const void* b1, const void* w2, const void* dy, const void* dx_residual,
                 void* dx, float* dw1, float* db1, float* dw2, float* db2, int T, int d_model, int d_ff, int block,
                 int act, hipStream_t stream) {
  int rc;
  const size_t nb = (size_t)block * d_ff;
  const size_t part = colsum_workspace_floats(d_ff > d_model ? d_ff : d_model);
  CallResources R(stream);
  rc = R.alloc(nb * 4 + nb * 2 + nb * 2 + part * 4);
  if (rc) return rc;
  float* h = (float*)R.ws;                       // pre-activation, float32 [block, d_ff]
  void* a = (char*)R.ws + nb * 4;                // activation, bf16
  void* dh = (char*)R.ws + nb * 6;               // gradient of the pre-activation, bf16
  float* parts = (float*)((char*)R.ws + nb * 8);  // column-sum partials
  for (int bi = 0, r0 = 0; r0 < T; ++bi, r0 += block) {
    const char* xb = (const char*)x + (size_t)r0 * d_model * 2;
    const char* dyb = (const char*)dy + (size_t)r0 * d_model * 2;
    GemmArgs up{};  // recompute H = x W1 + b1 and A = act(H)
    up.A = xb;
    up.B = w1;
    up.C = a;
    up.bias = b1;
    up.aux_f32 = h;
    up.lda = d_model;
    up.ldb = d_ff;
    up.ldc = d_ff;
    up.M = block;
    up.N = d_ff;
    up.K = d_model;
    up.act = act;
    if ((rc = gemm(up, false, false, EPI_ACT_STORE_H, stream))) return rc;
    GemmArgs gA{};  // dH = (dy W2^T) * act'(H)
    gA.A = dyb;
    gA.B = w2;
    gA.C = dh;
    gA.aux_f32 = h;
    gA.lda = d_model;
    gA.ldb = d_model;
    gA.ldc = d_ff;
    gA.M = block;
    gA.N = d_ff;
    gA.K = d_model;
    gA.act = act;
    if ((rc = gemm(gA, false, true, EPI_ACT_GRAD_BF16, stream))) return rc;
    GemmArgs gw2{};  // dW2 (+)= A^T dy
    gw2.A = a;
    gw2.B = dyb;
    gw2.C = dw2;
    gw2.lda = d_ff;
    gw2.ldb = d_model;
    gw2.ldc = d_model;
    gw2.M = d_ff;
    gw2.N = d_model;
    gw2.K = block;
    gw2.accumulate = bi > 0;
    if ((rc = gemm(gw2, true, false, EPI_F32, stream))) return rc;
    if (db2) RA_HIP(launch_colsum_bf16(dyb, parts, db2, block, d_model, bi > 0, stream));
    GemmArgs gw1{};  // dW1 (+)= x^T dH
    gw1.A = xb;
    gw1.B = dh;
    gw1.C = dw1;
    gw1.lda = d_model;
    gw1.ldb = d_ff;
    gw1.ldc = d_ff;
    gw1.M = d_model;
    gw1.N = d_ff;
    gw1.K = block;
    gw1.accumulate = bi > 0;
    if ((rc = gemm(gw1, true, false, EPI_F32, stream))) return rc;
    if (db1) RA_HIP(launch_colsum_bf16(dh, parts, db1, block, d_ff, bi > 0, stream));
    GemmArgs gx{};  // dx = dH W1^T
    gx.A = dh;
    gx.B = w1;
    gx.C = (char*)dx + (size_t)r0 * d_model * 2;
    gx.residual = dx_residual ? (const char*)dx_residual + (size_t)r0 * d_model * 2 : nullptr;
    gx.lda = d_ff;
    gx.ldb = d_ff;
    gx.ldc = d_model;
    gx.M = block;
    gx.N = d_model;
    gx.K = d_ff;
    if ((rc = gemm(gx, false, true, EPI_BF16, stream))) return rc;
  }
  return RA_OK;
}

}  // namespace ra

using namespace ra;

extern "C" {

int blockwise_ffn(const void* x, const void* w1, const void* b1, const void* w2, const void* b2, void* y, int T,
                  int d_model, int d_ff, int block, int act, hipStream_t stream) {
  g_err.clear();
  if (!x || !w1 || !w2 || !y) return set_err(RA_EINVAL, "null pointer argument");
  if (int e = check_aligned({x, w1, b1, w2, b2, y})) return e;
  if (act < 0 || act > 2) return set_err(RA_EINVAL, "act=%d is not an ra_act value", act);
  int rc = check_gemm_dims(T, d_model, d_ff, block);
  if (rc) return rc;
  return ffn_forward(x, w1, b1, w2, b2, nullptr, y, T, d_model, d_ff, block, act, stream);
}

int blockwise_ffn_bwd(const void* x, const void* w1, const void* b1, const void* w2, const void* dy, void* dx,
                      float* dw1, float* db1, float* dw2, float* db2, int T, int d_model, int d_ff, int block,
                      int act, hipStream_t stream) {
  g_err.clear();
  if (!x || !w1 || !w2 || !dy || !dx || !dw1 || !dw2) return set_err(RA_EINVAL, "null pointer argument");
  if (int e = check_aligned({x, w1, b1, w2, dy, dx, dw1, db1, dw2, db2})) return e;
  if (act < 0 || act > 2) return set_err(RA_EINVAL, "act=%d is not an ra_act value", act);
  int rc = check_gemm_dims(T, d_model, d_ff, block);
  if (rc) return rc;
  return ffn_backward(x, w1, b1, w2, dy, nullptr, dx, dw1, db1, dw2, db2, T, d_model, d_ff, block, act, stream);
}

int blockwise_linear(const void* x, const void* w, const void* residual, void* y, int T, int d_in, int d_out,
                     int block, hipStream_t stream) {
  g_err.clear();
  if (!x || !w || !y) return set_err(RA_EINVAL, "null pointer argument");
  if (int e = check_aligned({x, w, residual, y})) return e;
  int rc = check_gemm_dims(T, d_in, d_out, block);
  if (rc) return rc;
  for (int r0 = 0; r0 < T; r0 += block) {
    GemmArgs g{};
    g.A = (const char*)x + (size_t)r0 * d_in * 2;
    g.B = w;
    g.C = (char*)y + (size_t)r0 * d_out * 2;
    g.residual = residual ? (const char*)residual + (size_t)r0 * d_out * 2 : nullptr;
    g.lda = d_in;
    g.ldb = d_out;
    g.ldc = d_out;
    g.M = block;
    g.N = d_out;
    g.K = d_in;
    if ((rc = gemm(g, false, false, EPI_BF16, stream))) return rc;
  }
  return RA_OK;
}

int blockwise_linear_bwd(const void* x, const void* w, const void* dy, void* dx, float* dw, int T, int d_in,
                         int d_out, int block, hipStream_t stream) {
  g_err.clear();
  if (!x || !w || !dy || !dw) return set_err(RA_EINVAL, "null pointer argument");
  if (int e = check_aligned({x, w, dy, dx, dw})) return e;
  int rc = check_gemm_dims(T, d_in, d_out, block);
  if (rc) return rc;
  for (int bi = 0, r0 = 0; r0 < T; ++bi, r0 += block) {
    const char* dyb = (const char*)dy + (size_t)r0 * d_out * 2;
    if (dx) {
      GemmArgs g{};  // dx = dy W^T
      g.A = dyb;
      g.B = w;
      g.C = (char*)dx + (size_t)r0 * d_in * 2;
      g.lda = d_out;
      g.ldb = d_out;
      g.ldc = d_in;
      g.M = block;
      g.N = d_in;
      g.K = d_out;
      if ((rc = gemm(g, false, true, EPI_BF16, stream))) return rc;
    }
    GemmArgs gw{};  // dW (+)= x^T dy
    gw.A = (const char*)x + (size_t)r0 * d_in * 2;
    gw.B = dyb;
    gw.C = dw;
    gw.lda = d_in;
    gw.ldb = d_out;
    gw.ldc = d_out;
    gw.M = d_in;
    gw.N = d_out;
    gw.K = block;
    gw.accumulate = bi > 0;
    if ((rc = gemm(gw, true, false, EPI_F32, stream))) return rc;
  }
  return RA_OK;
}

}  // extern "C"
