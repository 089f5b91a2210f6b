// A LLaMA-style layer around ring attention, and a stack of them trained with full
// recomputation (batch 1).
//
// The paper trains LLaMA models with Ring Attention (Section 4, model configuration) and
// checkpoints attention and feed-forward entirely (Section 4 settings; the appendix on
// training details).  The LLaMA pieces around the attention are not part of the paper;
// they are implemented from their usual definitions:
//   * RMSNorm  y = x / sqrt(mean(x^2) + eps) * g, eps = 1e-6, learned bf16 gain g;
//   * rotary position embedding on q and k: in each head, the interleaved pair (2i, 2i+1)
//     at global position p is rotated by p * 10000^(-2i/D);
//   * SwiGLU feed-forward (silu(x W1) * (x W3)) W2;
//   * pre-norm residual layer
//        h = x + Attention(RoPE(n1 Wq), RoPE(n1 Wk), n1 Wv) Wo,  n1 = RMSNorm(x; g1)
//        z = h + SwiGLU(RMSNorm(h; g2)).
// Projections and the feed-forward products run on the bf16 matrix-core GEMM (the SwiGLU
// gate and its derivative fused into epilogues), the attention is the ring attention of
// this library over n_hosts virtual hosts, RMSNorm and RoPE are bandwidth-bound kernels
// here.  The backward pass recomputes the layer's forward from its input.
#include <math.h>

#include "ra_common.h"
#include "ra_gemm.h"
#include "ra_kernels.h"
#include "ra_ops.h"
#include "ra_runtime.h"
#include "ringattn.h"

namespace ra {
namespace {

constexpr float kNormEps = 1e-6f;
constexpr double kRopeBase = 10000.0;
constexpr int kNormMaxD = 8192;       // d_model limit of the RMSNorm kernels
constexpr int kNormChunks = kNormMaxD / 512;
constexpr int kNormSlab = 32;         // rows per workgroup of the RMSNorm backward

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
  return v;
}

// ---- RMSNorm -----------------------------------------------------------------------------
// One wave per row (4 rows per workgroup); each lane holds 8-element chunks lane, lane + 64,
// ...  Sum of squares in float32, y = bf16(x * rstd * g).
__global__ __launch_bounds__(256) void rmsnorm_fwd_kernel(const bf16* x, const bf16* g, bf16* y, float* rstd,
                                                          int T, int d, float eps) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (row >= T) return;
  const bf16* xr = x + (long long)row * d;
  float ss = 0.f;
  for (int c = lane * 8; c < d; c += 512) {
    const bf16x8 v = *(const bf16x8*)(xr + c);
#pragma unroll
    for (int e = 0; e < 8; ++e) ss = fmaf((float)v[e], (float)v[e], ss);
  }
  const float r = rsqrtf(wave_sum(ss) / d + eps);
  bf16* yr = y + (long long)row * d;
  for (int c = lane * 8; c < d; c += 512) {
    const bf16x8 v = *(const bf16x8*)(xr + c);
    const bf16x8 gg = *(const bf16x8*)(g + c);
    u32x4 o;
#pragma unroll
    for (int e = 0; e < 4; ++e)
      o[e] = pack_bf16x2((float)v[2 * e] * r * (float)gg[2 * e], (float)v[2 * e + 1] * r * (float)gg[2 * e + 1]);
    *(u32x4*)(yr + c) = o;
  }
  if (lane == 0 && rstd) rstd[row] = r;
}

// Backward of y = x * rstd * g for upstream dy (float32):
//   dx = rstd g dy - x rstd^3 / d * sum_j(g_j dy_j x_j),   dg = sum_rows dy x rstd.
// One wave per slab of kNormSlab rows; out = bf16(dres + dx) (dres may be null);
// dg_part[slab][d] holds the slab's column sums (added up in slab order afterwards).
__global__ __launch_bounds__(64) void rmsnorm_bwd_kernel(const bf16* x, const bf16* g, const float* dy,
                                                         const bf16* dres, bf16* out, float* dg_part, int T,
                                                         int d, float eps) {
  const int lane = threadIdx.x, slab = blockIdx.x;
  float dgacc[kNormChunks][8];
#pragma unroll
  for (int i = 0; i < kNormChunks; ++i)
#pragma unroll
    for (int e = 0; e < 8; ++e) dgacc[i][e] = 0.f;
  for (int rr = 0; rr < kNormSlab; ++rr) {
    const int row = slab * kNormSlab + rr;
    if (row >= T) break;
    const bf16* xr = x + (long long)row * d;
    const float* dyr = dy + (long long)row * d;
    float ss = 0.f, sgdx = 0.f;
#pragma unroll
    for (int i = 0; i < kNormChunks; ++i) {
      const int c = lane * 8 + 512 * i;
      if (c < d) {
        const bf16x8 v = *(const bf16x8*)(xr + c);
        const bf16x8 gg = *(const bf16x8*)(g + c);
        const f32x4 d0 = *(const f32x4*)(dyr + c), d1 = *(const f32x4*)(dyr + c + 4);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float xv = (float)v[e], dv = e < 4 ? d0[e] : d1[e - 4];
          ss = fmaf(xv, xv, ss);
          sgdx = fmaf((float)gg[e] * dv, xv, sgdx);
        }
      }
    }
    ss = wave_sum(ss);
    sgdx = wave_sum(sgdx);
    const float r = rsqrtf(ss / d + eps);
    const float coef = r * r * r * sgdx / d;
    bf16* outr = out + (long long)row * d;
#pragma unroll
    for (int i = 0; i < kNormChunks; ++i) {
      const int c = lane * 8 + 512 * i;
      if (c < d) {
        const bf16x8 v = *(const bf16x8*)(xr + c);
        const bf16x8 gg = *(const bf16x8*)(g + c);
        const f32x4 d0 = *(const f32x4*)(dyr + c), d1 = *(const f32x4*)(dyr + c + 4);
        bf16x8 rv;
        if (dres) rv = *(const bf16x8*)(dres + (long long)row * d + c);
        float o[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float xv = (float)v[e], dv = e < 4 ? d0[e] : d1[e - 4];
          o[e] = r * (float)gg[e] * dv - coef * xv + (dres ? (float)rv[e] : 0.f);
          dgacc[i][e] = fmaf(dv, xv * r, dgacc[i][e]);
        }
        *(u32x4*)(outr + c) = u32x4{pack_bf16x2(o[0], o[1]), pack_bf16x2(o[2], o[3]), pack_bf16x2(o[4], o[5]),
                                     pack_bf16x2(o[6], o[7])};
      }
    }
  }
  float* part = dg_part + (long long)slab * d;
#pragma unroll
  for (int i = 0; i < kNormChunks; ++i) {
    const int c = lane * 8 + 512 * i;
    if (c < d) {
      *(f32x4*)(part + c) = f32x4{dgacc[i][0], dgacc[i][1], dgacc[i][2], dgacc[i][3]};
      *(f32x4*)(part + c + 4) = f32x4{dgacc[i][4], dgacc[i][5], dgacc[i][6], dgacc[i][7]};
    }
  }
}

// dg[c] = sum over slabs (in order) of dg_part[slab][c]
__global__ __launch_bounds__(256) void slab_sum_kernel(const float* part, float* out, int n_slabs, int d) {
  const int c = blockIdx.x * 256 + threadIdx.x;
  if (c >= d) return;
  float s = 0.f;
  for (int k = 0; k < n_slabs; ++k) s += part[(long long)k * d + c];
  out[c] = s;
}

// ---- rotary position embedding --------------------------------------------------------------
// Table of (cos, sin) of p * base^(-2i/D) for positions pos0 .. pos0 + S - 1 and i < D/2,
// computed in double precision (positions reach 10^5 rad) and stored as float pairs.
__global__ __launch_bounds__(256) void rope_table_kernel(float2* table, int S, int D, int pos0) {
  const long long idx = (long long)blockIdx.x * 256 + threadIdx.x;
  const int half = D / 2;
  if (idx >= (long long)S * half) return;
  const int p = pos0 + (int)(idx / half), i = (int)(idx % half);
  const double ang = (double)p * pow(kRopeBase, -2.0 * i / D);
  table[idx] = make_float2((float)cos(ang), (float)sin(ang));
}

// In-place rotation of x [S, H, D] (bf16): each thread rotates two adjacent pairs.
// sign = +1 (forward) or -1 (inverse, i.e. the transpose used by the backward pass).
__global__ __launch_bounds__(256) void rope_apply_kernel(bf16* x, const float2* table, int S, int H, int D,
                                                         float sign) {
  const long long q = (long long)blockIdx.x * 256 + threadIdx.x;  // quad of elements
  const long long n4 = (long long)S * H * D / 4;
  if (q >= n4) return;
  const long long e0 = q * 4;
  const int s = (int)(e0 / ((long long)H * D));
  const int dd = (int)(e0 % D);
  const float4 cs = *(const float4*)(table + (long long)s * (D / 2) + dd / 2);  // (c0, s0, c1, s1)
  bf16x4 v = *(const bf16x4*)(x + e0);
  const float x0 = (float)v[0], x1 = (float)v[1], x2 = (float)v[2], x3 = (float)v[3];
  const float s0 = sign * cs.y, s1 = sign * cs.w;
  u32x2 o = {pack_bf16x2(x0 * cs.x - x1 * s0, x0 * s0 + x1 * cs.x),
             pack_bf16x2(x2 * cs.z - x3 * s1, x2 * s1 + x3 * cs.z)};
  *(u32x2*)(x + e0) = o;
}

}  // namespace

// ---- host-side building blocks ----------------------------------------------------------------
static int check_norm(int T, int d) {
  if (T <= 0 || d <= 0) return set_err(RA_EINVAL, "sizes must be positive (T=%d d=%d)", T, d);
  if (d % 8 || d > kNormMaxD) return set_err(RA_EUNSUPPORTED, "d=%d must be a multiple of 8 and at most %d", d, kNormMaxD);
  if ((long long)T * d >= (1ll << 31)) return set_err(RA_EUNSUPPORTED, "T*d exceeds 2^31-1 elements");
  return RA_OK;
}

static size_t norm_bwd_ws_floats(int T, int d) { return (size_t)((T + kNormSlab - 1) / kNormSlab) * d; }

static int norm_fwd(const void* x, const void* g, void* y, float* rstd, int T, int d, hipStream_t st) {
  hipLaunchKernelGGL(rmsnorm_fwd_kernel, dim3((T + 3) / 4), dim3(256), 0, st, (const bf16*)x, (const bf16*)g,
                     (bf16*)y, rstd, T, d, kNormEps);
  RA_HIP(hipGetLastError());
  return RA_OK;
}

static int norm_bwd(const void* x, const void* g, const float* dy, const void* dres, void* out, float* dg,
                    float* part, int T, int d, hipStream_t st) {
  const int slabs = (T + kNormSlab - 1) / kNormSlab;
  hipLaunchKernelGGL(rmsnorm_bwd_kernel, dim3(slabs), dim3(64), 0, st, (const bf16*)x, (const bf16*)g, dy,
                     (const bf16*)dres, (bf16*)out, part, T, d, kNormEps);
  RA_HIP(hipGetLastError());
  hipLaunchKernelGGL(slab_sum_kernel, dim3((d + 255) / 256), dim3(256), 0, st, part, dg, slabs, d);
  RA_HIP(hipGetLastError());
  return RA_OK;
}

static int rope_table(float2* table, int S, int D, int pos0, hipStream_t st) {
  const long long n = (long long)S * (D / 2);
  hipLaunchKernelGGL(rope_table_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, table, S, D, pos0);
  RA_HIP(hipGetLastError());
  return RA_OK;
}

static int rope_run(void* x, const float2* table, int S, int H, int D, int inverse, hipStream_t st) {
  const long long n4 = (long long)S * H * D / 4;
  hipLaunchKernelGGL(rope_apply_kernel, dim3((unsigned)((n4 + 255) / 256)), dim3(256), 0, st, (bf16*)x, table, S, H,
                     D, inverse ? -1.f : 1.f);
  RA_HIP(hipGetLastError());
  return RA_OK;
}

// SwiGLU forward over row blocks: y = (silu(x W1) * (x W3)) W2 (+ residual).
static int swiglu_forward(const void* x, const void* w1, const void* w3, const void* w2, const void* residual, void* y,
                          int T, int dm, int dff, int block, hipStream_t st) {
  const size_t nb = (size_t)block * dff;
  CallResources R(st);
  int rc = R.alloc(nb * 4 + nb * 2);
  if (rc) return rc;
  float* u = (float*)R.ws;              // x W1, float32 [block, d_ff]
  void* gte = (char*)R.ws + nb * 4;     // gate output, bf16
  for (int r0 = 0; r0 < T; r0 += block) {
    const char* xb = (const char*)x + (size_t)r0 * dm * 2;
    GemmArgs a{};
    a.A = xb;
    a.B = w1;
    a.C = u;
    a.lda = dm;
    a.ldb = dff;
    a.ldc = dff;
    a.M = block;
    a.N = dff;
    a.K = dm;
    if ((rc = gemm(a, false, false, EPI_F32, st))) return rc;
    GemmArgs b = a;  // gte = silu(u) * (x W3)
    b.B = w3;
    b.C = gte;
    b.aux_f32 = u;
    if ((rc = gemm(b, false, false, EPI_GLU_BF16, st))) return rc;
    GemmArgs c{};
    c.A = gte;
    c.B = w2;
    c.C = (char*)y + (size_t)r0 * dm * 2;
    c.residual = residual ? (const char*)residual + (size_t)r0 * dm * 2 : nullptr;
    c.lda = dff;
    c.ldb = dm;
    c.ldc = dm;
    c.M = block;
    c.N = dm;
    c.K = dff;
    if ((rc = gemm(c, false, false, EPI_BF16, st))) return rc;
  }
  return RA_OK;
}

// SwiGLU backward over row blocks: dx32 (float32, overwritten) = du W1^T + dw W3^T and the
// weight gradients (float32, overwritten), recomputing u = x W1 and w = x W3 per block.
static int swiglu_backward(const void* x, const void* w1, const void* w3, const void* w2, const void* dy, float* dx32,
                           float* dw1, float* dw3, float* dw2, int T, int dm, int dff, int block, hipStream_t st) {
  const size_t nb = (size_t)block * dff;
  CallResources R(st);
  int rc = R.alloc(nb * 4 * 2 + nb * 2 * 3);
  if (rc) return rc;
  float* u = (float*)R.ws;
  float* w = u + nb;
  char* gte = (char*)(w + nb);
  char* du = gte + nb * 2;
  char* dw = du + nb * 2;
  for (int bi = 0, r0 = 0; r0 < T; ++bi, r0 += block) {
    const char* xb = (const char*)x + (size_t)r0 * dm * 2;
    const char* dyb = (const char*)dy + (size_t)r0 * dm * 2;
    GemmArgs a{};
    a.A = xb;
    a.B = w1;
    a.C = u;
    a.lda = dm;
    a.ldb = dff;
    a.ldc = dff;
    a.M = block;
    a.N = dff;
    a.K = dm;
    if ((rc = gemm(a, false, false, EPI_F32, st))) return rc;
    GemmArgs b = a;  // gte = silu(u) * w, and w itself
    b.B = w3;
    b.C = gte;
    b.aux_f32 = u;
    b.aux2_f32 = w;
    if ((rc = gemm(b, false, false, EPI_GLU_BF16, st))) return rc;
    GemmArgs g2{};  // dW2 (+)= gte^T dy
    g2.A = gte;
    g2.B = dyb;
    g2.C = dw2;
    g2.lda = dff;
    g2.ldb = dm;
    g2.ldc = dm;
    g2.M = dff;
    g2.N = dm;
    g2.K = block;
    g2.accumulate = bi > 0;
    if ((rc = gemm(g2, true, false, EPI_F32, st))) return rc;
    GemmArgs gg{};  // dgte = dy W2^T  ->  du = dgte w silu'(u),  dw = dgte silu(u)
    gg.A = dyb;
    gg.B = w2;
    gg.C = du;
    gg.C2 = dw;
    gg.aux_f32 = u;
    gg.aux2_f32 = w;
    gg.lda = dm;
    gg.ldb = dm;
    gg.ldc = dff;
    gg.M = block;
    gg.N = dff;
    gg.K = dm;
    if ((rc = gemm(gg, false, true, EPI_GLU_GRAD, st))) return rc;
    GemmArgs g1{};  // dW1 (+)= x^T du, dW3 (+)= x^T dw
    g1.A = xb;
    g1.B = du;
    g1.C = dw1;
    g1.lda = dm;
    g1.ldb = dff;
    g1.ldc = dff;
    g1.M = dm;
    g1.N = dff;
    g1.K = block;
    g1.accumulate = bi > 0;
    if ((rc = gemm(g1, true, false, EPI_F32, st))) return rc;
    GemmArgs g3 = g1;
    g3.B = dw;
    g3.C = dw3;
    if ((rc = gemm(g3, true, false, EPI_F32, st))) return rc;
    GemmArgs gx{};  // dx = du W1^T + dw W3^T (float32)
    gx.A = du;
    gx.B = w1;
    gx.C = dx32 + (size_t)r0 * dm;
    gx.lda = dff;
    gx.ldb = dff;
    gx.ldc = dm;
    gx.M = block;
    gx.N = dm;
    gx.K = dff;
    if ((rc = gemm(gx, false, true, EPI_F32, st))) return rc;
    gx.A = dw;
    gx.B = w3;
    gx.accumulate = 1;
    if ((rc = gemm(gx, false, true, EPI_F32, st))) return rc;
  }
  return RA_OK;
}

static int check_llama(int S, int dm, int H, int dff, int N, int causal) {
  if (S <= 0 || dm <= 0 || H <= 0 || dff <= 0 || N <= 0) return set_err(RA_EINVAL, "sizes must be positive");
  if (causal != 0 && causal != 1) return set_err(RA_EINVAL, "causal must be 0 or 1");
  if (dm % H) return set_err(RA_EUNSUPPORTED, "d_model=%d is not a multiple of n_heads=%d", dm, H);
  const int D = dm / H;
  if (D != 64 && D != 128) return set_err(RA_EUNSUPPORTED, "head dim %d not supported (64 or 128)", D);
  if (dm > kNormMaxD) return set_err(RA_EUNSUPPORTED, "d_model=%d exceeds %d", dm, kNormMaxD);
  if (S % N) return set_err(RA_EUNSUPPORTED, "S=%d is not a multiple of n_hosts=%d", S, N);
  if (N > kMaxSlots) return set_err(RA_EUNSUPPORTED, "n_hosts=%d exceeds %d", N, kMaxSlots);
  return check_gemm_dims(S, dm, dff, S / N);  // host block = projection / FFN block (multiple of 256)
}

// The layer's forward activations, kept for the backward pass.
struct LlamaActs {
  char *n1, *q, *k, *v, *o, *h, *n2;  // bf16 [S, d_model]; q, k after the rotation
  float* lse;                          // [H, S]
  float2* rope;                        // [S, D/2]
  static size_t bytes(int S, int dm, int H) {
    return 7 * (size_t)S * dm * 2 + (size_t)H * S * 4 + (size_t)S * (dm / H / 2) * 8;
  }
  void carve(void* base, int S, int dm, int H) {
    const size_t t = (size_t)S * dm * 2;
    n1 = (char*)base;
    q = n1 + t;
    k = q + t;
    v = k + t;
    o = v + t;
    h = o + t;
    n2 = h + t;
    lse = (float*)(n2 + t);
    rope = (float2*)(lse + (size_t)H * S);
  }
};

// Forward of one layer; z may be null (activations only).
static int llama_forward(const void* x, const void* const* p, void* z, LlamaActs& a, int S, int dm, int H, int dff,
                         int N, int causal, hipStream_t st) {
  const void *g1 = p[0], *wq = p[1], *wk = p[2], *wv = p[3], *wo = p[4], *g2 = p[5], *w1 = p[6], *w3 = p[7],
             *w2 = p[8];
  const int c = S / N, D = dm / H;
  int rc;
  if ((rc = norm_fwd(x, g1, a.n1, nullptr, S, dm, st))) return rc;
  if ((rc = proj(a.n1, wq, nullptr, a.q, S, dm, dm, c, st))) return rc;
  if ((rc = proj(a.n1, wk, nullptr, a.k, S, dm, dm, c, st))) return rc;
  if ((rc = proj(a.n1, wv, nullptr, a.v, S, dm, dm, c, st))) return rc;
  if ((rc = rope_table(a.rope, S, D, 0, st))) return rc;
  if ((rc = rope_run(a.q, a.rope, S, H, D, 0, st))) return rc;
  if ((rc = rope_run(a.k, a.rope, S, H, D, 0, st))) return rc;
  if ((rc = ring_attn_fwd(a.q, a.k, a.v, a.o, a.lse, 1, H, S, D, N, causal, st))) return rc;
  if ((rc = proj(a.o, wo, x, a.h, S, dm, dm, c, st))) return rc;  // h = x + o Wo
  if ((rc = norm_fwd(a.h, g2, a.n2, nullptr, S, dm, st))) return rc;
  if (!z) return RA_OK;
  return swiglu_forward(a.n2, w1, w3, w2, a.h, z, S, dm, dff, c, st);  // z = h + SwiGLU(n2)
}

static int llama_backward(const void* x, const void* const* p, const void* dz, void* dx, float* const* gr, int S,
                          int dm, int H, int dff, int N, int causal, hipStream_t st) {
  const void *g1 = p[0], *wq = p[1], *wk = p[2], *wv = p[3], *wo = p[4], *g2 = p[5], *w1 = p[6], *w3 = p[7],
             *w2 = p[8];
  float *dg1 = gr[0], *dwq = gr[1], *dwk = gr[2], *dwv = gr[3], *dwo = gr[4], *dg2 = gr[5], *dw1 = gr[6],
        *dw3 = gr[7], *dw2 = gr[8];
  const int c = S / N, D = dm / H;
  const size_t t = (size_t)S * dm;
  CallResources R(st);
  int rc = R.alloc(LlamaActs::bytes(S, dm, H) + 5 * t * 2 + t * 4 + norm_bwd_ws_floats(S, dm) * 4);
  if (rc) return rc;
  LlamaActs a;
  a.carve(R.ws, S, dm, H);
  char* dh = (char*)R.ws + LlamaActs::bytes(S, dm, H);
  char* dO = dh + t * 2;
  char* dq = dO + t * 2;
  char* dk = dq + t * 2;
  char* dv = dk + t * 2;
  float* dn32 = (float*)(dv + t * 2);
  float* part = dn32 + t;
  if ((rc = llama_forward(x, p, nullptr, a, S, dm, H, dff, N, causal, st))) return rc;
  // z = h + SwiGLU(n2):  dn2 = SwiGLU'(n2)^T dz;  dh = dz + RMSNorm'(h)^T dn2
  if ((rc = swiglu_backward(a.n2, w1, w3, w2, dz, dn32, dw1, dw3, dw2, S, dm, dff, c, st))) return rc;
  if ((rc = norm_bwd(a.h, g2, dn32, dz, dh, dg2, part, S, dm, st))) return rc;
  // h = x + o Wo:  dWo = o^T dh,  dO = dh Wo^T
  if ((rc = wgrad(a.o, dh, dwo, S, dm, dm, c, st))) return rc;
  for (int r0 = 0; r0 < S; r0 += c) {
    GemmArgs g{};
    g.A = dh + (size_t)r0 * dm * 2;
    g.B = wo;
    g.C = dO + (size_t)r0 * dm * 2;
    g.lda = dm;
    g.ldb = dm;
    g.ldc = dm;
    g.M = c;
    g.N = dm;
    g.K = dm;
    if ((rc = gemm(g, false, true, EPI_BF16, st))) return rc;
  }
  if ((rc = ring_attn_bwd(a.q, a.k, a.v, a.o, a.lse, dO, dq, dk, dv, 1, H, S, D, N, causal, st))) return rc;
  // undo the rotation on the gradients of the rotated q and k (its transpose)
  if ((rc = rope_run(dq, a.rope, S, H, D, 1, st))) return rc;
  if ((rc = rope_run(dk, a.rope, S, H, D, 1, st))) return rc;
  if ((rc = wgrad(a.n1, dq, dwq, S, dm, dm, c, st))) return rc;
  if ((rc = wgrad(a.n1, dk, dwk, S, dm, dm, c, st))) return rc;
  if ((rc = wgrad(a.n1, dv, dwv, S, dm, dm, c, st))) return rc;
  if ((rc = dgrad32(dq, wq, dn32, 0, S, dm, dm, c, st))) return rc;
  if ((rc = dgrad32(dk, wk, dn32, 1, S, dm, dm, c, st))) return rc;
  if ((rc = dgrad32(dv, wv, dn32, 1, S, dm, dm, c, st))) return rc;
  // dx = dh + RMSNorm'(x)^T dn1
  return norm_bwd(x, g1, dn32, dh, dx, dg1, part, S, dm, st);
}

}  // namespace ra

using namespace ra;

extern "C" {

int rms_norm_fwd(const void* x, const void* g, void* y, float* rstd, int T, int d, hipStream_t stream) {
  g_err.clear();
  if (!x || !g || !y) return set_err(RA_EINVAL, "null pointer argument");
  if (int e = check_aligned({x, g, y}, {rstd})) return e;
  int rc = check_norm(T, d);
  if (rc) return rc;
  return norm_fwd(x, g, y, rstd, T, d, stream);
}

int rms_norm_bwd(const void* x, const void* g, const float* dy, const void* dres, void* dx, float* dg, int T, int d,
                 hipStream_t stream) {
  g_err.clear();
  if (!x || !g || !dy || !dx || !dg) return set_err(RA_EINVAL, "null pointer argument");
  if (int e = check_aligned({x, g, dy, dres, dx, dg})) return e;
  int rc = check_norm(T, d);
  if (rc) return rc;
  CallResources R(stream);
  if ((rc = R.alloc(norm_bwd_ws_floats(T, d) * 4))) return rc;
  return norm_bwd(x, g, dy, dres, dx, dg, (float*)R.ws, T, d, stream);
}

int rope_apply(void* x, int S, int H, int D, int pos0, int inverse, hipStream_t stream) {
  g_err.clear();
  if (!x) return set_err(RA_EINVAL, "null pointer argument");
  if (int e = check_aligned({x})) return e;
  if (S <= 0 || H <= 0 || D <= 0 || pos0 < 0) return set_err(RA_EINVAL, "sizes must be positive, pos0 >= 0");
  if (inverse != 0 && inverse != 1) return set_err(RA_EINVAL, "inverse must be 0 or 1");
  if (D % 4) return set_err(RA_EUNSUPPORTED, "head dim D=%d must be a multiple of 4", D);
  if ((long long)S * H * D >= (1ll << 31) || (long long)pos0 + S >= (1ll << 31))
    return set_err(RA_EUNSUPPORTED, "sizes exceed 2^31-1");
  CallResources R(stream);
  int rc = R.alloc((size_t)S * (D / 2) * sizeof(float2));
  if (rc) return rc;
  if ((rc = rope_table((float2*)R.ws, S, D, pos0, stream))) return rc;
  return rope_run(x, (const float2*)R.ws, S, H, D, inverse, stream);
}

int swiglu_ffn(const void* x, const void* w1, const void* w3, const void* w2, const void* residual, void* y, int T,
               int d_model, int d_ff, int block, hipStream_t stream) {
  g_err.clear();
  if (!x || !w1 || !w3 || !w2 || !y) return set_err(RA_EINVAL, "null pointer argument");
  if (int e = check_aligned({x, w1, w3, w2, residual, y})) return e;
  int rc = check_gemm_dims(T, d_model, d_ff, block);
  if (rc) return rc;
  return swiglu_forward(x, w1, w3, w2, residual, y, T, d_model, d_ff, block, stream);
}

int swiglu_ffn_bwd(const void* x, const void* w1, const void* w3, const void* w2, const void* dy, void* dx, float* dw1,
                   float* dw3, float* dw2, int T, int d_model, int d_ff, int block, hipStream_t stream) {
  g_err.clear();
  if (!x || !w1 || !w3 || !w2 || !dy || !dx || !dw1 || !dw3 || !dw2) return set_err(RA_EINVAL, "null pointer argument");
  if (int e = check_aligned({x, w1, w3, w2, dy, dx, dw1, dw3, dw2})) return e;
  int rc = check_gemm_dims(T, d_model, d_ff, block);
  if (rc) return rc;
  CallResources R(stream);
  if ((rc = R.alloc((size_t)T * d_model * 4))) return rc;
  if ((rc = swiglu_backward(x, w1, w3, w2, dy, (float*)R.ws, dw1, dw3, dw2, T, d_model, d_ff, block, stream)))
    return rc;
  RA_HIP(launch_cast_f32_bf16((const float*)R.ws, dx, (long long)T * d_model, stream));
  return RA_OK;
}

int llama_layer_fwd(const void* x, const void* const* params, void* z, int S, int d_model, int n_heads, int d_ff,
                    int n_hosts, int causal, hipStream_t stream) {
  g_err.clear();
  if (!x || !params || !z) return set_err(RA_EINVAL, "null pointer argument");
  for (int i = 0; i < 9; ++i)
    if (!params[i]) return set_err(RA_EINVAL, "null parameter pointer %d", i);
  if (int e = check_aligned({x, z})) return e;
  for (int i = 0; i < 9; ++i)
    if (int e = check_aligned({params[i]})) return e;
  int rc = check_llama(S, d_model, n_heads, d_ff, n_hosts, causal);
  if (rc) return rc;
  CallResources R(stream);
  if ((rc = R.alloc(LlamaActs::bytes(S, d_model, n_heads)))) return rc;
  LlamaActs a;
  a.carve(R.ws, S, d_model, n_heads);
  return llama_forward(x, params, z, a, S, d_model, n_heads, d_ff, n_hosts, causal, stream);
}

int llama_layer_bwd(const void* x, const void* const* params, const void* dz, void* dx, float* const* grads, int S,
                    int d_model, int n_heads, int d_ff, int n_hosts, int causal, hipStream_t stream) {
  g_err.clear();
  if (!x || !params || !dz || !dx || !grads) return set_err(RA_EINVAL, "null pointer argument");
  for (int i = 0; i < 9; ++i)
    if (!params[i] || !grads[i]) return set_err(RA_EINVAL, "null parameter or gradient pointer %d", i);
  if (int e = check_aligned({x, dz, dx})) return e;
  for (int i = 0; i < 9; ++i)
    if (int e = check_aligned({params[i], grads[i]})) return e;
  int rc = check_llama(S, d_model, n_heads, d_ff, n_hosts, causal);
  if (rc) return rc;
  return llama_backward(x, params, dz, dx, grads, S, d_model, n_heads, d_ff, n_hosts, causal, stream);
}

int llama_stack_train_step(const void* x, const void* const* params, const void* dz, void* z, void* dx,
                           float* const* grads, int n_layers, int S, int d_model, int n_heads, int d_ff, int n_hosts,
                           int causal, hipStream_t stream) {
  g_err.clear();
  if (!x || !params || !dz || !z || !dx || !grads) return set_err(RA_EINVAL, "null pointer argument");
  if (n_layers <= 0) return set_err(RA_EINVAL, "n_layers=%d must be positive", n_layers);
  for (int i = 0; i < 9 * n_layers; ++i)
    if (!params[i] || !grads[i]) return set_err(RA_EINVAL, "null parameter or gradient pointer %d", i);
  if (int e = check_aligned({x, dz, z, dx})) return e;
  for (int i = 0; i < 9 * n_layers; ++i)
    if (int e = check_aligned({params[i], grads[i]})) return e;
  int rc = check_llama(S, d_model, n_heads, d_ff, n_hosts, causal);
  if (rc) return rc;
  const size_t t = (size_t)S * d_model * 2;
  CallResources R(stream);
  // inputs of layers 1 .. L-1 (layer 0's is x), two gradient buffers, one layer's activations
  if ((rc = R.alloc((size_t)(n_layers - 1) * t + 2 * t + LlamaActs::bytes(S, d_model, n_heads)))) return rc;
  char* ckpt = (char*)R.ws;
  char* gbuf[2] = {ckpt + (size_t)(n_layers - 1) * t, ckpt + (size_t)n_layers * t};
  LlamaActs a;
  a.carve(ckpt + (size_t)(n_layers + 1) * t, S, d_model, n_heads);
  auto input = [&](int l) -> const void* { return l == 0 ? x : (const void*)(ckpt + (size_t)(l - 1) * t); };
  // forward, keeping only each layer's input (the paper's full recomputation policy)
  for (int l = 0; l < n_layers; ++l) {
    void* out = l + 1 < n_layers ? (void*)(ckpt + (size_t)l * t) : z;
    if ((rc = llama_forward(input(l), params + 9 * l, out, a, S, d_model, n_heads, d_ff, n_hosts, causal, stream)))
      return rc;
  }
  // backward, last layer first; each layer recomputes its forward from its input
  const void* g = dz;
  for (int l = n_layers - 1; l >= 0; --l) {
    void* out = l == 0 ? dx : (void*)gbuf[l & 1];
    if ((rc = llama_backward(input(l), params + 9 * l, g, out, grads + 9 * l, S, d_model, n_heads, d_ff, n_hosts,
                             causal, stream)))
      return rc;
    g = out;
  }
  return RA_OK;
}

}  // extern "C"
