// bf16 matrix-core GEMM for gfx950 with fused epilogues, and the column-sum reduction.
//
// C[M][N] = sum_k A[m][k] B[k][n] with A stored row-major [M][K] (TA = 0) or as its
// transpose [K][M] (TA = 1), B stored row-major [K][N] (TB = 0) or as [N][K] (TB = 1).
// Workgroup tile 256 x 256, K step 64, 4 waves each owning a 128 x 128 sub-tile
// (16 accumulators of 32 x 32).  Tiles are staged through LDS in their memory layout
// (double buffered); an operand whose registers must run along its contiguous
// dimension is read with the LDS transpose read.  Each wave computes C^T = B^T A^T so
// that a lane owns one row m of C and four consecutive columns n per register group:
// epilogues then read bias / residual / pre-activation and write C with vector accesses.
#include "ra_common.h"
#include "ra_gemm.h"
#include "ringattn.h"

namespace ra {
namespace {

constexpr int kTM = 256, kTN = 256, kTK = 64, kGT = 256;

template <int ACT>
__device__ __forceinline__ float act_apply(float h) {
  constexpr int act = ACT;
  if (act == 1) return fmaxf(h, 0.f);
  if (act == 2) {
    const float u = 0.7978845608028654f * (h + 0.044715f * h * h * h);
    return 0.5f * h * (1.f + tanhf(u));
  }
  return 0.5f * h * (1.f + erff(h * 0.7071067811865476f));
}

// silu(u) = u sigmoid(u) and its derivative sigmoid(u) (1 + u (1 - sigmoid(u))) (SwiGLU gate)
__device__ __forceinline__ float sigmoid_f(float u) { return __builtin_amdgcn_rcpf(1.f + __expf(-u)); }

template <int ACT>
__device__ __forceinline__ float act_grad(float h) {
  constexpr int act = ACT;
  if (act == 1) return h > 0.f ? 1.f : 0.f;
  if (act == 2) {
    const float u = 0.7978845608028654f * (h + 0.044715f * h * h * h);
    const float t = tanhf(u);
    const float du = 0.7978845608028654f * (1.f + 3.f * 0.044715f * h * h);
    return 0.5f * (1.f + t) + 0.5f * h * (1.f - t * t) * du;
  }
  const float cdf = 0.5f * (1.f + erff(h * 0.7071067811865476f));
  const float pdf = 0.3989422804014327f * expf(-0.5f * h * h);
  return cdf + h * pdf;
}

template <bool TA, bool TB>
struct TileShape {
  // LDS tiles kept in memory layout: rows x (cols + pad) elements
  static constexpr int A_ROWS = TA ? kTK : kTM, A_COLS = TA ? kTM : kTK, A_LD = A_COLS + (TA ? 16 : 8);
  static constexpr int B_ROWS = TB ? kTN : kTK, B_COLS = TB ? kTK : kTN, B_LD = B_COLS + (TB ? 8 : 16);
  static constexpr int A_ELEMS = A_ROWS * A_LD, B_ELEMS = B_ROWS * B_LD;
  static constexpr int A_CHUNKS = A_ROWS * A_COLS / 8 / kGT;  // 16-byte chunks per thread
  static constexpr int B_CHUNKS = B_ROWS * B_COLS / 8 / kGT;
};

// ACT: the activation of the ACT epilogues (an ra_act value, fixed at compile time so
// that each kernel holds the code of one activation only).
template <bool TA, bool TB, int EPI, int ACT>
__global__ __launch_bounds__(kGT, 1) void gemm_kernel(const GemmArgs g) {
  using TS = TileShape<TA, TB>;
  extern __shared__ __attribute__((aligned(16))) bf16 smem[];
  // buffer b of A at smem + b*A_ELEMS; buffer b of B at smem + 2*A_ELEMS + b*B_ELEMS

  // tile order: XCD-contiguous ranges, then groups of 8 tile-rows sweeping across N
  const int tiles_m = g.M / kTM, tiles_n = g.N / kTN;
  const int total = tiles_m * tiles_n;
  const int L = xcd_swizzle(blockIdx.x, total);
  const int GM = 8;
  const int group = L / (GM * tiles_n);
  const int first_m = group * GM;
  const int gsize = min(GM, tiles_m - first_m);
  const int tm = first_m + (L % (GM * tiles_n)) % gsize;
  const int tn = (L % (GM * tiles_n)) / gsize;
  const int m0 = tm * kTM, n0 = tn * kTN;

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, l32 = lane & 31, hi = lane >> 5;
  const int wm = wave >> 1, wn = wave & 1;
  const bf16* A = (const bf16*)g.A;
  const bf16* B = (const bf16*)g.B;

  f32x16 acc[4][4];  // [n tile][m tile] of C^T
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b)
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[a][b][i] = 0.f;

  u32x4 apre[TS::A_CHUNKS], bpre[TS::B_CHUNKS];
  auto gload = [&](int kt) {
    const int k0 = kt * kTK;
#pragma unroll
    for (int c = 0; c < TS::A_CHUNKS; ++c) {
      const int ch = tid + c * kGT;
      const int r = ch / (TS::A_COLS / 8), col = (ch % (TS::A_COLS / 8)) * 8;
      const long long off = TA ? (long long)(k0 + r) * g.lda + m0 + col : (long long)(m0 + r) * g.lda + k0 + col;
      apre[c] = *(const u32x4*)(A + off);
    }
#pragma unroll
    for (int c = 0; c < TS::B_CHUNKS; ++c) {
      const int ch = tid + c * kGT;
      const int r = ch / (TS::B_COLS / 8), col = (ch % (TS::B_COLS / 8)) * 8;
      const long long off = TB ? (long long)(n0 + r) * g.ldb + k0 + col : (long long)(k0 + r) * g.ldb + n0 + col;
      bpre[c] = *(const u32x4*)(B + off);
    }
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int c = 0; c < TS::A_CHUNKS; ++c) {
      const int ch = tid + c * kGT;
      const int r = ch / (TS::A_COLS / 8), col = (ch % (TS::A_COLS / 8)) * 8;
      *(u32x4*)(smem + buf * TS::A_ELEMS + r * TS::A_LD + col) = apre[c];
    }
#pragma unroll
    for (int c = 0; c < TS::B_CHUNKS; ++c) {
      const int ch = tid + c * kGT;
      const int r = ch / (TS::B_COLS / 8), col = (ch % (TS::B_COLS / 8)) * 8;
      *(u32x4*)(smem + 2 * TS::A_ELEMS + buf * TS::B_ELEMS + r * TS::B_LD + col) = bpre[c];
    }
  };

  const int gq = lane >> 4, li = lane & 15;
  const int tcol = 16 * (gq & 1) + 4 * (li & 3);  // transpose-read column offset
  const int trow = 8 * hi + (li >> 2);            // transpose-read row offset
  const int nk = g.K / kTK;
  gload(0);
  lstore(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) gload(kt + 1);
    const bf16* a_s = smem + buf * TS::A_ELEMS;
    const bf16* b_s = smem + 2 * TS::A_ELEMS + buf * TS::B_ELEMS;
#pragma unroll
    for (int kk = 0; kk < kTK / 16; ++kk) {
      bf16x8 bop[4], aop[4];
#pragma unroll
      for (int ni = 0; ni < 4; ++ni) {
        const int nb = wn * 128 + 32 * ni;
        if (TB) {
          bop[ni] = *(const bf16x8*)(b_s + (nb + l32) * TS::B_LD + 16 * kk + 8 * hi);
        } else {
          const bf16* p = b_s + (16 * kk + trow) * TS::B_LD + nb + tcol;
          const bf16x4 lo = lds_read_tr16(p), up = lds_read_tr16(p + 4 * TS::B_LD);
          bop[ni] = bf16x8{lo[0], lo[1], lo[2], lo[3], up[0], up[1], up[2], up[3]};
        }
      }
#pragma unroll
      for (int mi = 0; mi < 4; ++mi) {
        const int mb = wm * 128 + 32 * mi;
        if (!TA) {
          aop[mi] = *(const bf16x8*)(a_s + (mb + l32) * TS::A_LD + 16 * kk + 8 * hi);
        } else {
          const bf16* p = a_s + (16 * kk + trow) * TS::A_LD + mb + tcol;
          const bf16x4 lo = lds_read_tr16(p), up = lds_read_tr16(p + 4 * TS::A_LD);
          aop[mi] = bf16x8{lo[0], lo[1], lo[2], lo[3], up[0], up[1], up[2], up[3]};
        }
      }
#pragma unroll
      for (int ni = 0; ni < 4; ++ni)
#pragma unroll
        for (int mi = 0; mi < 4; ++mi) acc[ni][mi] = mfma32(bop[ni], aop[mi], acc[ni][mi]);
    }
    if (kt + 1 < nk) lstore(buf ^ 1);
    __syncthreads();
  }

  // ---- epilogue: lane owns row m, registers 4g..4g+3 hold columns n0..n0+3 ----------
#pragma unroll
  for (int mi = 0; mi < 4; ++mi) {
    const int m = m0 + wm * 128 + 32 * mi + l32;
#pragma unroll
    for (int ni = 0; ni < 4; ++ni)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const int n = n0 + wn * 128 + 32 * ni + 8 * q4 + 4 * hi;
        float v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = acc[ni][mi][4 * q4 + e];
        const long long off = (long long)m * g.ldc + n;
        if (EPI == EPI_BF16 || EPI == EPI_ACT_BF16 || EPI == EPI_ACT_STORE_H) {
          if (g.bias) {
            const bf16x4 bb = *(const bf16x4*)((const bf16*)g.bias + n);
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] += (float)bb[e];
          }
          if (EPI == EPI_ACT_STORE_H) *(f32x4*)(g.aux_f32 + off) = f32x4{v[0], v[1], v[2], v[3]};
          if (EPI != EPI_BF16) {
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] = act_apply<ACT>(v[e]);
          }
          if (g.residual) {
            const bf16x4 rr = *(const bf16x4*)((const bf16*)g.residual + off);
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] += (float)rr[e];
          }
          *(u32x2*)((bf16*)g.C + off) = u32x2{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
        } else if (EPI == EPI_ACT_GRAD_BF16) {
          const f32x4 h = *(const f32x4*)(g.aux_f32 + off);
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] *= act_grad<ACT>(h[e]);
          *(u32x2*)((bf16*)g.C + off) = u32x2{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
        } else if (EPI == EPI_GLU_BF16) {
          const f32x4 u = *(const f32x4*)(g.aux_f32 + off);
          if (g.aux2_f32) *(f32x4*)(g.aux2_f32 + off) = f32x4{v[0], v[1], v[2], v[3]};
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] *= u[e] * sigmoid_f(u[e]);
          *(u32x2*)((bf16*)g.C + off) = u32x2{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
        } else if (EPI == EPI_GLU_GRAD) {
          const f32x4 u = *(const f32x4*)(g.aux_f32 + off);
          const f32x4 w = *(const f32x4*)(g.aux2_f32 + off);
          float du[4], dw[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float sg = sigmoid_f(u[e]);
            du[e] = v[e] * w[e] * sg * (1.f + u[e] * (1.f - sg));
            dw[e] = v[e] * u[e] * sg;
          }
          *(u32x2*)((bf16*)g.C + off) = u32x2{pack_bf16x2(du[0], du[1]), pack_bf16x2(du[2], du[3])};
          *(u32x2*)((bf16*)g.C2 + off) = u32x2{pack_bf16x2(dw[0], dw[1]), pack_bf16x2(dw[2], dw[3])};
        } else {  // EPI_F32: overwrite, or add into C
          f32x4* cp = (f32x4*)((float*)g.C + off);
          if (g.accumulate) {
            const f32x4 c = *cp;
            *cp = f32x4{c[0] + v[0], c[1] + v[1], c[2] + v[2], c[3] + v[3]};
          } else {
            *cp = f32x4{v[0], v[1], v[2], v[3]};
          }
        }
      }
  }
}

// Column sums of a [M, N] matrix (bf16 or float32), deterministic two-pass reduction:
// pass 1 writes partial sums of row slabs, pass 2 adds the slabs into out (+= or =).
constexpr int kCS = 64;  // row slabs
template <typename T>
__global__ __launch_bounds__(256) void colsum_partial_kernel(const T* x, float* part, int M, int N) {
  const int n = blockIdx.x * 256 + threadIdx.x;
  const int slab = blockIdx.y;
  if (n >= N) return;
  const int rows = (M + kCS - 1) / kCS;
  const int r0 = slab * rows, r1 = min(M, r0 + rows);
  float s = 0.f;
  for (int r = r0; r < r1; ++r) s += (float)x[(long long)r * N + n];
  part[(long long)slab * N + n] = s;
}
__global__ __launch_bounds__(256) void colsum_final_kernel(const float* part, float* out, int N, int accumulate) {
  const int n = blockIdx.x * 256 + threadIdx.x;
  if (n >= N) return;
  float s = 0.f;
  for (int sl = 0; sl < kCS; ++sl) s += part[(long long)sl * N + n];
  out[n] = accumulate ? out[n] + s : s;
}

template <bool TA, bool TB, int EPI, int ACT>
hipError_t launch_t(const GemmArgs& g, hipStream_t st) {
  using TS = TileShape<TA, TB>;
  const size_t lds = (size_t)(2 * TS::A_ELEMS + 2 * TS::B_ELEMS) * sizeof(bf16);
  // the tiles need more than the default dynamic LDS limit (set on the current device)
  hipError_t e = hipFuncSetAttribute((const void*)gemm_kernel<TA, TB, EPI, ACT>,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  const int total = (g.M / kTM) * (g.N / kTN);
  hipLaunchKernelGGL((gemm_kernel<TA, TB, EPI, ACT>), dim3(total), dim3(kGT), lds, st, g);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm(const GemmArgs& g, bool ta, bool tb, int epi, hipStream_t st) {
  if (g.M % kTM || g.N % kTN || g.K % kTK) return hipErrorInvalidValue;
#define RA_GEMM_CASE(TA_, TB_, E_) \
  if (ta == TA_ && tb == TB_ && epi == E_) return launch_t<TA_, TB_, E_, 0>(g, st);
#define RA_GEMM_CASE_ACT(TA_, TB_, E_)                                                 \
  if (ta == TA_ && tb == TB_ && epi == E_) {                                           \
    if (g.act == RA_ACT_RELU) return launch_t<TA_, TB_, E_, RA_ACT_RELU>(g, st);       \
    if (g.act == RA_ACT_GELU_TANH) return launch_t<TA_, TB_, E_, RA_ACT_GELU_TANH>(g, st); \
    return launch_t<TA_, TB_, E_, RA_ACT_GELU_ERF>(g, st);                             \
  }
  RA_GEMM_CASE(false, false, EPI_BF16)
  RA_GEMM_CASE_ACT(false, false, EPI_ACT_BF16)
  RA_GEMM_CASE_ACT(false, false, EPI_ACT_STORE_H)
  RA_GEMM_CASE(false, true, EPI_BF16)
  RA_GEMM_CASE_ACT(false, true, EPI_ACT_GRAD_BF16)
  RA_GEMM_CASE(true, false, EPI_F32)
  RA_GEMM_CASE(false, true, EPI_F32)
  RA_GEMM_CASE(false, false, EPI_F32)
  RA_GEMM_CASE(false, false, EPI_GLU_BF16)
  RA_GEMM_CASE(false, true, EPI_GLU_GRAD)
#undef RA_GEMM_CASE
#undef RA_GEMM_CASE_ACT
  return hipErrorInvalidValue;
}

int gemm_tile_m() { return kTM; }
int gemm_tile_n() { return kTN; }
int gemm_tile_k() { return kTK; }

hipError_t launch_colsum_bf16(const void* x, float* part, float* out, int M, int N, int accumulate,
                              hipStream_t st) {
  hipLaunchKernelGGL(colsum_partial_kernel<bf16>, dim3((N + 255) / 256, kCS), dim3(256), 0, st, (const bf16*)x,
                     part, M, N);
  hipLaunchKernelGGL(colsum_final_kernel, dim3((N + 255) / 256), dim3(256), 0, st, part, out, N, accumulate);
  return hipGetLastError();
}

size_t colsum_workspace_floats(int N) { return (size_t)kCS * N; }

namespace {
__global__ __launch_bounds__(256) void add_cast_kernel(const float* a, const bf16* b, bf16* out, long long n) {
  const long long i = ((long long)blockIdx.x * 256 + threadIdx.x) * 4;
  if (i + 3 < n) {
    const f32x4 x = *(const f32x4*)(a + i);
    const bf16x4 y = *(const bf16x4*)(b + i);
    *(u32x2*)(out + i) = u32x2{pack_bf16x2(x[0] + (float)y[0], x[1] + (float)y[1]),
                               pack_bf16x2(x[2] + (float)y[2], x[3] + (float)y[3])};
  } else {
    for (long long j = i; j < n; ++j) out[j] = (bf16)(a[j] + (float)b[j]);
  }
}
}  // namespace

hipError_t launch_add_cast_bf16(const float* a, const void* b, void* out, long long n, hipStream_t st) {
  const long long blocks = (n / 4 + 255) / 256 + 1;
  hipLaunchKernelGGL(add_cast_kernel, dim3(blocks), dim3(256), 0, st, a, (const bf16*)b, (bf16*)out, n);
  return hipGetLastError();
}

}  // namespace ra
