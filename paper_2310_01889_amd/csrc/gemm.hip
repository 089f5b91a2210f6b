// bf16 matrix-core GEMM for gfx950 with fused epilogues, and the column-sum reduction.
//
// C[M][N] = sum_k A[m][k] B[k][n] with A stored row-major [M][K] (TA = 0) or as its
// transpose [K][M] (TA = 1), B stored row-major [K][N] (TB = 0) or as [N][K] (TB = 1).
// Workgroup tile 256 x 256, 8 waves (two per SIMD) each owning a 128 x 64 sub-tile (8
// accumulators of 32 x 32): while one wave waits for operands or the barrier, the other
// keeps the matrix core busy.  K advances 32 at a time through a ring of five LDS stages
// (all 160 KB of the CU's LDS) filled by direct-to-LDS buffer loads four steps ahead of
// their use.  Tiles are kept in their
// memory layout, unpadded, with 16-byte chunks XOR-swizzled per row so that both the row
// reads and the transpose reads (an operand whose registers must run along its contiguous
// dimension) are free of bank conflicts.  Each wave computes C^T = B^T A^T so that a lane
// owns one row m of C and four consecutive columns n per register group: epilogues then
// read bias / residual / pre-activation and write C with vector accesses.
#include "ra_common.h"
#include "ra_dma.h"
#include "ra_gemm.h"
#include "ringattn.h"

namespace ra {
namespace {

constexpr int kTM = 256, kTN = 256, kTK = 32, kGT = 512;
constexpr int kNS = 5;                      // ring stages
constexpr int kTileB = 256 * kTK * 2;       // bytes of one operand tile (16 KB)
constexpr int kLoadsPerTile = kTileB / 1024 / (kGT / 64);  // 1 KB loads per wave per tile

// Tile layouts in LDS (no padding; chunk = 16 bytes = 8 elements):
//   row tile   [256][32] (A with TA = 0, B with TB = 1): 64-byte rows of 4 chunks, logical
//              chunk c of row r stored at c ^ ((r >> 2) & 3);
//   k-major    [32][256] (A with TA = 1, B with TB = 0): 512-byte rows of 32 chunks,
//              logical chunk c of row r stored at c ^ (4 (r & 3)).
// A one-wave direct-to-LDS load fills 1 KB: 16 rows of a row tile, or 2 rows of a k-major
// tile, lane i landing at byte 16 i; the swizzle is applied to the global address.
__device__ __forceinline__ int swz_row(int r) { return (r >> 2) & 3; }
__device__ __forceinline__ int swz_kmaj(int r) { return 4 * (r & 3); }

// sigmoid(u); silu(u) = u sigmoid(u) has derivative sigmoid(u) (1 + u (1 - sigmoid(u)))
// (SwiGLU gate)
__device__ __forceinline__ float sigmoid_f(float u) { return __builtin_amdgcn_rcpf(1.f + __expf(-u)); }

// Exact GeLU h Phi(h) and Phi(h), phi(h) (standard normal CDF and density) from the erfc
// approximation of Abramowitz and Stegun, formula 7.1.26: with a = |h| / sqrt(2),
//   0.5 erfc(a) = Phi(-|h|) ~ t (b1 + t (b2 + t (b3 + t (b4 + t b5)))) exp(-a^2),
//   t = 1 / (1 + p a), p = 0.3275911, b_i half the published a_i
// (absolute error below 1.5e-7 in erf).  The lower tail is formed directly, without the
// cancellation of 1 + erf for negative h; one reciprocal and one exponential, a third of
// the instructions of a library erf in the epilogue.
__device__ __forceinline__ float gauss_lower(float h, float& e) {  // Phi(-|h|); e = exp(-h^2 / 2)
  const float t = __builtin_amdgcn_rcpf(fmaf(0.3275911f * 0.7071067811865476f, fabsf(h), 1.f));
  e = fast_exp2(h * (h * (-0.5f * kLog2e)));
  const float poly =
      t * fmaf(t, fmaf(t, fmaf(t, fmaf(t, 0.5307027145f, -0.7265760135f), 0.7107068705f), -0.142248368f), 0.127414796f);
  return poly * e;
}
__device__ __forceinline__ float gelu_erf(float h) {
  float e;
  const float hl = h * gauss_lower(h, e);
  return h >= 0.f ? h - hl : hl;
}
__device__ __forceinline__ float gauss_cdf(float h, float& pdf) {
  float e;
  const float lower = gauss_lower(h, e);
  pdf = 0.3989422804014327f * e;
  return h >= 0.f ? 1.f - lower : lower;
}

template <int ACT>
__device__ __forceinline__ float act_apply(float h) {
  constexpr int act = ACT;
  if (act == 1) return fmaxf(h, 0.f);
  if (act == 2) {  // 0.5 (1 + tanh(u)) = sigmoid(2 u)
    const float u = 0.7978845608028654f * (h + 0.044715f * h * h * h);
    return h * sigmoid_f(2.f * u);
  }
  return gelu_erf(h);
}


template <int ACT>
__device__ __forceinline__ float act_grad(float h) {
  constexpr int act = ACT;
  if (act == 1) return h > 0.f ? 1.f : 0.f;
  if (act == 2) {  // with s = sigmoid(2 u): 0.5 (1 + tanh u) = s, 0.5 (1 - tanh^2 u) = 2 s (1 - s)
    const float u = 0.7978845608028654f * (h + 0.044715f * h * h * h);
    const float sg = sigmoid_f(2.f * u);
    const float du = 0.7978845608028654f * (1.f + 3.f * 0.044715f * h * h);
    return sg + 2.f * h * sg * (1.f - sg) * du;
  }
  float pdf;
  const float cdf = gauss_cdf(h, pdf);
  return cdf + h * pdf;
}


// ACT: the activation of the ACT epilogues (an ra_act value, fixed at compile time so
// that each kernel holds the code of one activation only).
template <bool TA, bool TB, int EPI, int ACT>
__global__ __launch_bounds__(kGT, 1) void gemm_kernel(const GemmArgs g) {
  // one LDS object per stage (A tile, then B tile), so that reads of one stage are known not
  // to alias the direct-to-LDS loads in flight into the others
  __shared__ __attribute__((aligned(1024))) char sS0[2 * kTileB];
  __shared__ __attribute__((aligned(1024))) char sS1[2 * kTileB];
  __shared__ __attribute__((aligned(1024))) char sS2[2 * kTileB];
  __shared__ __attribute__((aligned(1024))) char sS3[2 * kTileB];
  __shared__ __attribute__((aligned(1024))) char sS4[2 * kTileB];
  auto stage = [&](auto Sc) __attribute__((always_inline)) -> char* {
    constexpr int S = decltype(Sc)::value % kNS;
    if constexpr (S == 0) return sS0; else if constexpr (S == 1) return sS1; else if constexpr (S == 2) return sS2;
    else if constexpr (S == 3) return sS3; else return sS4;
  };

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
  const int wm = wave >> 2, wn = wave & 3;  // 128 rows x 64 columns per wave
  const bf16* A = (const bf16*)g.A;
  const bf16* B = (const bf16*)g.B;
  const int nk = g.K / kTK;

  f32x16 acc[2][4];  // [n tile][m tile] of C^T
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b)
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[a][b][i] = 0.f;

  // ---- direct-to-LDS loads: per-lane byte offsets from the tile origin (fixed), and
  // the tile origin, which moves by kTK along K (scalar) ------------------------------
  // load j of this wave fills LDS bytes [(wave * kLoadsPerTile + j) * 1024, +1024)
  auto lane_off = [&](bool kmajor, long long ld, int j) __attribute__((always_inline)) -> int {
    const int blk = wave * kLoadsPerTile + j;
    if (!kmajor) {  // 16 rows x 4 chunks
      const int r = blk * 16 + (lane >> 2), pc = lane & 3;
      return (int)(2 * (r * ld + 8 * (pc ^ swz_row(r))));
    }
    const int r = blk * 2 + (lane >> 5), pc = lane & 31;  // 2 rows x 32 chunks
    return (int)(2 * (r * ld + 8 * (pc ^ swz_kmaj(r))));
  };
  int aoff[kLoadsPerTile], boff[kLoadsPerTile];
#pragma unroll
  for (int j = 0; j < kLoadsPerTile; ++j) {
    aoff[j] = lane_off(TA, g.lda, j);
    boff[j] = lane_off(!TB, g.ldb, j);
  }
  // extent of a tile's reads (bytes from its origin), for the buffer descriptors
  const int a_ext = (int)(2 * (TA ? (long long)(kTK - 1) * g.lda + kTM : (long long)(kTM - 1) * g.lda + kTK));
  const int b_ext = (int)(2 * (TB ? (long long)(kTN - 1) * g.ldb + kTK : (long long)(kTK - 1) * g.ldb + kTN));
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);
  auto load_stage = [&](int kt, auto Sc) __attribute__((always_inline)) {
    const int k0 = kt * kTK;
    const bf16* at = TA ? A + (long long)k0 * g.lda + m0 : A + (long long)m0 * g.lda + k0;
    const bf16* bt = TB ? B + (long long)n0 * g.ldb + k0 : B + (long long)k0 * g.ldb + n0;
    const __amdgpu_buffer_rsrc_t ra_ = make_rsrc(at, a_ext), rb_ = make_rsrc(bt, b_ext);
    const unsigned st = lds_addr(stage(Sc)) + wave_u * kLoadsPerTile * 1024;
#pragma unroll
    for (int j = 0; j < kLoadsPerTile; ++j) {
      dma_lds16(ra_, st + j * 1024, aoff[j]);  // tile loads the loop waits for itself
      dma_lds16(rb_, st + kTileB + j * 1024, boff[j]);
    }
  };

  // ---- LDS read offsets (bytes within an operand tile) --------------------------------
  // row-tile operand: rows base + l32 (base a multiple of 32), logical chunk 2 kk + hi
  int roff[2];
#pragma unroll
  for (int kk = 0; kk < 2; ++kk) roff[kk] = l32 * 64 + 16 * ((2 * kk + hi) ^ swz_row(l32));
  // k-major operand by transpose reads: rows 16 kk + 8 hi + li / 4 (and + 4), columns
  // base + 32 t + 16 (gq & 1) + 4 (li & 3) for t = 0..3 (A: base 128 wm, a multiple of 128,
  // which the swizzle leaves in place) or t = 0..1 (B: columns 64 wn + ..., swizzled whole)
  const int gq = lane >> 4, li = lane & 15;
  const int trow = 8 * hi + (li >> 2);
  int toff[4], tboff[2];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const int col = 32 * t + 16 * (gq & 1) + 4 * (li & 3);
    toff[t] = trow * 512 + 16 * ((col >> 3) ^ swz_kmaj(trow)) + 2 * (col & 7);
  }
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const int col = 64 * wn + 32 * t + 16 * (gq & 1) + 4 * (li & 3);
    tboff[t] = trow * 512 + 16 * ((col >> 3) ^ swz_kmaj(trow)) + 2 * (col & 7);
  }
  // operand fetch for k-slice kk of a stage: A operand rows m (bop: B^T rows n)
  auto fetch = [&](const char* st, int kk, bf16x8* aop, bf16x8* bop) __attribute__((always_inline)) {
    const char* as = st;
    const char* bs = st + kTileB;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      if (!TA) {
        aop[i] = *(const bf16x8*)(as + (wm * 128 + 32 * i) * 64 + roff[kk]);
      } else {
        const char* p = as + kk * 16 * 512 + wm * 256 + toff[i];
        const bf16x4 lo = lds_read_tr16((const bf16*)p), up = lds_read_tr16((const bf16*)(p + 4 * 512));
        aop[i] = bf16x8{lo[0], lo[1], lo[2], lo[3], up[0], up[1], up[2], up[3]};
      }
    }
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      if (TB) {
        bop[i] = *(const bf16x8*)(bs + (wn * 64 + 32 * i) * 64 + roff[kk]);
      } else {
        const char* p = bs + kk * 16 * 512 + tboff[i];
        const bf16x4 lo = lds_read_tr16((const bf16*)p), up = lds_read_tr16((const bf16*)(p + 4 * 512));
        bop[i] = bf16x8{lo[0], lo[1], lo[2], lo[3], up[0], up[1], up[2], up[3]};
      }
    }
  };
  auto mfmas = [&](const bf16x8* aop, const bf16x8* bop, int n0i, int n1i) __attribute__((always_inline)) {
#pragma unroll
    for (int ni = n0i; ni < n1i; ++ni)
#pragma unroll
      for (int mi = 0; mi < 4; ++mi) acc[ni][mi] = mfma32(bop[ni], aop[mi], acc[ni][mi]);
  };

  // ---- main loop ----------------------------------------------------------------------
  // Step kt (stage kt % 5): issue the loads of step kt+4 into the stage step kt-1 used;
  // slice 0's products while slice 1's operands are read; then wait for step kt+1's loads
  // (those of kt+2 .. kt+4 may stay in flight -- loads complete in issue order), the
  // barrier (every read of this stage has been issued by now), and step kt+1's slice-0
  // reads, covered by slice 1's products.
  bf16x8 a0[4], b0[2], a1[4], b1[2];
#pragma unroll
  for (int s = 0; s < kNS - 1; ++s)
    if (s < nk) {
      if (s == 0) load_stage(s, std::integral_constant<int, 0>{});
      if (s == 1) load_stage(s, std::integral_constant<int, 1>{});
      if (s == 2) load_stage(s, std::integral_constant<int, 2>{});
      if (s == 3) load_stage(s, std::integral_constant<int, 3>{});
    }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  fetch(sS0, 0, a0, b0);
  auto step = [&](auto Sc, int kt) __attribute__((always_inline)) {
    constexpr int S = decltype(Sc)::value;
    if (kt + kNS - 1 < nk) load_stage(kt + kNS - 1, std::integral_constant<int, (S + kNS - 1) % kNS>{});
    fetch(stage(Sc), 1, a1, b1);
    mfmas(a0, b0, 0, 2);
    // step kt+1 must have landed: at most the loads of steps kt+2 .. kt+4 outstanding
    constexpr int LPS = 2 * kLoadsPerTile;  // loads per step per wave
    if (kt + 4 < nk)
      asm volatile("s_waitcnt vmcnt(%0)" ::"n"(3 * LPS) : "memory");
    else if (kt + 3 < nk)
      asm volatile("s_waitcnt vmcnt(%0)" ::"n"(2 * LPS) : "memory");
    else if (kt + 2 < nk)
      asm volatile("s_waitcnt vmcnt(%0)" ::"n"(LPS) : "memory");
    else
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    lds_barrier();
    if (kt + 1 < nk) fetch(stage(std::integral_constant<int, S + 1>{}), 0, a0, b0);
    mfmas(a1, b1, 0, 2);
  };
  int kt = 0;
  for (; kt + kNS - 1 < nk; kt += kNS) {
    step(std::integral_constant<int, 0>{}, kt);
    step(std::integral_constant<int, 1>{}, kt + 1);
    step(std::integral_constant<int, 2>{}, kt + 2);
    step(std::integral_constant<int, 3>{}, kt + 3);
    step(std::integral_constant<int, 4>{}, kt + 4);
  }
  if (kt < nk) step(std::integral_constant<int, 0>{}, kt++);
  if (kt < nk) step(std::integral_constant<int, 1>{}, kt++);
  if (kt < nk) step(std::integral_constant<int, 2>{}, kt++);
  if (kt < nk) step(std::integral_constant<int, 3>{}, kt++);

  // ---- epilogue --------------------------------------------------------------------
  // The float32 accumulators pass through LDS (the stage buffers are free now) in two
  // passes of 128 rows: the two waves owning those rows write them, 32 rows per stage
  // buffer (1 KB rows; 16-byte chunk c of row r stored at c ^ (r & 15), so both the
  // writes -- 32 rows at one column -- and the row reads are free of bank conflicts);
  // then every wave takes 4 rows of each buffer and a lane handles 4 consecutive columns,
  // so bias, residual, pre-activation and output accesses are contiguous along rows.
  auto epi4 = [&](int m, int n, float* v) __attribute__((always_inline)) {
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
  };
#pragma unroll
  for (int pass = 0; pass < 2; ++pass) {
    if (wm == pass) {
      // lane: row 32 mi + l32 of the pass (stage buffer mi, local row l32), columns
      // 64 wn + 32 ni + 8 q4 + 4 hi .. +3 (chunk 16 wn + 8 ni + 2 q4 + hi)
      static_for<0, 4>([&](auto Mi) __attribute__((always_inline)) {
        constexpr int mi = decltype(Mi)::value;
        char* sb = stage(std::integral_constant<int, mi>{}) + l32 * 1024;
#pragma unroll
        for (int ni = 0; ni < 2; ++ni)
#pragma unroll
          for (int q4 = 0; q4 < 4; ++q4) {
            const int c = 16 * wn + 8 * ni + 2 * q4 + hi;
            *(f32x4*)(sb + 16 * (c ^ (l32 & 15))) =
                f32x4{acc[ni][mi][4 * q4], acc[ni][mi][4 * q4 + 1], acc[ni][mi][4 * q4 + 2], acc[ni][mi][4 * q4 + 3]};
          }
      });
    }
    __syncthreads();
    static_for<0, 4>([&](auto Bi) __attribute__((always_inline)) {
      constexpr int bi = decltype(Bi)::value;
      const char* sb = stage(std::integral_constant<int, bi>{});
#pragma unroll 2
      for (int rr = 0; rr < 4; ++rr) {
        const int lr = 4 * wave + rr;  // local row of the buffer
        const f32x4 t = *(const f32x4*)(sb + lr * 1024 + 16 * (lane ^ (lr & 15)));
        float v[4] = {t[0], t[1], t[2], t[3]};
        epi4(m0 + 128 * pass + 32 * bi + lr, n0 + 4 * lane, v);
      }
    });
    if (pass == 0) __syncthreads();
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
  const int total = (g.M / kTM) * (g.N / kTN);
  hipLaunchKernelGGL((gemm_kernel<TA, TB, EPI, ACT>), dim3(total), dim3(kGT), 0, st, g);
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
