// Ring-attention backward step kernels for gfx950.
//
// The backward pass of the paper's Appendix A keeps dq on the host and lets dk, dv
// travel with their key/value block; each step adds one block's contribution.  With
// the saved log-sum-exp of each query row, the normalised probabilities are recomputed
// (gradient checkpointing: nothing of size [queries, keys] is stored) and
//     P = exp(s - lse),  dV += P^T dO,  dP = dO V^T,  dS = P * (dP - Delta),
//     dQ += dS K / sqrt(D),  dK += dS^T Q / sqrt(D),   Delta_r = sum_d dO_rd O_rd.
// Each step runs two kernels: one owning key tiles (dK, dV in registers, looping over
// the host's query tiles) and one owning query tiles (dQ in registers, looping over the
// block's key tiles).  Both write their tile once per step, so no atomics are needed.
#include "ra_common.h"
#include "ra_dma.h"
#include "ra_kernels.h"

namespace ra {
namespace {


// -------------------------------------------------------------------------------------
// Delta_r = sum_d dO_rd * O_rd  (float32 [B, H, S]).  A workgroup takes a tile of kPreR
// consecutive query rows x kPreH consecutive heads of one batch: TPR threads per (row,
// head) read that row of o and dO, heads fastest (so a row's kPreH heads are one contiguous
// run of memory); the sums pass through LDS, and the results (and lse) are then written
// (read) head by head as runs of kPreR consecutive floats.
// The bf16 step kernels take -Delta and -lse sqrt(D) (their accumulators start there:
// the score accumulators hold q.k, in units of the unscaled products).
// -------------------------------------------------------------------------------------
constexpr int kPreR = 16, kPreH = 8, kPreTile = kPreR * kPreH;

__device__ __forceinline__ void pre_tile(int S, int H, int& b, int& r0, int& h0) {
  const int nht = (H + kPreH - 1) / kPreH, nrt = (S + kPreR - 1) / kPreR;
  const int t = blockIdx.x;
  h0 = (t % nht) * kPreH;
  r0 = ((t / nht) % nrt) * kPreR;
  b = t / (nht * nrt);
}

template <int D>
__global__ __launch_bounds__(256) void bwd_pre_bf16_kernel(const bf16* o, const bf16* dO, const float* lse,
                                                           float* ndelta, float* nlse_s, int B, int S, int H) {
  constexpr int TPR = D / 8;      // threads per (row, head)
  constexpr int RPP = 256 / TPR;  // (row, head) pairs per pass
  constexpr int NP = kPreTile / RPP;
  __shared__ float sums[kPreTile];
  int b, r0, h0;
  pre_tile(S, H, b, r0, h0);
  const int c = (threadIdx.x % TPR) * 8;
  float s[NP];
#pragma unroll
  for (int k = 0; k < NP; ++k) {
    const int q = k * RPP + threadIdx.x / TPR, r = r0 + q / kPreH, h = h0 + q % kPreH;
    s[k] = 0.f;
    if (r < S && h < H) {
      const long long row = ((long long)b * S + r) * H + h;
      const bf16x8 a = *(const bf16x8*)(o + row * D + c);
      const bf16x8 g = *(const bf16x8*)(dO + row * D + c);
#pragma unroll
      for (int e = 0; e < 8; ++e) s[k] = fmaf((float)a[e], (float)g[e], s[k]);
    }
  }
#pragma unroll
  for (int k = 0; k < NP; ++k) {
    for (int off = TPR / 2; off > 0; off >>= 1) s[k] += __shfl_xor(s[k], off, 64);
    if (threadIdx.x % TPR == 0) sums[k * RPP + threadIdx.x / TPR] = s[k];
  }
  __syncthreads();
  if (threadIdx.x < kPreTile) {
    const int r = r0 + threadIdx.x % kPreR, h = h0 + threadIdx.x / kPreR;
    if (r < S && h < H) {
      const long long idx = ((long long)b * H + h) * S + r;
      ndelta[idx] = -sums[(threadIdx.x % kPreR) * kPreH + threadIdx.x / kPreR];
      nlse_s[idx] = -lse[idx] * sqrtf((float)D);  // lse / scale: units of q.k
    }
  }
}

template <int D>
__global__ __launch_bounds__(256) void bwd_pre_f32_kernel(const float* o, const float* dO, float* delta,
                                                          int B, int S, int H) {
  constexpr int TPR = D / 4;
  constexpr int RPP = 256 / TPR;
  constexpr int NP = kPreTile / RPP;
  __shared__ float sums[kPreTile];
  int b, r0, h0;
  pre_tile(S, H, b, r0, h0);
  const int c = (threadIdx.x % TPR) * 4;
  float s[NP];
#pragma unroll
  for (int k = 0; k < NP; ++k) {
    const int q = k * RPP + threadIdx.x / TPR, r = r0 + q / kPreH, h = h0 + q % kPreH;
    s[k] = 0.f;
    if (r < S && h < H) {
      const long long row = ((long long)b * S + r) * H + h;
      const f32x4 a = *(const f32x4*)(o + row * D + c);
      const f32x4 g = *(const f32x4*)(dO + row * D + c);
#pragma unroll
      for (int e = 0; e < 4; ++e) s[k] = fmaf(a[e], g[e], s[k]);
    }
  }
#pragma unroll
  for (int k = 0; k < NP; ++k) {
    for (int off = TPR / 2; off > 0; off >>= 1) s[k] += __shfl_xor(s[k], off, 64);
    if (threadIdx.x % TPR == 0) sums[k * RPP + threadIdx.x / TPR] = s[k];
  }
  __syncthreads();
  if (threadIdx.x < kPreTile) {
    const int r = r0 + threadIdx.x % kPreR, h = h0 + threadIdx.x / kPreR;
    if (r < S && h < H) delta[((long long)b * H + h) * S + r] = sums[(threadIdx.x % kPreR) * kPreH + threadIdx.x / kPreR];
  }
}

// Adds a workgroup's dK (DK) or dV contribution (lanes over keys, accumulated transposed:
// register 4 gg + e of product tile dt holds d = 32 dt + 8 gg + 4 hi + e) into the float32
// gradient of the block (its home rows); dK carries the 1/sqrt(D).  The block's first
// contribution is written, not added; its last goes out in bf16.  The sums are formed in
// the accumulators, every carried value loaded before the first store.
template <int NDT, bool DK>
__device__ __forceinline__ void dkdv_epilogue(const BwdStep& p, int slot, int b, int h, int key_in_blk, int hi,
                                                   f32x16 (&acc)[NDT]) {
  constexpr int D = 32 * NDT;
  const int rs = p.H * D;
  const long long grow = (long long)b * p.dkv_bstride + (long long)(p.dkv_row0[slot] + key_in_blk) * rs + h * D;
  const int kf = p.dkv_flags[slot];
  float* g32 = DK ? p.dk : p.dv;
  const float sc = DK ? p.scale : 1.f;
  if (kf & kFirst) {
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[dt][i] = DK ? 0.f + acc[dt][i] * sc : 0.f + acc[dt][i];
  } else {
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int gg = 0; gg < 4; ++gg) {
        const int d = 32 * dt + 8 * gg + 4 * hi;
        const f32x4 c4 = *(const f32x4*)(g32 + grow + d);
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[dt][4 * gg + e] = DK ? c4[e] + acc[dt][4 * gg + e] * sc : c4[e] + acc[dt][4 * gg + e];
      }
  }
  if (kf & kLast) {
    bf16* o16 = (bf16*)(DK ? p.dk_out : p.dv_out);
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int gg = 0; gg < 4; ++gg) {
        const int d = 32 * dt + 8 * gg + 4 * hi;
        const f32x16& a = acc[dt];
        *(u32x2*)(o16 + grow + d) = u32x2{pack_bf16x2(a[4 * gg], a[4 * gg + 1]), pack_bf16x2(a[4 * gg + 2], a[4 * gg + 3])};
      }
  } else {
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int gg = 0; gg < 4; ++gg) {
        const int d = 32 * dt + 8 * gg + 4 * hi;
        const f32x16& a = acc[dt];
        *(f32x4*)(g32 + grow + d) = f32x4{a[4 * gg], a[4 * gg + 1], a[4 * gg + 2], a[4 * gg + 3]};
      }
  }
}

// =====================================================================================
// bf16 dK/dV kernel (D = 64; D = 128 runs the split kernel below, whose waves hold the
// same products): 4 waves x 32 keys = 128 keys per workgroup; loops over 32-query tiles
// of the host's block.  Per wave, lanes run over the wave's keys:
//   S' = Q K^T - lse sqrt(D)   [query x key] (A = Q rows from LDS with row bits 2 and 3
//        swapped, B = K of the wave's keys in registers, as stored: the products are
//        exact in float32; the accumulator starts at -lse sqrt(D) of its query)
//   P  = exp2(S' log2e / sqrt(D))  (the scale in float32)       (masked -> 0)
//   dP = dO V^T - Delta   (A = dO rows, B = V in registers; starts at -Delta)
//   dS = P * dP
//   dV^T += dO^T P        (A = dO^T by LDS transpose read, B = P)
//   dK^T += Q^T dS        (A = Q^T by LDS transpose read, B = dS)
// Q and dO tiles (XOR-swizzled rows) and the tile's lse*log2e and Delta are filled by
// direct-to-LDS buffer loads into a ring of three buffers (48 KB for D = 128, so every
// LDS address fits the reads' immediate offsets).  The loop is software pipelined: while
// tile t's P and dS are formed on the vector ALUs and its dV, dK products run, the S' and
// dP products of tile t+1 are issued and tile t+2 streams in.
// =====================================================================================
constexpr int kKB = 128, kQB = 32, kBT = 256;

template <int D>
__global__ __launch_bounds__(kBT, 1) void bwd_dkdv_bf16_kernel(const BwdStep p) {
  constexpr int NKK = D / 16, NDT = D / 32, CPR = D / 8;
  constexpr int ROWS_PER_LOAD = 64 / CPR, LOADS = kQB / 4 / ROWS_PER_LOAD;
  static_assert(LOADS >= 1, "each wave fills at least one 1 KB row group");
  // one LDS object per buffer, so that reads of one are known not to alias the
  // direct-to-LDS loads in flight into another (else the compiler waits for them)
  __shared__ __attribute__((aligned(1024))) bf16 sQ0[kQB * D];
  __shared__ __attribute__((aligned(1024))) bf16 sQ1[kQB * D];
  __shared__ __attribute__((aligned(1024))) bf16 sQ2[kQB * D];
  __shared__ __attribute__((aligned(1024))) bf16 sO0[kQB * D];  // dO tiles
  __shared__ __attribute__((aligned(1024))) bf16 sO1[kQB * D];
  __shared__ __attribute__((aligned(1024))) bf16 sO2[kQB * D];
  // lse * log2e and Delta: 64 floats each, as a one-wave 4-byte load writes 256 bytes
  // (lanes past the tile read zero)
  __shared__ __attribute__((aligned(256))) float sL0[64];  // -lse sqrt(D)
  __shared__ __attribute__((aligned(256))) float sL1[64];
  __shared__ __attribute__((aligned(256))) float sL2[64];
  __shared__ __attribute__((aligned(256))) float sD0[64];  // -Delta
  __shared__ __attribute__((aligned(256))) float sD1[64];
  __shared__ __attribute__((aligned(256))) float sD2[64];
  auto pick = [](auto Bc, auto* a, auto* b, auto* c) __attribute__((always_inline)) {
    constexpr int B = decltype(Bc)::value % 3;
    if constexpr (B == 0) return a; else if constexpr (B == 1) return b; else return c;
  };

  const int n_kt = p.c / kKB;
  const int BH = p.B * p.H;
  const int total = p.n_slots * BH * n_kt;
  const int Lid = xcd_swizzle(blockIdx.x, total);
  const int grp = Lid / n_kt, kt = Lid % n_kt;
  const int slot = grp / BH, bh = grp % BH;
  const int b = bh / p.H, h = bh % p.H;
  const StepHost hs = p.host[slot];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, l32 = lane & 31, hi = lane >> 5;
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);  // uniform: LDS destinations in scalar registers
  const int rs = p.H * D;
  const float sl2 = p.scale * kLog2e;

  const int key_in_blk = kt * kKB + wave * 32 + l32;  // this lane's key (B-operand column)
  const int kpos = hs.k_pos0 + key_in_blk;
  const bf16* krow = (const bf16*)hs.k + (long long)b * hs.kv_bstride + (long long)key_in_blk * rs + h * D;
  const bf16* vrow = (const bf16*)hs.v + (long long)b * hs.kv_bstride + (long long)key_in_blk * rs + h * D;
  // forwarding: the workgroup writes the rows of its 128 keys, as loaded, into the next
  // host's receive slot for the next ring step (layout [B, c, H, D])
  const int fto = p.fwd.to[slot] - 1;  // destination slot, or -1
  bf16* fkrow = nullptr;
  bf16* fvrow = nullptr;
  if (fto >= 0 && p.fwd.k0 != nullptr && p.fwd.v0 != nullptr) {
    const long long off = (long long)fto * p.fwd.blk_bytes + 2 * (((long long)b * p.c + key_in_blk) * rs + h * D);
    fkrow = (bf16*)((char*)p.fwd.k0 + off);
    fvrow = (bf16*)((char*)p.fwd.v0 + off);
  }
  bf16x8 kreg[NKK], vreg[NKK];
#pragma unroll
  for (int kk = 0; kk < NKK; ++kk) {
    const bf16x8 kx = *(const bf16x8*)(krow + 16 * kk + 8 * hi);
    vreg[kk] = *(const bf16x8*)(vrow + 16 * kk + 8 * hi);
    if (fkrow) {
      *(bf16x8*)(fkrow + 16 * kk + 8 * hi) = kx;
      *(bf16x8*)(fvrow + 16 * kk + 8 * hi) = vreg[kk];
    }
    kreg[kk] = kx;
  }
  f32x16 dkacc[NDT], dvacc[NDT];
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
    for (int i = 0; i < 16; ++i) dkacc[dt][i] = dvacc[dt][i] = 0.f;

  // query tiles with at least one query that sees a key of this workgroup; from
  // qt_free on every query sees every key (no mask)
  const int wg_first_k = hs.k_pos0 + kt * kKB;
  const int n_qtiles = p.c / kQB;
  int qt0 = 0, qt_free = 0;
  if (p.causal) {
    const int rel = wg_first_k - hs.q_pos0;
    qt0 = rel <= 0 ? 0 : min(n_qtiles, rel / kQB);
    const int rel_last = wg_first_k + kKB - 1 - hs.q_pos0;  // last key's offset in the q block
    qt_free = rel_last < 0 ? 0 : min(n_qtiles, (rel_last + kQB - 1) / kQB);
    qt_free = max(qt_free, qt0);
  }

  const bf16* qbase = (const bf16*)p.q + (long long)b * p.q_bstride + h * D;
  const bf16* obase = (const bf16*)p.dO + (long long)b * p.q_bstride + h * D;
  const long long lrow0 = (long long)bh * p.Sq + hs.q_row0;
  constexpr int RPW = kQB / 4;  // tile rows each wave fills
  int goff[LOADS];
#pragma unroll
  for (int j = 0; j < LOADS; ++j) {
    const int r = wave * RPW + j * ROWS_PER_LOAD + lane / CPR;
    goff[j] = 2 * (r * rs + 8 * ((lane % CPR) ^ swz<D>(r)));
  }
  auto load_tile = [&](int qt, auto Bc) __attribute__((always_inline)) {
    const long long t0 = (long long)(hs.q_row0 + qt * kQB) * rs;
#pragma unroll
    for (int j = 0; j < LOADS; ++j) {
      buffer_load_lds16(qbase + t0, kQB * rs * 2, pick(Bc, sQ0, sQ1, sQ2) + (wave_u * RPW + j * ROWS_PER_LOAD) * D,
                        goff[j]);
      buffer_load_lds16(obase + t0, kQB * rs * 2, pick(Bc, sO0, sO1, sO2) + (wave_u * RPW + j * ROWS_PER_LOAD) * D,
                        goff[j]);
    }
    if (wave_u == 0) buffer_load_lds4(p.lse + lrow0 + qt * kQB, kQB * 4, pick(Bc, sL0, sL1, sL2), 4 * lane);
    if (wave_u == 1) buffer_load_lds4(p.delta + lrow0 + qt * kQB, kQB * 4, pick(Bc, sD0, sD1, sD2), 4 * lane);
  };
  const int qrow = swap_bits23(l32);
  int roff[NKK];
#pragma unroll
  for (int kk = 0; kk < NKK; ++kk) roff[kk] = qrow * D + 8 * ((2 * kk + hi) ^ swz<D>(qrow));
  const int g16 = lane >> 4, li = lane & 15;
  int toff[2][NDT];
#pragma unroll
  for (int r = 0; r < 2; ++r)
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) {
      const int row = 8 * hi + 4 * r + (li >> 2);
      const int d = 32 * dt + 16 * (g16 & 1) + 4 * (li & 3);
      toff[r][dt] = row * D + 8 * ((d >> 3) ^ swz<D>(row)) + (d & 7);
    }

  // accumulator starts of S' (-lse sqrt(D)) and dP (-Delta), stored negated by the
  // preprocess kernel, of a tile: register 8 g + e of a lane holds query 16 g + 8 hi + e
  auto inits = [&](auto Bc, f32x16& si, f32x16& di) __attribute__((always_inline)) {
    const float* sl = pick(Bc, sL0, sL1, sL2);
    const float* sd = pick(Bc, sD0, sD1, sD2);
#pragma unroll
    for (int g = 0; g < 2; ++g) {
      const int q0 = 16 * g + 8 * hi;
      const f32x4 la = *(const f32x4*)&sl[q0], lb = *(const f32x4*)&sl[q0 + 4];
      const f32x4 da = *(const f32x4*)&sd[q0], db = *(const f32x4*)&sd[q0 + 4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        si[8 * g + e] = la[e];
        si[8 * g + 4 + e] = lb[e];
        di[8 * g + e] = da[e];
        di[8 * g + 4 + e] = db[e];
      }
    }
  };
  // P and dS (bf16 pairs) of group g (16 queries) of a tile, pair u of the group's 4
  auto unit = [&](auto Mc, const f32x16& sc, const f32x16& dpc, int qpos0, int g, int u, uint32_t& w1,
                  uint32_t& w2) __attribute__((always_inline)) {
    constexpr bool MASK = decltype(Mc)::value;
    float pv[2], dsv[2];
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      const int r = 8 * g + 2 * u + e;
      float pr = fast_exp2(sc[r] * sl2);
      if (MASK && kpos > qpos0 + 16 * g + 8 * hi + 2 * u + e) pr = 0.f;
      pv[e] = pr;
      dsv[e] = pr * dpc[r];
    }
    w1 = pack_bf16x2(pv[0], pv[1]);
    w2 = pack_bf16x2(dsv[0], dsv[1]);
  };

  // One tile t (buffer Bc): loads of tile t+2 (buffer Bc+2), the S'/dP products of tile t+1
  // (buffer Bc+1; Nc: it exists) and, for tile t, P and dS in two groups of 16 queries, each
  // followed by its dV and dK products; then the wait for tile t+2 and the barrier that frees
  // buffer Bc.  For D = 128 the region is laid out by hand in 20 fenced steps: step s issues
  // S'/dP product s (s < 16; S' and dP alternate, so consecutive products are independent),
  // the dV/dK product s - 4 (s >= 4; group (s - 4) / 8) and the vector work of one pair unit
  // (group 0 at steps 0..3, group 1 at steps 4, 6, 8, 10), with LDS operand reads two steps
  // ahead.  Other head dims run the same work in program order.
  auto tile = [&](auto Bc, auto Mc, auto Nc, int qt, f32x16& s_cur, f32x16& dp_cur) __attribute__((always_inline)) {
    constexpr int B = decltype(Bc)::value;
    constexpr bool NX = decltype(Nc)::value;
    using Bn = std::integral_constant<int, (B + 1) % 3>;
    using Bl = std::integral_constant<int, (B + 2) % 3>;
    if (qt + 2 < n_qtiles) load_tile(qt + 2, Bl{});
    const bf16* qn = pick(Bn{}, sQ0, sQ1, sQ2);  // next tile: row reads
    const bf16* on = pick(Bn{}, sO0, sO1, sO2);
    const bf16* qc = pick(Bc, sQ0, sQ1, sQ2);    // this tile: transpose reads
    const bf16* oc = pick(Bc, sO0, sO1, sO2);
    const int qpos0 = hs.q_pos0 + qt * kQB;
    f32x16 s_nx, dp_nx;
    if constexpr (NX) inits(Bn{}, s_nx, dp_nx);
    if constexpr (D == 128) {
      bf16x8 aop[16], top[16];
      uint32_t wp[2][4], ws[2][4];
      bf16x8 pb[2], dsb[2];
      constexpr int kPF = 2;
      auto read_a = [&](auto Sc) __attribute__((always_inline)) {  // product s: kk = s / 2, dP if odd
        constexpr int S = decltype(Sc)::value;
        aop[S] = *(const bf16x8*)(((S & 1) ? on : qn) + roff[S / 2]);
      };
      auto read_t = [&](auto Qc) __attribute__((always_inline)) {  // product q: group q / 8, dt (q % 8) / 2
        constexpr int Q = decltype(Qc)::value, g = Q / 8, dt = (Q % 8) / 2;
        const bf16* src = (Q & 1) ? qc : oc;
        const bf16x4 lo = lds_read_tr16(src + 16 * g * D + toff[0][dt]);
        const bf16x4 up = lds_read_tr16(src + 16 * g * D + toff[1][dt]);
        top[Q] = bf16x8{lo[0], lo[1], lo[2], lo[3], up[0], up[1], up[2], up[3]};
      };
      if constexpr (NX) static_for<0, kPF>([&](auto Sc) __attribute__((always_inline)) { read_a(Sc); });
      static_for<0, 20>([&](auto Sc) __attribute__((always_inline)) {
        constexpr int S = decltype(Sc)::value;
        if constexpr (NX && S + kPF < 16) read_a(std::integral_constant<int, S + kPF>{});
        if constexpr (S + kPF >= 4 && S + kPF < 20) read_t(std::integral_constant<int, S + kPF - 4>{});
        if constexpr (NX && S < 16) {
          if constexpr (S & 1)
            dp_nx = mfma32(aop[S], vreg[S / 2], dp_nx);
          else
            s_nx = mfma32(aop[S], kreg[S / 2], s_nx);
        }
        if constexpr (S >= 4) {
          constexpr int q = S - 4, g = q / 8, dt = (q % 8) / 2;
          if constexpr (q % 8 == 0) {
            pb[g] = __builtin_bit_cast(bf16x8, u32x4{wp[g][0], wp[g][1], wp[g][2], wp[g][3]});
            dsb[g] = __builtin_bit_cast(bf16x8, u32x4{ws[g][0], ws[g][1], ws[g][2], ws[g][3]});
          }
          if constexpr (q & 1)
            dkacc[dt] = mfma32(top[q], dsb[g], dkacc[dt]);
          else
            dvacc[dt] = mfma32(top[q], pb[g], dvacc[dt]);
        }
        if constexpr (S < 4) {
          unit(Mc, s_cur, dp_cur, qpos0, 0, S, wp[0][S], ws[0][S]);
        } else if constexpr (S < 12 && S % 2 == 0) {
          unit(Mc, s_cur, dp_cur, qpos0, 1, (S - 4) / 2, wp[1][(S - 4) / 2], ws[1][(S - 4) / 2]);
        }
        __builtin_amdgcn_sched_barrier(0);
      });
    } else {
      if constexpr (NX) {
#pragma unroll
        for (int kk = 0; kk < NKK; ++kk) {
          s_nx = mfma32(*(const bf16x8*)(qn + roff[kk]), kreg[kk], s_nx);
          dp_nx = mfma32(*(const bf16x8*)(on + roff[kk]), vreg[kk], dp_nx);
        }
      }
#pragma unroll
      for (int g = 0; g < 2; ++g) {
        uint32_t wp[4], ws[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) unit(Mc, s_cur, dp_cur, qpos0, g, u, wp[u], ws[u]);
        const bf16x8 pbg = __builtin_bit_cast(bf16x8, u32x4{wp[0], wp[1], wp[2], wp[3]});
        const bf16x8 dsg = __builtin_bit_cast(bf16x8, u32x4{ws[0], ws[1], ws[2], ws[3]});
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) {
          const bf16x4 olo = lds_read_tr16(oc + 16 * g * D + toff[0][dt]);
          const bf16x4 oup = lds_read_tr16(oc + 16 * g * D + toff[1][dt]);
          dvacc[dt] = mfma32(bf16x8{olo[0], olo[1], olo[2], olo[3], oup[0], oup[1], oup[2], oup[3]}, pbg, dvacc[dt]);
          const bf16x4 qlo = lds_read_tr16(qc + 16 * g * D + toff[0][dt]);
          const bf16x4 qup = lds_read_tr16(qc + 16 * g * D + toff[1][dt]);
          dkacc[dt] = mfma32(bf16x8{qlo[0], qlo[1], qlo[2], qlo[3], qup[0], qup[1], qup[2], qup[3]}, dsg, dkacc[dt]);
        }
      }
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // tile t+2 landed
    __syncthreads();                                   // and buffer Bc is free again
    if constexpr (NX) {
      s_cur = s_nx;
      dp_cur = dp_nx;
    }
  };

  if (qt0 < n_qtiles) {
    load_tile(qt0, std::integral_constant<int, 0>{});
    if (qt0 + 1 < n_qtiles) load_tile(qt0 + 1, std::integral_constant<int, 1>{});
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    f32x16 s_cur, dp_cur;  // S' and dP of the tile being processed
    inits(std::integral_constant<int, 0>{}, s_cur, dp_cur);
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) {
      s_cur = mfma32(*(const bf16x8*)(sQ0 + roff[kk]), kreg[kk], s_cur);
      dp_cur = mfma32(*(const bf16x8*)(sO0 + roff[kk]), vreg[kk], dp_cur);
    }
    // buffer of tile qt is (qt - qt0) % 3, known at compile time in a loop unrolled by 3;
    // tiles [a, e) all have a successor
    using I0 = std::integral_constant<int, 0>;
    using I1 = std::integral_constant<int, 1>;
    using I2 = std::integral_constant<int, 2>;
    auto run = [&](auto Mc, int a, int e) __attribute__((always_inline)) {
      int it = a;
      if (it < e && (it - qt0) % 3 == 1) tile(I1{}, Mc, std::true_type{}, it++, s_cur, dp_cur);
      if (it < e && (it - qt0) % 3 == 2) tile(I2{}, Mc, std::true_type{}, it++, s_cur, dp_cur);
      for (; it + 2 < e; it += 3) {
        tile(I0{}, Mc, std::true_type{}, it, s_cur, dp_cur);
        tile(I1{}, Mc, std::true_type{}, it + 1, s_cur, dp_cur);
        tile(I2{}, Mc, std::true_type{}, it + 2, s_cur, dp_cur);
      }
      if (it < e) tile(I0{}, Mc, std::true_type{}, it++, s_cur, dp_cur);
      if (it < e) tile(I1{}, Mc, std::true_type{}, it++, s_cur, dp_cur);
    };
    const int ql = n_qtiles - 1;
    const int split = max(qt0, min(qt_free, ql));  // masked tiles first
    run(std::true_type{}, qt0, split);
    run(std::false_type{}, split, ql);
    // last tile: no successor
    const int ph = (ql - qt0) % 3;
    auto last = [&](auto Mc) __attribute__((always_inline)) {
      if (ph == 0) tile(I0{}, Mc, std::false_type{}, ql, s_cur, dp_cur);
      else if (ph == 1) tile(I1{}, Mc, std::false_type{}, ql, s_cur, dp_cur);
      else tile(I2{}, Mc, std::false_type{}, ql, s_cur, dp_cur);
    };
    if (ql < qt_free) last(std::true_type{}); else last(std::false_type{});
  }

  dkdv_epilogue<NDT, true>(p, slot, b, h, key_in_blk, hi, dkacc);
  dkdv_epilogue<NDT, false>(p, slot, b, h, key_in_blk, hi, dvacc);
}

// =====================================================================================
// bf16 dK/dV kernel for D = 128 with the work of each 32-key column split over three
// waves: 12 waves and 128 keys per workgroup, three waves on every SIMD.
//   row wave (w < 4, column w): holds K and V of keys 32 w .. 32 w + 31 in registers and,
//     per 32-query tile, runs the products contracted over D and the vector work
//       S' = Q K^T - lse sqrt(D),  dP = dO V^T - Delta,
//       P = exp2(S' log2e / sqrt(D)) (masked -> 0),  dS = P * dP,
//     and stores P and dS, packed to bf16 in the lane order of a B operand, to LDS;
//   dV wave (w = 4 + column), one tile later:  dV^T += dO^T P;
//   dK wave (w = 8 + column), one tile later:  dK^T += Q^T dS
//     (A operands by LDS transpose reads; each of the two holds 64 accumulator registers).
// At 162 registers a wave, three waves share each SIMD: the row wave is mostly vector
// work, the other two only matrix products and LDS reads, so each covers the others'
// waits for LDS and for the barrier (with one wave per SIMD, as in the kernel above, those
// waits leave the matrix core idle).  The operands and their order of accumulation are
// those of the one-wave kernel, so the results are the same bit for bit.
// Q and dO tiles (XOR-swizzled rows) with the tile's -lse sqrt(D) and -Delta stream by
// direct-to-LDS loads (waves 0-7, 4 rows each) into a ring of four buffers: in the region
// of tile t the row waves read tile t+1, the dV and dK waves tile t-1, and tile t+2 streams
// in.  The packed P and dS pass through two exchange buffers; one barrier per tile.
// =====================================================================================
constexpr int kPT = 768;

__global__ __launch_bounds__(kPT) void bwd_dkdv_split_kernel(const BwdStep p) {
  constexpr int D = 128, NKK = D / 16, NDT = D / 32, CPR = D / 8, ROWS_PER_LOAD = 64 / CPR;
  static_assert(kQB == 8 * ROWS_PER_LOAD, "waves 0-7 fill 4 rows of a tile each");
  // Q tiles 0-3, then dO tiles 0-3, in one LDS object, so that every read of a ring buffer
  // is one lane offset plus an immediate; filled by direct-to-LDS loads the compiler does
  // not track (the region's explicit vmcnt wait and barrier order them)
  __shared__ __attribute__((aligned(1024))) bf16 sQO[8 * kQB * D];
  // -lse sqrt(D) of tiles 0-3, then -Delta: 64 floats each, as a one-wave 4-byte load
  // writes 256 bytes (lanes past the tile read zero)
  __shared__ __attribute__((aligned(1024))) float sLD[8 * 64];
  // packed P and dS of a tile: [column][P of queries 0-15, 16-31, dS of 0-15, 16-31][lane]
  __shared__ __attribute__((aligned(1024))) u32x4 sX0[4 * 4 * 64];
  __shared__ __attribute__((aligned(1024))) u32x4 sX1[4 * 4 * 64];
  auto qt_lds = [&](auto Bc) __attribute__((always_inline)) { return sQO + (decltype(Bc)::value % 4) * kQB * D; };
  auto ot_lds = [&](auto Bc) __attribute__((always_inline)) { return sQO + (4 + decltype(Bc)::value % 4) * kQB * D; };
  auto l_lds = [&](auto Bc) __attribute__((always_inline)) { return sLD + (decltype(Bc)::value % 4) * 64; };
  auto d_lds = [&](auto Bc) __attribute__((always_inline)) { return sLD + (4 + decltype(Bc)::value % 4) * 64; };
  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  using I2 = std::integral_constant<int, 2>;
  using I3 = std::integral_constant<int, 3>;

  const int n_kt = p.c / kKB;
  const int BH = p.B * p.H;
  const int total = p.n_slots * BH * n_kt;
  const int Lid = xcd_swizzle(blockIdx.x, total);
  const int grp = Lid / n_kt, kt = Lid % n_kt;
  const int slot = grp / BH, bh = grp % BH;
  const int b = bh / p.H, h = bh % p.H;
  const StepHost hs = p.host[slot];
  const int tid = threadIdx.x, lane = tid & 63, l32 = lane & 31, hi = lane >> 5;
  const int wave_u = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: LDS destinations in scalar registers
  const int col = wave_u & 3;                                   // the wave's 32-key column
  const int rs = p.H * D;
  const int key_in_blk = kt * kKB + col * 32 + l32;  // this lane's key (B-operand column)

  // query tiles with at least one query that sees a key of this workgroup; from
  // qt_free on every query sees every key (no mask)
  const int wg_first_k = hs.k_pos0 + kt * kKB;
  const int n_qtiles = p.c / kQB;
  int qt0 = 0, qt_free = 0;
  if (p.causal) {
    const int rel = wg_first_k - hs.q_pos0;
    qt0 = rel <= 0 ? 0 : min(n_qtiles, rel / kQB);
    const int rel_last = wg_first_k + kKB - 1 - hs.q_pos0;  // last key's offset in the q block
    qt_free = rel_last < 0 ? 0 : min(n_qtiles, (rel_last + kQB - 1) / kQB);
    qt_free = max(qt_free, qt0);
  }
  const int n = n_qtiles - qt0;  // tiles visited; tile i of the workgroup is query tile qt0 + i

  const bf16* qbase = (const bf16*)p.q + (long long)b * p.q_bstride + h * D;
  const bf16* obase = (const bf16*)p.dO + (long long)b * p.q_bstride + h * D;
  const long long lrow0 = (long long)bh * p.Sq + hs.q_row0;
  const int lrow = (wave_u & 7) * ROWS_PER_LOAD + lane / CPR;  // the tile row this lane fills (waves 0-7)
  const int goff = 2 * (lrow * rs + 8 * ((lane % CPR) ^ swz<D>(lrow)));
  // tile i into ring buffer buf: the Q and dO rows by waves 0-7, -lse sqrt(D) by wave 0,
  // -Delta by wave 1
  auto load_tile = [&](int i, int buf) __attribute__((always_inline)) {
    const int qt = qt0 + i;
    const long long t0 = (long long)(hs.q_row0 + qt * kQB) * rs;
    if (wave_u < 8) {
      dma_lds16(make_rsrc(qbase + t0, kQB * rs * 2), lds_addr(sQO + (buf * kQB + wave_u * ROWS_PER_LOAD) * D), goff);
      dma_lds16(make_rsrc(obase + t0, kQB * rs * 2), lds_addr(sQO + ((4 + buf) * kQB + wave_u * ROWS_PER_LOAD) * D),
                goff);
    }
    if (wave_u == 0) dma_lds4(make_rsrc(p.lse + lrow0 + qt * kQB, kQB * 4), lds_addr(sLD + buf * 64), 4 * lane);
    if (wave_u == 1) dma_lds4(make_rsrc(p.delta + lrow0 + qt * kQB, kQB * 4), lds_addr(sLD + (4 + buf) * 64), 4 * lane);
  };
  // regions [a, e) with the buffer of region i (i % 4) known at compile time
  auto run4 = [&](int a, int e, auto&& f) __attribute__((always_inline)) {
    int i = a;
    if (i < e && (i & 3) == 1) f(I1{}, i++);
    if (i < e && (i & 3) == 2) f(I2{}, i++);
    if (i < e && (i & 3) == 3) f(I3{}, i++);
    for (; i + 3 < e; i += 4) {
      f(I0{}, i);
      f(I1{}, i + 1);
      f(I2{}, i + 2);
      f(I3{}, i + 3);
    }
    if (i < e) f(I0{}, i++);
    if (i < e) f(I1{}, i++);
    if (i < e) f(I2{}, i++);
  };
  auto at = [&](int i, auto&& f) __attribute__((always_inline)) {  // one region, buffer i % 4
    switch (i & 3) {
      case 0: f(I0{}, i); break;
      case 1: f(I1{}, i); break;
      case 2: f(I2{}, i); break;
      default: f(I3{}, i); break;
    }
  };
  auto sync = [&]() __attribute__((always_inline)) {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // this wave's loads of tile i+2 landed
    __syncthreads();                                   // every wave's; the exchange written
  };

  if (n > 0) {
    load_tile(0, 0);
    if (n > 1) load_tile(1, 1);
  }

  if (wave_u < 4) {
    // ---------------------------------------------------------------- row wave
    const int kpos = hs.k_pos0 + key_in_blk;
    const float sl2 = p.scale * kLog2e;
    const bf16* krow = (const bf16*)hs.k + (long long)b * hs.kv_bstride + (long long)key_in_blk * rs + h * D;
    const bf16* vrow = (const bf16*)hs.v + (long long)b * hs.kv_bstride + (long long)key_in_blk * rs + h * D;
    // forwarding: the row waves write the rows of the workgroup's 128 keys, as loaded,
    // into the next host's receive slot for the next ring step (layout [B, c, H, D])
    const int fto = p.fwd.to[slot] - 1;  // destination slot, or -1
    bf16* fkrow = nullptr;
    bf16* fvrow = nullptr;
    if (fto >= 0 && p.fwd.k0 != nullptr && p.fwd.v0 != nullptr) {
      const long long off = (long long)fto * p.fwd.blk_bytes + 2 * (((long long)b * p.c + key_in_blk) * rs + h * D);
      fkrow = (bf16*)((char*)p.fwd.k0 + off);
      fvrow = (bf16*)((char*)p.fwd.v0 + off);
    }
    bf16x8 kreg[NKK], vreg[NKK];
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) {
      const bf16x8 kx = *(const bf16x8*)(krow + 16 * kk + 8 * hi);
      vreg[kk] = *(const bf16x8*)(vrow + 16 * kk + 8 * hi);
      if (fkrow) {
        *(bf16x8*)(fkrow + 16 * kk + 8 * hi) = kx;
        *(bf16x8*)(fvrow + 16 * kk + 8 * hi) = vreg[kk];
      }
      kreg[kk] = kx;
    }
    if (n == 0) return;
    const int qrow = swap_bits23(l32);
    int roff[NKK];
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) roff[kk] = qrow * D + 8 * ((2 * kk + hi) ^ swz<D>(qrow));
    // accumulator starts of S' (-lse sqrt(D)) and dP (-Delta) of a tile: register 8 g + e
    // of a lane holds query 16 g + 8 hi + e
    auto inits = [&](auto Bc, f32x16& si, f32x16& di) __attribute__((always_inline)) {
      const float* sl = l_lds(Bc);
      const float* sd = d_lds(Bc);
#pragma unroll
      for (int g = 0; g < 2; ++g) {
        const int q0 = 16 * g + 8 * hi;
        const f32x4 la = *(const f32x4*)&sl[q0], lb = *(const f32x4*)&sl[q0 + 4];
        const f32x4 da = *(const f32x4*)&sd[q0], db = *(const f32x4*)&sd[q0 + 4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          si[8 * g + e] = la[e];
          si[8 * g + 4 + e] = lb[e];
          di[8 * g + e] = da[e];
          di[8 * g + 4 + e] = db[e];
        }
      }
    };
    // P and dS (bf16 pairs) of group g (16 queries) of a tile, pair u of the group's 4
    auto unit = [&](auto Mc, const f32x16& sc, const f32x16& dpc, int qpos0, int g, int u, uint32_t& w1,
                    uint32_t& w2) __attribute__((always_inline)) {
      constexpr bool MASK = decltype(Mc)::value;
      float pv[2], dsv[2];
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        const int r = 8 * g + 2 * u + e;
        float pr = fast_exp2(sc[r] * sl2);
        if (MASK && kpos > qpos0 + 16 * g + 8 * hi + 2 * u + e) pr = 0.f;
        pv[e] = pr;
        dsv[e] = pr * dpc[r];
      }
      w1 = pack_bf16x2(pv[0], pv[1]);
      w2 = pack_bf16x2(dsv[0], dsv[1]);
    };
    sync();
    f32x16 s_cur, dp_cur;  // S' and dP of the tile whose P and dS are formed next
    inits(I0{}, s_cur, dp_cur);
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) {
      s_cur = mfma32(*(const bf16x8*)(qt_lds(I0{}) + roff[kk]), kreg[kk], s_cur);
      dp_cur = mfma32(*(const bf16x8*)(ot_lds(I0{}) + roff[kk]), vreg[kk], dp_cur);
    }
    // Region of tile i (buffer Bc; Nc: tile i+1 exists): loads of tile i+2, the S'/dP
    // products of tile i+1 in 16 fenced steps (S' and dP alternate; operand reads two
    // steps ahead), and P, dS of tile i, one pair unit at every even step; each group's
    // packed P and dS go to the exchange buffer of tile i once formed.
    auto region = [&](auto Bc, auto Mc, auto Nc, int i) __attribute__((always_inline)) {
      constexpr int B = decltype(Bc)::value;
      constexpr bool NX = decltype(Nc)::value;
      using Bn = std::integral_constant<int, (B + 1) % 4>;
      using Bl = std::integral_constant<int, (B + 2) % 4>;
      if (i + 2 < n) load_tile(i + 2, Bl::value);
      const bf16* qn = qt_lds(Bn{});
      const bf16* on = ot_lds(Bn{});
      u32x4* xw = ((B & 1) ? sX1 : sX0) + col * 4 * 64 + lane;
      const int qpos0 = hs.q_pos0 + (qt0 + i) * kQB;
      f32x16 s_nx, dp_nx;
      if constexpr (NX) inits(Bn{}, s_nx, dp_nx);
      bf16x8 aop[16];
      uint32_t wp[2][4], ws[2][4];
      constexpr int kPF = 2;
      auto read_a = [&](auto Sc) __attribute__((always_inline)) {  // product s: kk = s / 2, dP if odd
        constexpr int S = decltype(Sc)::value;
        aop[S] = *(const bf16x8*)(((S & 1) ? on : qn) + roff[S / 2]);
      };
      if constexpr (NX) static_for<0, kPF>([&](auto Sc) __attribute__((always_inline)) { read_a(Sc); });
      static_for<0, 16>([&](auto Sc) __attribute__((always_inline)) {
        constexpr int S = decltype(Sc)::value;
        if constexpr (NX && S + kPF < 16) read_a(std::integral_constant<int, S + kPF>{});
        if constexpr (NX) {
          if constexpr (S & 1)
            dp_nx = mfma32(aop[S], vreg[S / 2], dp_nx);
          else
            s_nx = mfma32(aop[S], kreg[S / 2], s_nx);
        }
        if constexpr (S % 2 == 0) {
          constexpr int g = S / 8, u = (S % 8) / 2;
          unit(Mc, s_cur, dp_cur, qpos0, g, u, wp[g][u], ws[g][u]);
        }
        if constexpr (S % 8 == 7) {
          constexpr int g = S / 8;
          xw[g * 64] = u32x4{wp[g][0], wp[g][1], wp[g][2], wp[g][3]};
          xw[(2 + g) * 64] = u32x4{ws[g][0], ws[g][1], ws[g][2], ws[g][3]};
        }
        __builtin_amdgcn_sched_barrier(0);
      });
      sync();
      if constexpr (NX) {
        s_cur = s_nx;
        dp_cur = dp_nx;
      }
    };
    // masked tiles first; every tile but the last has a successor
    const int ms = max(0, min(qt_free - qt0, n - 1));
    run4(0, ms, [&](auto Bc, int i) __attribute__((always_inline)) {
      region(Bc, std::true_type{}, std::true_type{}, i);
    });
    run4(ms, n - 1, [&](auto Bc, int i) __attribute__((always_inline)) {
      region(Bc, std::false_type{}, std::true_type{}, i);
    });
    if (qt0 + n - 1 < qt_free)
      at(n - 1, [&](auto Bc, int i) __attribute__((always_inline)) { region(Bc, std::true_type{}, std::false_type{}, i); });
    else
      at(n - 1, [&](auto Bc, int i) __attribute__((always_inline)) { region(Bc, std::false_type{}, std::false_type{}, i); });
    return;
  }

  // ------------------------------------------------------------------ column waves
  // waves 4-7 accumulate dV, waves 8-11 dK, of the column
  auto column = [&](auto Kc) __attribute__((always_inline)) {
    constexpr bool DK = decltype(Kc)::value;
    f32x16 acc[NDT];
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[dt][i] = 0.f;
    if (n > 0) {
      const int g16 = lane >> 4, li = lane & 15;
      int toff[2][NDT];
#pragma unroll
      for (int r = 0; r < 2; ++r)
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) {
          const int row = 8 * hi + 4 * r + (li >> 2);
          const int d = 32 * dt + 16 * (g16 & 1) + 4 * (li & 3);
          toff[r][dt] = row * D + 8 * ((d >> 3) ^ swz<D>(row)) + (d & 7);
        }
      sync();
      for (int i = 0; i <= n; ++i) {
        if (i + 2 < n) load_tile(i + 2, (i + 2) & 3);
        if (i >= 1) {
          const u32x4* xr = (((i - 1) & 1) ? sX1 : sX0) + col * 4 * 64 + lane + (DK ? 128 : 0);
          const bf16x8 bop[2] = {__builtin_bit_cast(bf16x8, xr[0]), __builtin_bit_cast(bf16x8, xr[64])};
          const bf16* src = sQO + ((DK ? 0 : 4) + ((i - 1) & 3)) * kQB * D;
          bf16x8 top[8];
          constexpr int kPF = 2;
          auto read_t = [&](auto Qc) __attribute__((always_inline)) {  // product q: group q / 4, dt q % 4
            constexpr int Q = decltype(Qc)::value, g = Q / 4, dt = Q % 4;
            const bf16x4 lo = lds_read_tr16(src + 16 * g * D + toff[0][dt]);
            const bf16x4 up = lds_read_tr16(src + 16 * g * D + toff[1][dt]);
            top[Q] = bf16x8{lo[0], lo[1], lo[2], lo[3], up[0], up[1], up[2], up[3]};
          };
          static_for<0, kPF>([&](auto Qc) __attribute__((always_inline)) { read_t(Qc); });
          static_for<0, 8>([&](auto Qc) __attribute__((always_inline)) {
            constexpr int Q = decltype(Qc)::value, g = Q / 4, dt = Q % 4;
            if constexpr (Q + kPF < 8) read_t(std::integral_constant<int, Q + kPF>{});
            acc[dt] = mfma32(top[Q], bop[g], acc[dt]);
            __builtin_amdgcn_sched_barrier(0);
          });
        }
        if (i < n) sync();
      }
    }
    dkdv_epilogue<NDT, DK>(p, slot, b, h, key_in_blk, hi, acc);
  };
  if (wave_u >= 8) column(std::true_type{});
  else column(std::false_type{});
}

// bf16 dQ kernel: 4 waves x 32 queries = 128 queries per workgroup; loops over 64-key
// tiles of the block.  Per wave, lanes run over queries:
//   S^T  = K Q^T            (A = K rows from LDS, B = Q in registers)
//   dP^T = V dO^T - Delta   (A = V rows, B = dO in registers; the accumulator starts at
//                            -Delta of the lane's query, so the subtraction is free)
//   P^T  = exp2(S^T log2e/sqrt(D) - lse log2e),  dS^T = P^T * dP^T   (masked -> 0), the
//          scale applied in float32
//   dQ^T += K^T dS^T        (A = K^T by LDS transpose read, B = dS^T)
// K and V tiles are filled by direct-to-LDS buffer loads into XOR-swizzled unpadded rows
// (see swz), double buffered: tile it+1 streams in while tile it is processed.
// =====================================================================================
constexpr int kQQ = 128, kKK = 64;

template <int D>
__global__ __launch_bounds__(kBT, 2) void bwd_dq_bf16_kernel(const BwdStep p) {
  constexpr int NKK = D / 16, NDT = D / 32, CPR = D / 8;
  constexpr int ROWS_PER_LOAD = 64 / CPR, LOADS = kKK / 4 / ROWS_PER_LOAD;
  // one LDS object per buffer (see the dK/dV kernel)
  // one LDS array (K0, K1, V0, V1 tiles), filled by direct-to-LDS loads the compiler does
  // not track (each tile's loads are waited for before the barrier that ends the tile), so
  // that every read address is one register plus an immediate offset
  __shared__ __attribute__((aligned(1024))) bf16 lds[4 * kKK * D];
  bf16* const sK0 = lds;
  bf16* const sK1 = lds + kKK * D;
  bf16* const sV0 = lds + 2 * kKK * D;
  bf16* const sV1 = lds + 3 * kKK * D;
  auto pick = [](auto Bc, auto* a, auto* b) __attribute__((always_inline)) {
    if constexpr (decltype(Bc)::value == 0) return a; else return b;
  };

  const int n_qt = p.c / kQQ;
  const int BH = p.B * p.H;
  const int total = p.n_slots * BH * n_qt;
  const int Lid = xcd_swizzle(blockIdx.x, total);
  const int grp = Lid / n_qt;
  const int qt = n_qt - 1 - (Lid % n_qt);
  const int slot = grp / BH, bh = grp % BH;
  const int b = bh / p.H, h = bh % p.H;
  const StepHost hs = p.host[slot];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, l32 = lane & 31, hi = lane >> 5;
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);  // uniform: LDS destinations in scalar registers
  const int rs = p.H * D;

  const int qr = hs.q_row0 + qt * kQQ + wave * 32 + l32;
  const int qpos = hs.q_pos0 + qt * kQQ + wave * 32 + l32;
  const int tile_first_q = hs.q_pos0 + qt * kQQ;
  const long long lrow = (long long)bh * p.Sq + qr;
  const float nlse_s = p.lse[lrow];  // -lse sqrt(D) (written by the preprocess kernel)
  const float ndlt = p.delta[lrow];  // -Delta

  bf16x8 qreg[NKK], oreg[NKK];
  {
    const long long off = (long long)b * p.q_bstride + (long long)qr * rs + h * D + 8 * hi;
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) {
      qreg[kk] = *(const bf16x8*)((const bf16*)p.q + off + 16 * kk);
      oreg[kk] = *(const bf16x8*)((const bf16*)p.dO + off + 16 * kk);
    }
    // consume the loads here: otherwise the compiler, unsure whether they are still in
    // flight, waits on the load counter inside the loop, where it also counts the
    // prefetch of the next tile
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) asm volatile("" ::"v"(qreg[kk]), "v"(oreg[kk]));
  }
  f32x16 dqacc[NDT];
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
    for (int i = 0; i < 16; ++i) dqacc[dt][i] = 0.f;

  int nt = p.c / kKK, n_full = nt;
  if (p.causal) {
    const int vis = tile_first_q + kQQ - hs.k_pos0;
    nt = min(nt, max(0, (vis + kKK - 1) / kKK));
    n_full = min(nt, max(0, (tile_first_q - hs.k_pos0 + 1) / kKK));
  }
  const bf16* kbase = (const bf16*)hs.k + (long long)b * hs.kv_bstride + h * D;
  const bf16* vbase = (const bf16*)hs.v + (long long)b * hs.kv_bstride + h * D;

  // direct-to-LDS staging: load j of wave w fills rows j * 4 ROWS_PER_LOAD + w ROWS_PER_LOAD +
  // lane / CPR.  The swizzle of those rows does not depend on j, so all loads of a lane read
  // at one byte offset goff plus a wave-uniform j * 8 ROWS_PER_LOAD * rs bytes.
  static_assert(16 == LOADS * ROWS_PER_LOAD, "each wave fills LOADS row groups");
  const int goff = 2 * ((wave * ROWS_PER_LOAD + lane / CPR) * rs +
                        8 * ((lane % CPR) ^ swz<D>(wave * ROWS_PER_LOAD + lane / CPR)));
  auto load_tile = [&](int it, auto Bc) __attribute__((always_inline)) {
    const long long t0 = (long long)it * kKK * rs;
    const __amdgpu_buffer_rsrc_t rk = make_rsrc(kbase + t0, kKK * rs * 2), rv = make_rsrc(vbase + t0, kKK * rs * 2);
#pragma unroll
    for (int j = 0; j < LOADS; ++j) {
      const int row = (j * 4 + wave_u) * ROWS_PER_LOAD, so = j * 8 * ROWS_PER_LOAD * rs;
      dma_lds16_so(rk, lds_addr(pick(Bc, sK0, sK1) + row * D), goff, so);
      dma_lds16_so(rv, lds_addr(pick(Bc, sV0, sV1) + row * D), goff, so);
    }
  };
  // row reads (A operand, rows 32 mt + swap_bits23(l32)) and transpose reads of the tiles
  const int krow = swap_bits23(l32);
  int roff[NKK];
#pragma unroll
  for (int kk = 0; kk < NKK; ++kk) roff[kk] = krow * D + 8 * ((2 * kk + hi) ^ swz<D>(krow));
  const int g16 = lane >> 4, li = lane & 15;
  int toff[2][NDT];
#pragma unroll
  for (int r = 0; r < 2; ++r)
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) {
      const int row = 8 * hi + 4 * r + (li >> 2);
      const int d = 32 * dt + 16 * (g16 & 1) + 4 * (li & 3);
      toff[r][dt] = row * D + 8 * ((d >> 3) ^ swz<D>(row)) + (d & 7);
    }
  const float sl2 = p.scale * kLog2e;
  const float nl2 = nlse_s * sl2;  // -lse log2(e): the exponent is q.k sl2 + nl2 in float32

  // One 64-key tile, laid out by hand in fenced steps: the S^T and dP^T products of the
  // first 32 keys (the two chains alternating), then those of the last 32 keys while the
  // first 32 keys' probabilities and dS are formed, then the 16 dQ^T products while the
  // last 32 keys' dS are formed; operand reads PF steps ahead.
  auto body_sched = [&](auto Bc, auto Mc, int it) __attribute__((always_inline)) {
    constexpr int B = decltype(Bc)::value;
    constexpr bool MASK = decltype(Mc)::value;
    if (it + 1 < nt) load_tile(it + 1, std::integral_constant<int, B ^ 1>{});
    const bf16* kt = pick(Bc, sK0, sK1);
    const bf16* vt = pick(Bc, sV0, sV1);
    constexpr int NA = 2 * NKK;       // S^T and dP^T products of one 32-key half
    constexpr int NQ = 4 * NDT;       // dQ^T products of the tile
    constexpr int NST = 2 * NA + NQ;  // steps
    constexpr int PF = 2;
    f32x16 sacc[2], dpacc[2];
    bf16x8 aop[2 * NA], top[NQ];
    u32x4 w[4];  // dS^T of the four 16-key groups, packed bf16: the B operands as they are
    const int kpos0 = hs.k_pos0 + it * kKK;
    // step S < 2 NA: half h = S / NA, product j = S % NA of it (S^T if j even, dP^T if odd,
    // reduction slice kk = j / 2); step S >= 2 NA: dQ^T product q = S - 2 NA (keys of group
    // kb = q / NDT, dims 32 (q % NDT)..)
    auto fetch = [&](auto Sc) __attribute__((always_inline)) {
      constexpr int S = decltype(Sc)::value;
      if constexpr (S < 2 * NA) {
        constexpr int h = S / NA, j = S % NA, kk = j / 2;
        aop[S] = *(const bf16x8*)(((j & 1) ? vt : kt) + 32 * h * D + roff[kk]);
      } else {
        constexpr int q = S - 2 * NA, kb = q / NDT, dt = q % NDT;
        const bf16x4 lo = lds_read_tr16(kt + 16 * kb * D + toff[0][dt]);
        const bf16x4 up = lds_read_tr16(kt + 16 * kb * D + toff[1][dt]);
        top[q] = bf16x8{lo[0], lo[1], lo[2], lo[3], up[0], up[1], up[2], up[3]};
      }
    };
    // pair jj of the 4 of key group kb: probabilities and dS, packed bf16
    auto unit = [&](int kb, int jj) __attribute__((always_inline)) {
      float ds2[2];
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        const int i = 8 * (kb & 1) + 2 * jj + e;
        const int mt = kb >> 1;
        float pv = fast_exp2(fmaf(sacc[mt][i], sl2, nl2));
        if (MASK) {
          const int kpos = kpos0 + 32 * mt + 16 * (i >> 3) + 8 * hi + (i & 7);
          if (kpos > qpos) pv = 0.f;
        }
        ds2[e] = pv * dpacc[mt][i];
      }
      w[kb][jj] = pack_bf16x2(ds2[0], ds2[1]);
    };
    // vector work: group kb's four pairs at steps VSTEP(kb) .. + 3 (groups 0, 1 once the
    // first half's chains are complete, groups 2, 3 once the second half's are)
    static_assert(NKK == 8 && NDT == 4, "hand schedule written for D = 128");
    constexpr int V0 = NA + 2, V2 = 2 * NA;
    static_for<0, PF>([&](auto Sc) __attribute__((always_inline)) { fetch(Sc); });
    static_for<0, NST>([&](auto Sc) __attribute__((always_inline)) {
      constexpr int S = decltype(Sc)::value;
      if constexpr (S + PF < NST) fetch(std::integral_constant<int, S + PF>{});
      if constexpr (S < 2 * NA) {
        constexpr int h = S / NA, j = S % NA, kk = j / 2;
        if constexpr (j == 1) {  // dP^T of half h starts at -Delta (set here: shorter live range)
#pragma unroll
          for (int i = 0; i < 16; ++i) dpacc[h][i] = ndlt;
        }
        if constexpr (j & 1)
          dpacc[h] = mfma32(aop[S], oreg[kk], dpacc[h]);
        else
          sacc[h] = mfma32(aop[S], qreg[kk], kk == 0 ? f32x16{} : sacc[h]);
      } else {
        constexpr int q = S - 2 * NA, kb = q / NDT, dt = q % NDT;
        dqacc[dt] = mfma32(top[q], __builtin_bit_cast(bf16x8, w[kb]), dqacc[dt]);
      }
      if constexpr (S >= V0 && S < V0 + 8) unit((S - V0) / 4, (S - V0) % 4);
      if constexpr (S >= V2 && S < V2 + 8) unit(2 + (S - V2) / 4, (S - V2) % 4);
      __builtin_amdgcn_sched_barrier(0);
    });
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
  };
  // other head dims: the same work, ordered by the compiler
  auto body_plain = [&](auto Bc, auto Mc, int it) __attribute__((always_inline)) {
    constexpr int B = decltype(Bc)::value;
    constexpr bool MASK = decltype(Mc)::value;
    if (it + 1 < nt) load_tile(it + 1, std::integral_constant<int, B ^ 1>{});
    const bf16* kt = pick(Bc, sK0, sK1);
    const bf16* vt = pick(Bc, sV0, sV1);
    f32x16 sacc[2], dpacc[2];
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        sacc[mt][i] = 0.f;
        dpacc[mt][i] = ndlt;
      }
#pragma unroll
      for (int kk = 0; kk < NKK; ++kk) {
        sacc[mt] = mfma32(*(const bf16x8*)(kt + 32 * mt * D + roff[kk]), qreg[kk], sacc[mt]);
        dpacc[mt] = mfma32(*(const bf16x8*)(vt + 32 * mt * D + roff[kk]), oreg[kk], dpacc[mt]);
      }
    }
    const int kpos0 = hs.k_pos0 + it * kKK;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      u32x4 w;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        float ds2[2];
#pragma unroll
        for (int e = 0; e < 2; ++e) {
          const int i = 8 * (kb & 1) + 2 * j + e;
          const int mt = kb >> 1;
          float pv = fast_exp2(fmaf(sacc[mt][i], sl2, nl2));
          if (MASK) {
            const int kpos = kpos0 + 32 * mt + 16 * (i >> 3) + 8 * hi + (i & 7);
            if (kpos > qpos) pv = 0.f;
          }
          ds2[e] = pv * dpacc[mt][i];
        }
        w[j] = pack_bf16x2(ds2[0], ds2[1]);
      }
      const bf16x8 dsb = __builtin_bit_cast(bf16x8, w);
      // dQ^T += K^T dS^T for these 16 keys
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) {
        const bf16x4 lo = lds_read_tr16(kt + 16 * kb * D + toff[0][dt]);
        const bf16x4 up = lds_read_tr16(kt + 16 * kb * D + toff[1][dt]);
        const bf16x8 a = {lo[0], lo[1], lo[2], lo[3], up[0], up[1], up[2], up[3]};
        dqacc[dt] = mfma32(a, dsb, dqacc[dt]);
      }
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
  };
  auto body = [&](auto Bc, auto Mc, int it) __attribute__((always_inline)) {
    if constexpr (D == 128)
      body_sched(Bc, Mc, it);
    else
      body_plain(Bc, Mc, it);
  };
  auto run = [&](auto Mc, int a, int e) __attribute__((always_inline)) {
    int it = a;
    if ((it & 1) && it < e) body(std::integral_constant<int, 1>{}, Mc, it++);
    for (; it + 1 < e; it += 2) {
      body(std::integral_constant<int, 0>{}, Mc, it);
      body(std::integral_constant<int, 1>{}, Mc, it + 1);
    }
    if (it < e) body(std::integral_constant<int, 0>{}, Mc, it);
  };
  if (nt > 0) load_tile(0, std::integral_constant<int, 0>{});
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  run(std::false_type{}, 0, n_full);
  run(std::true_type{}, n_full, nt);

  // dq (float32, [B, Sq, H, D]) += scale * dQ; with dq_out set, the host's first active
  // step writes instead of adding and its last writes the bf16 result
  const long long qoff = (long long)b * p.q_bstride + (long long)qr * rs + h * D;
  float* dqrow = p.dq + qoff;
  const bool first = p.dq_out != nullptr && (hs.flags & kFirst);
  const bool fin = p.dq_out != nullptr && (hs.flags & kLast);
  // all carried values loaded before the first store (one memory round trip, not 16)
  f32x4 qin[NDT][4];
  if (first) {
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int gg = 0; gg < 4; ++gg) qin[dt][gg] = f32x4{0.f, 0.f, 0.f, 0.f};
  } else {
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int gg = 0; gg < 4; ++gg) qin[dt][gg] = *(const f32x4*)(dqrow + 32 * dt + 8 * gg + 4 * hi);
  }
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
    for (int gg = 0; gg < 4; ++gg) {
      const int d = 32 * dt + 8 * gg + 4 * hi;
      f32x4 t = qin[dt][gg];
#pragma unroll
      for (int e = 0; e < 4; ++e) t[e] += dqacc[dt][4 * gg + e] * p.scale;
      if (fin)
        *(u32x2*)((bf16*)p.dq_out + qoff + d) = u32x2{pack_bf16x2(t[0], t[1]), pack_bf16x2(t[2], t[3])};
      else
        *(f32x4*)(dqrow + d) = t;
    }
}

// =====================================================================================
// float32 backward (exact float32, no matrix cores).  dK/dV: one thread per key;
// dQ: one thread per query.  Query / key rows are staged through LDS 32 at a time.
// =====================================================================================
constexpr int kF = 64, kFT = 32;

template <int D>
__global__ __launch_bounds__(64) void bwd_dkdv_f32_kernel(const BwdStep p) {
  __shared__ float sQ[kFT * D], sO[kFT * D], sL[kFT], sD[kFT];
  const int n_kt = p.c / kF;
  const int BH = p.B * p.H;
  const int total = p.n_slots * BH * n_kt;
  const int L = blockIdx.x;
  if (L >= total) return;
  const int grp = L / n_kt, kt = L % n_kt;
  const int slot = grp / BH, bh = grp % BH;
  const int b = bh / p.H, h = bh % p.H;
  const StepHost hs = p.host[slot];
  const int t = threadIdx.x, rs = p.H * D;
  const int key = kt * kF + t;
  const int kpos = hs.k_pos0 + key;
  const float* kr = (const float*)hs.k + (long long)b * hs.kv_bstride + (long long)key * rs + h * D;
  const float* vr = (const float*)hs.v + (long long)b * hs.kv_bstride + (long long)key * rs + h * D;
  float k[D], v[D], dk[D], dv[D];
  #pragma unroll
  for (int d = 0; d < D; ++d) {
    k[d] = kr[d];
    v[d] = vr[d];
    dk[d] = 0.f;
    dv[d] = 0.f;
  }
  const float* qb = (const float*)p.q + (long long)b * p.q_bstride + h * D;
  const float* ob = (const float*)p.dO + (long long)b * p.q_bstride + h * D;
  const long long lrow0 = (long long)bh * p.Sq + hs.q_row0;
  for (int q0 = 0; q0 < p.c; q0 += kFT) {
    if (p.causal && hs.q_pos0 + q0 + kFT - 1 < hs.k_pos0 + kt * kF) continue;  // uniform
    __syncthreads();
    for (int e = t; e < kFT * D; e += 64) {
      const int r = e / D, d = e % D;
      const long long off = (long long)(hs.q_row0 + q0 + r) * rs + d;
      sQ[e] = qb[off];
      sO[e] = ob[off];
    }
    if (t < kFT) {
      sL[t] = p.lse[lrow0 + q0 + t];
      sD[t] = p.delta[lrow0 + q0 + t];
    }
    __syncthreads();
    for (int j = 0; j < kFT; ++j) {
      const int qpos = hs.q_pos0 + q0 + j;
      if (p.causal && kpos > qpos) continue;
      float s = 0.f, dp = 0.f;
      #pragma unroll
      for (int d = 0; d < D; ++d) {
        s = fmaf(sQ[j * D + d], k[d], s);
        dp = fmaf(sO[j * D + d], v[d], dp);
      }
      const float pr = expf(s * p.scale - sL[j]);
      const float ds = pr * (dp - sD[j]);
      #pragma unroll
      for (int d = 0; d < D; ++d) {
        dv[d] = fmaf(pr, sO[j * D + d], dv[d]);
        dk[d] = fmaf(ds, sQ[j * D + d], dk[d]);
      }
    }
  }
  const long long grow = (long long)b * p.dkv_bstride + (long long)(p.dkv_row0[slot] + key) * rs + h * D;
  #pragma unroll
  for (int d = 0; d < D; ++d) {
    p.dk[grow + d] += dk[d] * p.scale;
    p.dv[grow + d] += dv[d];
  }
}

template <int D>
__global__ __launch_bounds__(64) void bwd_dq_f32_kernel(const BwdStep p) {
  __shared__ float sK[kFT * D], sV[kFT * D];
  const int n_qt = p.c / kF;
  const int BH = p.B * p.H;
  const int total = p.n_slots * BH * n_qt;
  const int L = blockIdx.x;
  if (L >= total) return;
  const int grp = L / n_qt, qt = L % n_qt;
  const int slot = grp / BH, bh = grp % BH;
  const int b = bh / p.H, h = bh % p.H;
  const StepHost hs = p.host[slot];
  const int t = threadIdx.x, rs = p.H * D;
  const int qr = hs.q_row0 + qt * kF + t;
  const int qpos = hs.q_pos0 + qt * kF + t;
  const long long lrow = (long long)bh * p.Sq + qr;
  const float lse = p.lse[lrow], dlt = p.delta[lrow];
  const long long qoff = (long long)b * p.q_bstride + (long long)qr * rs + h * D;
  float q[D], o[D], dq[D];
  #pragma unroll
  for (int d = 0; d < D; ++d) {
    q[d] = ((const float*)p.q)[qoff + d];
    o[d] = ((const float*)p.dO)[qoff + d];
    dq[d] = 0.f;
  }
  const float* kb = (const float*)hs.k + (long long)b * hs.kv_bstride + h * D;
  const float* vb = (const float*)hs.v + (long long)b * hs.kv_bstride + h * D;
  for (int k0 = 0; k0 < p.c; k0 += kFT) {
    if (p.causal && hs.k_pos0 + k0 > hs.q_pos0 + qt * kF + kF - 1) break;  // uniform
    __syncthreads();
    for (int e = t; e < kFT * D; e += 64) {
      const int r = e / D, d = e % D;
      const long long off = (long long)(k0 + r) * rs + d;
      sK[e] = kb[off];
      sV[e] = vb[off];
    }
    __syncthreads();
    for (int j = 0; j < kFT; ++j) {
      if (p.causal && hs.k_pos0 + k0 + j > qpos) continue;
      float s = 0.f, dp = 0.f;
      #pragma unroll
      for (int d = 0; d < D; ++d) {
        s = fmaf(q[d], sK[j * D + d], s);
        dp = fmaf(o[d], sV[j * D + d], dp);
      }
      const float ds = expf(s * p.scale - lse) * (dp - dlt);
      #pragma unroll
      for (int d = 0; d < D; ++d) dq[d] = fmaf(ds, sK[j * D + d], dq[d]);
    }
  }
  float* dqrow = p.dq + qoff;
  #pragma unroll
  for (int d = 0; d < D; ++d) dqrow[d] += dq[d] * p.scale;
}

__global__ void cast_f32_bf16_kernel(const float* src, bf16* dst, long long n) {
  const long long i = ((long long)blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (i + 3 < n) {
    const f32x4 v = *(const f32x4*)(src + i);
    u32x2 w = {pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
    *(u32x2*)(dst + i) = w;
  } else {
    for (long long j = i; j < n; ++j) dst[j] = (bf16)src[j];
  }
}

__global__ void zero_f32_kernel(float* p, long long n) {
  const long long i = ((long long)blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (i + 3 < n) {
    *(f32x4*)(p + i) = f32x4{0.f, 0.f, 0.f, 0.f};
  } else {
    for (long long j = i; j < n; ++j) p[j] = 0.f;
  }
}

}  // namespace

hipError_t launch_bwd_pre_bf16(const void* o, const void* dO, const float* lse, float* delta, float* nlse_s, int B,
                               int S, int H, int D, hipStream_t st) {
  const long long blocks = (long long)B * ((S + kPreR - 1) / kPreR) * ((H + kPreH - 1) / kPreH);
  if (D == 128)
    hipLaunchKernelGGL(bwd_pre_bf16_kernel<128>, dim3(blocks), dim3(256), 0, st, (const bf16*)o, (const bf16*)dO, lse, delta, nlse_s, B, S, H);
  else
    hipLaunchKernelGGL(bwd_pre_bf16_kernel<64>, dim3(blocks), dim3(256), 0, st, (const bf16*)o, (const bf16*)dO, lse, delta, nlse_s, B, S, H);
  return hipGetLastError();
}

hipError_t launch_bwd_pre_f32(const float* o, const float* dO, float* delta, int B, int S, int H, int D,
                              hipStream_t st) {
  const long long blocks = (long long)B * ((S + kPreR - 1) / kPreR) * ((H + kPreH - 1) / kPreH);
  if (D == 128)
    hipLaunchKernelGGL(bwd_pre_f32_kernel<128>, dim3(blocks), dim3(256), 0, st, o, dO, delta, B, S, H);
  else
    hipLaunchKernelGGL(bwd_pre_f32_kernel<64>, dim3(blocks), dim3(256), 0, st, o, dO, delta, B, S, H);
  return hipGetLastError();
}

hipError_t launch_bwd_bf16(const BwdStep& s, int D, hipStream_t st) {
  if (s.n_slots == 0) return hipSuccess;
  // a forwarding destination needs both receive bases and a slot size
  for (int n = 0; n < s.n_slots; ++n)
    if (s.fwd.to[n] != 0 && (s.fwd.to[n] < 0 || s.fwd.k0 == nullptr || s.fwd.v0 == nullptr || s.fwd.blk_bytes <= 0))
      return hipErrorInvalidValue;
  // a last touch needs the bf16 outputs
  for (int n = 0; n < s.n_slots; ++n)
    if ((s.dkv_flags[n] & kLast) && (s.dk_out == nullptr || s.dv_out == nullptr)) return hipErrorInvalidValue;
  const int g1 = s.n_slots * s.B * s.H * (s.c / kKB);
  const int g2 = s.n_slots * s.B * s.H * (s.c / kQQ);
  if (D == 128) {
    hipLaunchKernelGGL(bwd_dkdv_split_kernel, dim3(g1), dim3(kPT), 0, st, s);
    hipLaunchKernelGGL(bwd_dq_bf16_kernel<128>, dim3(g2), dim3(kBT), 0, st, s);
  } else {
    hipLaunchKernelGGL(bwd_dkdv_bf16_kernel<64>, dim3(g1), dim3(kBT), 0, st, s);
    hipLaunchKernelGGL(bwd_dq_bf16_kernel<64>, dim3(g2), dim3(kBT), 0, st, s);
  }
  return hipGetLastError();
}

hipError_t launch_bwd_f32(const BwdStep& s, int D, hipStream_t st) {
  if (s.n_slots == 0) return hipSuccess;
  const int g = s.n_slots * s.B * s.H * (s.c / kF);
  if (D == 128) {
    hipLaunchKernelGGL(bwd_dkdv_f32_kernel<128>, dim3(g), dim3(64), 0, st, s);
    hipLaunchKernelGGL(bwd_dq_f32_kernel<128>, dim3(g), dim3(64), 0, st, s);
  } else {
    hipLaunchKernelGGL(bwd_dkdv_f32_kernel<64>, dim3(g), dim3(64), 0, st, s);
    hipLaunchKernelGGL(bwd_dq_f32_kernel<64>, dim3(g), dim3(64), 0, st, s);
  }
  return hipGetLastError();
}

hipError_t launch_cast_f32_bf16(const float* src, void* dst, long long n, hipStream_t st) {
  const long long blocks = (n / 4 + 255) / 256 + 1;
  hipLaunchKernelGGL(cast_f32_bf16_kernel, dim3(blocks), dim3(256), 0, st, src, (bf16*)dst, n);
  return hipGetLastError();
}

hipError_t launch_zero_f32(float* p, long long n, hipStream_t st) {
  const long long blocks = (n / 4 + 255) / 256 + 1;
  hipLaunchKernelGGL(zero_f32_kernel, dim3(blocks), dim3(256), 0, st, p, n);
  return hipGetLastError();
}

}  // namespace ra
