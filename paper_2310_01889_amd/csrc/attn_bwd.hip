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
#include "ra_kernels.h"

namespace ra {
namespace {

__device__ __forceinline__ int swap_bits23(int r) {
  return (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1);
}

// -------------------------------------------------------------------------------------
// Delta_r = sum_d dO_rd * O_rd  (float32 [B, H, S]); rows in memory order (b, r, h).
// -------------------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(256) void bwd_pre_bf16_kernel(const bf16* o, const bf16* dO, float* delta,
                                                           int B, int S, int H) {
  constexpr int TPR = D / 8;  // threads per row
  const long long row = (long long)blockIdx.x * (256 / TPR) + threadIdx.x / TPR;
  const int c = (threadIdx.x % TPR) * 8;
  const long long nrows = (long long)B * S * H;
  float s = 0.f;
  if (row < nrows) {
    const bf16x8 a = *(const bf16x8*)(o + row * D + c);
    const bf16x8 g = *(const bf16x8*)(dO + row * D + c);
    #pragma unroll
    for (int e = 0; e < 8; ++e) s = fmaf((float)a[e], (float)g[e], s);
  }
  for (int off = TPR / 2; off > 0; off >>= 1) s += __shfl_xor(s, off, 64);
  if (row < nrows && threadIdx.x % TPR == 0) {
    const int h = (int)(row % H);
    const long long br = row / H;
    const int r = (int)(br % S), b = (int)(br / S);
    delta[((long long)b * H + h) * S + r] = s;
  }
}

template <int D>
__global__ __launch_bounds__(256) void bwd_pre_f32_kernel(const float* o, const float* dO, float* delta,
                                                          int B, int S, int H) {
  constexpr int TPR = D / 4;
  const long long row = (long long)blockIdx.x * (256 / TPR) + threadIdx.x / TPR;
  const int c = (threadIdx.x % TPR) * 4;
  const long long nrows = (long long)B * S * H;
  float s = 0.f;
  if (row < nrows) {
    const f32x4 a = *(const f32x4*)(o + row * D + c);
    const f32x4 g = *(const f32x4*)(dO + row * D + c);
    #pragma unroll
    for (int e = 0; e < 4; ++e) s = fmaf(a[e], g[e], s);
  }
  for (int off = TPR / 2; off > 0; off >>= 1) s += __shfl_xor(s, off, 64);
  if (row < nrows && threadIdx.x % TPR == 0) {
    const int h = (int)(row % H);
    const long long br = row / H;
    const int r = (int)(br % S), b = (int)(br / S);
    delta[((long long)b * H + h) * S + r] = s;
  }
}

// =====================================================================================
// bf16 dK/dV kernel: 4 waves x 32 keys = 128 keys per workgroup; loops over 64-query
// tiles of the host's block staged in LDS.  Per wave:
//   S  = Q K^T   [query x key], lanes run over keys (A = Q rows from LDS, with row bits
//                2 and 3 swapped; B = K of the wave's keys held in registers)
//   P  = exp2(S * log2e/sqrt(D) - lse * log2e), masked -> 0
//   dV^T += dO^T P     (A = dO^T by LDS transpose read, B = P from registers)
//   dP = dO V^T        (A = dO rows, B = V of the wave's keys in registers)
//   dS = P * (dP - Delta)
//   dK^T += Q^T dS     (A = Q^T by LDS transpose read, B = dS)
// =====================================================================================
constexpr int kKB = 128, kQB = 64, kBT = 256;

template <int D>
__global__ __launch_bounds__(kBT, 1) void bwd_dkdv_bf16_kernel(const BwdStep p) {
  constexpr int QS = D + 8;    // LDS row stride for Q and dO tiles
  constexpr int NKK = D / 16, NDT = D / 32;
  constexpr int CPR = D / 8, RPP = kBT / CPR, NPASS = kQB / RPP;
  __shared__ __attribute__((aligned(16))) bf16 sQ[2][kQB * QS];
  __shared__ __attribute__((aligned(16))) bf16 sO[2][kQB * QS];  // dO tile
  __shared__ __attribute__((aligned(16))) float sL[2][kQB];       // lse * log2e
  __shared__ __attribute__((aligned(16))) float sD[2][kQB];       // Delta

  const int n_kt = p.c / kKB;
  const int BH = p.B * p.H;
  const int total = p.n_slots * BH * n_kt;
  const int Lid = xcd_swizzle(blockIdx.x, total);
  const int grp = Lid / n_kt, kt = Lid % n_kt;
  const int slot = grp / BH, bh = grp % BH;
  const int b = bh / p.H, h = bh % p.H;
  const StepHost hs = p.host[slot];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, l32 = lane & 31, hi = lane >> 5;
  const int rs = p.H * D;

  const int key_in_blk = kt * kKB + wave * 32 + l32;  // this lane's key (as B-operand column)
  const int kpos = hs.k_pos0 + key_in_blk;
  const bf16* krow = (const bf16*)hs.k + (long long)b * hs.kv_bstride + (long long)key_in_blk * rs + h * D;
  const bf16* vrow = (const bf16*)hs.v + (long long)b * hs.kv_bstride + (long long)key_in_blk * rs + h * D;
  bf16x8 kreg[NKK], vreg[NKK];
  #pragma unroll
  for (int kk = 0; kk < NKK; ++kk) {
    kreg[kk] = *(const bf16x8*)(krow + 16 * kk + 8 * hi);
    vreg[kk] = *(const bf16x8*)(vrow + 16 * kk + 8 * hi);
  }
  f32x16 dkacc[NDT], dvacc[NDT];
  #pragma unroll
  for (int dt = 0; dt < NDT; ++dt)
    #pragma unroll
    for (int i = 0; i < 16; ++i) dkacc[dt][i] = dvacc[dt][i] = 0.f;

  // query tiles with at least one query that sees a key of this workgroup
  const int wg_first_k = hs.k_pos0 + kt * kKB;
  int qt0 = 0;
  const int n_qtiles = p.c / kQB;
  if (p.causal) {
    // first query position >= wg_first_k
    const int rel = wg_first_k - hs.q_pos0;
    qt0 = rel <= 0 ? 0 : min(n_qtiles, rel / kQB);
  }

  const bf16* qbase = (const bf16*)p.q + (long long)b * p.q_bstride + h * D;
  const bf16* obase = (const bf16*)p.dO + (long long)b * p.q_bstride + h * D;
  const long long lrow0 = (long long)bh * p.Sq + hs.q_row0;
  const int st_r = tid / CPR, st_c = (tid % CPR) * 8;
  u32x4 qpre[NPASS], opre[NPASS];
  float lpre = 0.f, dpre = 0.f;
  auto gload = [&](int qt) {
    #pragma unroll
    for (int ps = 0; ps < NPASS; ++ps) {
      const long long off = (long long)(hs.q_row0 + qt * kQB + st_r + ps * RPP) * rs + st_c;
      qpre[ps] = *(const u32x4*)(qbase + off);
      opre[ps] = *(const u32x4*)(obase + off);
    }
    if (tid < kQB) {
      lpre = p.lse[lrow0 + qt * kQB + tid] * kLog2e;
      dpre = p.delta[lrow0 + qt * kQB + tid];
    }
  };
  auto lstore = [&](int buf) {
    #pragma unroll
    for (int ps = 0; ps < NPASS; ++ps) {
      const int r = st_r + ps * RPP;
      *(u32x4*)(&sQ[buf][r * QS + st_c]) = qpre[ps];
      *(u32x4*)(&sO[buf][r * QS + st_c]) = opre[ps];
    }
    if (tid < kQB) {
      sL[buf][tid] = lpre;
      sD[buf][tid] = dpre;
    }
  };

  const float sl2 = p.scale * kLog2e;
  const int prow = swap_bits23(l32);
  if (qt0 < n_qtiles) {
    gload(qt0);
    lstore(0);
  }
  __syncthreads();
  for (int qt = qt0; qt < n_qtiles; ++qt) {
    const int buf = (qt - qt0) & 1;
    if (qt + 1 < n_qtiles) gload(qt + 1);
    const int qpos0 = hs.q_pos0 + qt * kQB;

    // S = Q K^T : two 32-query tiles
    f32x16 sacc[2];
    #pragma unroll
    for (int qm = 0; qm < 2; ++qm) {
      #pragma unroll
      for (int i = 0; i < 16; ++i) sacc[qm][i] = 0.f;
      const bf16* qr = &sQ[buf][(32 * qm + prow) * QS + 8 * hi];
      #pragma unroll
      for (int kk = 0; kk < NKK; ++kk) sacc[qm] = mfma32(*(const bf16x8*)(qr + 16 * kk), kreg[kk], sacc[qm]);
    }
    // P (queries 32qm + 16(i/8) + 8hi + i%8 of the tile)
    const bool need_mask = p.causal && (wg_first_k + kKB - 1 > qpos0);
    #pragma unroll
    for (int qm = 0; qm < 2; ++qm)
      #pragma unroll
      for (int hb = 0; hb < 2; ++hb) {
        const int q0 = 32 * qm + 16 * hb + 8 * hi;
        const f32x4 la = *(const f32x4*)&sL[buf][q0];
        const f32x4 lb = *(const f32x4*)&sL[buf][q0 + 4];
        #pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float lv = e < 4 ? la[e] : lb[e - 4];
          float pv = fast_exp2(fmaf(sacc[qm][8 * hb + e], sl2, -lv));
          if (need_mask && kpos > qpos0 + q0 + e) pv = 0.f;
          sacc[qm][8 * hb + e] = pv;
        }
      }
    // dV^T += dO^T P
    bf16x8 pb[4];
    #pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      u32x4 w;
      #pragma unroll
      for (int j = 0; j < 4; ++j)
        w[j] = pack_bf16x2(sacc[kb >> 1][8 * (kb & 1) + 2 * j], sacc[kb >> 1][8 * (kb & 1) + 2 * j + 1]);
      pb[kb] = __builtin_bit_cast(bf16x8, w);
    }
    const int g = lane >> 4, li = lane & 15;
    const int tcol = 16 * (g & 1) + 4 * (li & 3);
    const int trow = 8 * hi + (li >> 2);
    #pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      const bf16* op = &sO[buf][(16 * kb + trow) * QS + tcol];
      #pragma unroll
      for (int dt = 0; dt < NDT; ++dt) {
        const bf16x4 lo = lds_read_tr16(op + 32 * dt);
        const bf16x4 up = lds_read_tr16(op + 4 * QS + 32 * dt);
        const bf16x8 a = {lo[0], lo[1], lo[2], lo[3], up[0], up[1], up[2], up[3]};
        dvacc[dt] = mfma32(a, pb[kb], dvacc[dt]);
      }
    }
    // dP = dO V^T, then dS = P * (dP - Delta)
    #pragma unroll
    for (int qm = 0; qm < 2; ++qm) {
      f32x16 dp;
      #pragma unroll
      for (int i = 0; i < 16; ++i) dp[i] = 0.f;
      const bf16* orr = &sO[buf][(32 * qm + prow) * QS + 8 * hi];
      #pragma unroll
      for (int kk = 0; kk < NKK; ++kk) dp = mfma32(*(const bf16x8*)(orr + 16 * kk), vreg[kk], dp);
      #pragma unroll
      for (int hb = 0; hb < 2; ++hb) {
        const int q0 = 32 * qm + 16 * hb + 8 * hi;
        const f32x4 da = *(const f32x4*)&sD[buf][q0];
        const f32x4 db = *(const f32x4*)&sD[buf][q0 + 4];
        #pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float dv = e < 4 ? da[e] : db[e - 4];
          sacc[qm][8 * hb + e] = sacc[qm][8 * hb + e] * (dp[8 * hb + e] - dv);
        }
      }
    }
    // dK^T += Q^T dS
    #pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      u32x4 w;
      #pragma unroll
      for (int j = 0; j < 4; ++j)
        w[j] = pack_bf16x2(sacc[kb >> 1][8 * (kb & 1) + 2 * j], sacc[kb >> 1][8 * (kb & 1) + 2 * j + 1]);
      const bf16x8 dsb = __builtin_bit_cast(bf16x8, w);
      const bf16* qp = &sQ[buf][(16 * kb + trow) * QS + tcol];
      #pragma unroll
      for (int dt = 0; dt < NDT; ++dt) {
        const bf16x4 lo = lds_read_tr16(qp + 32 * dt);
        const bf16x4 up = lds_read_tr16(qp + 4 * QS + 32 * dt);
        const bf16x8 a = {lo[0], lo[1], lo[2], lo[3], up[0], up[1], up[2], up[3]};
        dkacc[dt] = mfma32(a, dsb, dkacc[dt]);
      }
    }
    if (qt + 1 < n_qtiles) lstore(buf ^ 1);
    __syncthreads();
  }

  // add into the float32 gradient of the block (its home rows)
  const long long grow = (long long)b * p.dkv_bstride + (long long)(p.dkv_row0[slot] + key_in_blk) * rs + h * D;
  #pragma unroll
  for (int dt = 0; dt < NDT; ++dt)
    #pragma unroll
    for (int gg = 0; gg < 4; ++gg) {
      const int d = 32 * dt + 8 * gg + 4 * hi;
      f32x4* dkp = (f32x4*)(p.dk + grow + d);
      f32x4* dvp = (f32x4*)(p.dv + grow + d);
      f32x4 k4 = *dkp, v4 = *dvp;
      #pragma unroll
      for (int e = 0; e < 4; ++e) {
        k4[e] += dkacc[dt][4 * gg + e] * p.scale;
        v4[e] += dvacc[dt][4 * gg + e];
      }
      *dkp = k4;
      *dvp = v4;
    }
}

// =====================================================================================
// bf16 dQ kernel: 4 waves x 32 queries = 128 queries per workgroup; loops over 64-key
// tiles.  Per wave, lanes run over queries:
//   S^T = K Q^T (A = K rows from LDS with bits 2,3 swapped, B = Q in registers)
//   P^T = exp2(S^T * log2e/sqrt(D) - lse*log2e)
//   dP^T = V dO^T (A = V rows, B = dO in registers)
//   dS^T = P^T * (dP^T - Delta)
//   dQ^T += K^T dS^T (A = K^T by LDS transpose read, B = dS^T)
// =====================================================================================
constexpr int kQQ = 128, kKK = 64;

template <int D>
__global__ __launch_bounds__(kBT, 1) void bwd_dq_bf16_kernel(const BwdStep p) {
  constexpr int KS = D + 8;
  constexpr int NKK = D / 16, NDT = D / 32;
  constexpr int CPR = D / 8, RPP = kBT / CPR, NPASS = kKK / RPP;
  __shared__ __attribute__((aligned(16))) bf16 sK[2][kKK * KS];
  __shared__ __attribute__((aligned(16))) bf16 sV[2][kKK * KS];

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
  const int rs = p.H * D;

  const int qr = hs.q_row0 + qt * kQQ + wave * 32 + l32;
  const int qpos = hs.q_pos0 + qt * kQQ + wave * 32 + l32;
  const int tile_first_q = hs.q_pos0 + qt * kQQ;
  const long long lrow = (long long)bh * p.Sq + qr;
  const float lse2 = p.lse[lrow] * kLog2e;
  const float dlt = p.delta[lrow];

  bf16x8 qreg[NKK], oreg[NKK];
  {
    const long long off = (long long)b * p.q_bstride + (long long)qr * rs + h * D + 8 * hi;
    #pragma unroll
    for (int kk = 0; kk < NKK; ++kk) {
      qreg[kk] = *(const bf16x8*)((const bf16*)p.q + off + 16 * kk);
      oreg[kk] = *(const bf16x8*)((const bf16*)p.dO + off + 16 * kk);
    }
  }
  f32x16 dqacc[NDT];
  #pragma unroll
  for (int dt = 0; dt < NDT; ++dt)
    #pragma unroll
    for (int i = 0; i < 16; ++i) dqacc[dt][i] = 0.f;

  int nt = p.c / kKK;
  if (p.causal) {
    const int vis = tile_first_q + kQQ - hs.k_pos0;
    nt = min(nt, max(0, (vis + kKK - 1) / kKK));
  }
  const bf16* kbase = (const bf16*)hs.k + (long long)b * hs.kv_bstride + h * D;
  const bf16* vbase = (const bf16*)hs.v + (long long)b * hs.kv_bstride + h * D;
  const int st_r = tid / CPR, st_c = (tid % CPR) * 8;
  u32x4 kpre[NPASS], vpre[NPASS];
  auto gload = [&](int it) {
    #pragma unroll
    for (int ps = 0; ps < NPASS; ++ps) {
      const long long off = (long long)(it * kKK + st_r + ps * RPP) * rs + st_c;
      kpre[ps] = *(const u32x4*)(kbase + off);
      vpre[ps] = *(const u32x4*)(vbase + off);
    }
  };
  auto lstore = [&](int buf) {
    #pragma unroll
    for (int ps = 0; ps < NPASS; ++ps) {
      const int r = st_r + ps * RPP;
      *(u32x4*)(&sK[buf][r * KS + st_c]) = kpre[ps];
      *(u32x4*)(&sV[buf][r * KS + st_c]) = vpre[ps];
    }
  };
  const float sl2 = p.scale * kLog2e;
  const int krow_perm = swap_bits23(l32);
  if (nt > 0) {
    gload(0);
    lstore(0);
  }
  __syncthreads();
  for (int it = 0; it < nt; ++it) {
    const int buf = it & 1;
    if (it + 1 < nt) gload(it + 1);
    f32x16 sacc[2], dpacc[2];
    #pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
      #pragma unroll
      for (int i = 0; i < 16; ++i) sacc[mt][i] = dpacc[mt][i] = 0.f;
      const bf16* kr = &sK[buf][(32 * mt + krow_perm) * KS + 8 * hi];
      const bf16* vr = &sV[buf][(32 * mt + krow_perm) * KS + 8 * hi];
      #pragma unroll
      for (int kk = 0; kk < NKK; ++kk) {
        sacc[mt] = mfma32(*(const bf16x8*)(kr + 16 * kk), qreg[kk], sacc[mt]);
        dpacc[mt] = mfma32(*(const bf16x8*)(vr + 16 * kk), oreg[kk], dpacc[mt]);
      }
    }
    const int kpos0 = hs.k_pos0 + it * kKK;
    const bool need_mask = p.causal && (kpos0 + kKK - 1 > tile_first_q);
    bf16x8 dsb[4];
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
          float pv = fast_exp2(fmaf(sacc[mt][i], sl2, -lse2));
          if (need_mask) {
            const int kpos = kpos0 + 32 * mt + 16 * (i >> 3) + 8 * hi + (i & 7);
            if (kpos > qpos) pv = 0.f;
          }
          ds2[e] = pv * (dpacc[mt][i] - dlt);
        }
        w[j] = pack_bf16x2(ds2[0], ds2[1]);
      }
      dsb[kb] = __builtin_bit_cast(bf16x8, w);
    }
    // dQ^T += K^T dS^T
    const int g = lane >> 4, li = lane & 15;
    const int tcol = 16 * (g & 1) + 4 * (li & 3);
    const int trow = 8 * hi + (li >> 2);
    #pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      const bf16* kp = &sK[buf][(16 * kb + trow) * KS + tcol];
      #pragma unroll
      for (int dt = 0; dt < NDT; ++dt) {
        const bf16x4 lo = lds_read_tr16(kp + 32 * dt);
        const bf16x4 up = lds_read_tr16(kp + 4 * KS + 32 * dt);
        const bf16x8 a = {lo[0], lo[1], lo[2], lo[3], up[0], up[1], up[2], up[3]};
        dqacc[dt] = mfma32(a, dsb[kb], dqacc[dt]);
      }
    }
    if (it + 1 < nt) lstore(buf ^ 1);
    __syncthreads();
  }
  // dq (float32, [B, Sq, H, D]) += scale * dQ
  float* dqrow = p.dq + (long long)b * p.q_bstride + (long long)qr * rs + h * D;
  #pragma unroll
  for (int dt = 0; dt < NDT; ++dt)
    #pragma unroll
    for (int gg = 0; gg < 4; ++gg) {
      const int d = 32 * dt + 8 * gg + 4 * hi;
      f32x4* dp = (f32x4*)(dqrow + d);
      f32x4 t = *dp;
      #pragma unroll
      for (int e = 0; e < 4; ++e) t[e] += dqacc[dt][4 * gg + e] * p.scale;
      *dp = t;
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

hipError_t launch_bwd_pre_bf16(const void* o, const void* dO, float* delta, int B, int S, int H, int D,
                               hipStream_t st) {
  const long long rows = (long long)B * S * H;
  const int rpb = 256 / (D / 8);
  const long long blocks = (rows + rpb - 1) / rpb;
  if (D == 128)
    hipLaunchKernelGGL(bwd_pre_bf16_kernel<128>, dim3(blocks), dim3(256), 0, st, (const bf16*)o, (const bf16*)dO, delta, B, S, H);
  else
    hipLaunchKernelGGL(bwd_pre_bf16_kernel<64>, dim3(blocks), dim3(256), 0, st, (const bf16*)o, (const bf16*)dO, delta, B, S, H);
  return hipGetLastError();
}

hipError_t launch_bwd_pre_f32(const float* o, const float* dO, float* delta, int B, int S, int H, int D,
                              hipStream_t st) {
  const long long rows = (long long)B * S * H;
  const int rpb = 256 / (D / 4);
  const long long blocks = (rows + rpb - 1) / rpb;
  if (D == 128)
    hipLaunchKernelGGL(bwd_pre_f32_kernel<128>, dim3(blocks), dim3(256), 0, st, o, dO, delta, B, S, H);
  else
    hipLaunchKernelGGL(bwd_pre_f32_kernel<64>, dim3(blocks), dim3(256), 0, st, o, dO, delta, B, S, H);
  return hipGetLastError();
}

hipError_t launch_bwd_bf16(const BwdStep& s, int D, hipStream_t st) {
  if (s.n_slots == 0) return hipSuccess;
  const int g1 = s.n_slots * s.B * s.H * (s.c / kKB);
  const int g2 = s.n_slots * s.B * s.H * (s.c / kQQ);
  if (D == 128) {
    hipLaunchKernelGGL(bwd_dkdv_bf16_kernel<128>, dim3(g1), dim3(kBT), 0, st, s);
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
