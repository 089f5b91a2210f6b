// Ring-attention forward step kernels for gfx950.
//
// One launch folds, for every host listed in the step, the key/value block that host
// holds into its running state -- running row maximum m, running denominator l and
// unnormalised output (numerator) acc -- as the online-softmax recurrence of the
// paper's blockwise attention (Section 2 "Blockwise Parallel Transformers"; Section 3;
// the carry of the Appendix A forward scan):
//     m' = max(m, rowmax(s)),  p = exp(s - m'),
//     l' = l * exp(m - m') + rowsum(p),  acc' = acc * exp(m - m') + p v
// with s = q k^T / sqrt(D), masked (causal, by global position) keys giving p = 0.
// On a host's first active step the state starts from (m=-inf, l=0, acc=0) in
// registers; on its last it is finalised into o = acc / l and lse = m + ln l.
#include <type_traits>

#include "ra_common.h"
#include "ra_kernels.h"

namespace ra {

// ===================================================================================
// bf16 kernel: 4 waves, 128 queries per workgroup (32 per wave), 64-key tiles.
//
// Per wave, scores are formed transposed, S^T = K Q^T (32x32x16 MFMA, A = K rows from
// LDS, B = Q held in registers), so that each lane owns one query: its row max and
// row sum are in-lane reductions plus one exchange with lane l^32.  K rows are loaded
// with bits 2 and 3 of the row index swapped, which makes each lane half hold 8
// consecutive keys per 16-key group; the probabilities P^T then serve directly as the
// B operand of O^T += V^T P^T, whose A operand is read from the row-major V tile with
// the LDS transpose read.  O^T (128 dims x 32 queries per wave) stays in registers.
// ===================================================================================
namespace {

constexpr int kBM = 128, kBN = 64, kThreads = 256;
constexpr float kTau = 8.f;  // lazy-rescale threshold (log2 units)
constexpr int kPF = 2;       // LDS operand reads issued this many schedule steps ahead


// LDS tiles are unpadded [64 rows][D] with the 16-byte chunks of each row permuted by
// an XOR swizzle, so that every read pattern below is free of bank conflicts:
//   * row reads (A operand of S^T): 16 lanes read 16 consecutive rows at one chunk;
//   * transpose reads (V^T): 16 lanes read 4 consecutive rows x 32 contiguous bytes.
// For D = 128 (16 chunks per row): chunk c of row r lives at c ^ (4 (r & 3) + ((r >> 2) & 3));
// for D = 64 (8 chunks, two rows per 256-byte bank sweep) at c ^ s, s = (r >> 1) & 7 with
// bit 2 flipped on odd s.  Tiles are filled with direct-to-LDS loads (no registers):
// lane i of a 1 KB load lands at byte 16 i of its destination, so each lane fetches the
// logical chunk that the swizzle puts there.
template <int D>
__global__ __launch_bounds__(kThreads, 2) void fwd_bf16_kernel(const FwdStep p) {
  constexpr int NKK = D / 16;  // 16-wide reduction steps of q.k
  constexpr int NDT = D / 32;  // 32-row output tiles of O^T
  constexpr int CPR = D / 8;   // 16-byte chunks per row
  constexpr int ROWS_PER_LOAD = 64 / CPR;               // rows filled by one 1 KB wave load
  constexpr int RPW = kBN / 4;                           // tile rows each wave fills
  constexpr int LOADS = RPW / ROWS_PER_LOAD;             // 1 KB loads per wave per tile
  constexpr int TILE = kBN * D;                          // elements per tile
  // Four separate LDS objects (not one [2][TILE] array per operand): the compiler then
  // knows that reads of one buffer do not alias direct-to-LDS loads in flight into the
  // other, and does not wait for those loads before every read.
  __shared__ __attribute__((aligned(1024))) bf16 sK0[TILE];
  __shared__ __attribute__((aligned(1024))) bf16 sK1[TILE];
  __shared__ __attribute__((aligned(1024))) bf16 sV0[TILE];
  __shared__ __attribute__((aligned(1024))) bf16 sV1[TILE];
  auto kbuf = [&](auto Bc) __attribute__((always_inline)) -> bf16* {
    if constexpr (decltype(Bc)::value == 0) return sK0; else return sK1;
  };
  auto vbuf = [&](auto Bc) __attribute__((always_inline)) -> bf16* {
    if constexpr (decltype(Bc)::value == 0) return sV0; else return sV1;
  };
  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;

  const int n_qt = p.c / kBM;
  const int BH = p.B * p.H;
  const int total = p.n_slots * BH * n_qt;
  const int L = xcd_swizzle(blockIdx.x, total);
  const int grp = L / n_qt;
  const int qt = n_qt - 1 - (L % n_qt);  // longest causal rows first
  const int slot = grp / BH, bh = grp % BH;
  const int b = bh / p.H, h = bh % p.H;
  const StepHost hs = p.host[slot];

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);  // uniform: LDS destinations in scalar registers
  const int l32 = lane & 31, hi = lane >> 5;
  const int rs = p.H * D;  // row stride of q / k / v / o (elements)

  const int q_tile_row = hs.q_row0 + qt * kBM;       // first q-space row of the workgroup
  const int qr = q_tile_row + wave * 32 + l32;       // this lane's query row
  const int qpos = hs.q_pos0 + qt * kBM + wave * 32 + l32;
  const int tile_first_q = hs.q_pos0 + qt * kBM;

  const bf16* qbase = (const bf16*)p.q + (long long)b * p.q_bstride + h * D;
  const bf16* kbase = (const bf16*)hs.k + (long long)b * hs.kv_bstride + h * D;
  const bf16* vbase = (const bf16*)hs.v + (long long)b * hs.kv_bstride + h * D;

  // key tiles with at least one visible key; the first n_full need no mask
  int nt = p.c / kBN, n_full = nt;
  if (p.causal) {
    const int vis = tile_first_q + kBM - hs.k_pos0;  // keys visible to the last row
    nt = min(nt, max(0, (vis + kBN - 1) / kBN));
    n_full = min(nt, max(0, (tile_first_q - hs.k_pos0 + 1) / kBN));
  }

  // ---- running state -------------------------------------------------------------
  f32x16 oacc[NDT];
  float m_run, l_run;
  const long long st_row = (long long)bh * p.Sq + qr;
  float* acc_tile = p.acc + ((long long)bh * (p.Sq / kBM) + q_tile_row / kBM) * (kBM * D);
  if (hs.flags & kFirst) {
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int i = 0; i < 16; ++i) oacc[dt][i] = 0.f;
    m_run = -INFINITY;
    l_run = 0.f;
  } else {
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const f32x4 t = ((const f32x4*)acc_tile)[((wave * NDT + dt) * 4 + g) * 64 + lane];
#pragma unroll
        for (int e = 0; e < 4; ++e) oacc[dt][4 * g + e] = t[e];
      }
    m_run = p.m[st_row];
    l_run = hi ? 0.f : p.l[st_row];
  }

  // ---- Q in registers: B operand of S^T = K Q^T (n = query, k = dim) ---------------
  // Q as stored (bf16): the products q.k are exact in the float32 accumulators, and the
  // scale log2(e)/sqrt(D) is applied in float32 (the paper's float32 logits), once per
  // score, right before its exponential.
  const float sl2 = p.scale * kLog2e;
  const float isl2 = 1.f / sl2;
  bf16x8 qreg[NKK];
  {
    const bf16* qrow = qbase + (long long)qr * rs;
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) qreg[kk] = *(const bf16x8*)(qrow + 16 * kk + 8 * hi);
  }
  // Scores in log2 units are sl2 * q.k.  The score accumulators start from -m_eff / sl2
  // (m_eff = running maximum in log2 units, 0 while it is still -inf), so each MFMA chain
  // yields (s - m_eff) / sl2, and one multiply as soon as a tile's chains are complete
  // gives s - m_eff, the exponent.  thr: a row whose new scores exceed it forces a
  // rescale (kTau above the maximum, any visible key at all while the maximum is still
  // -inf).
  float m_eff = (m_run == -INFINITY) ? 0.f : m_run;
  float thr = (m_run == -INFINITY) ? -INFINITY : kTau;
  f32x16 minit;
#pragma unroll
  for (int i = 0; i < 16; ++i) minit[i] = -m_eff * isl2;

  // ---- direct-to-LDS staging: each wave fills 16 rows of a tile ---------------------
  // load j of a wave covers rows wave*RPW + j*ROWS_PER_LOAD + lane / CPR; the lane's
  // physical chunk is lane % CPR, its logical (global) chunk that ^ swz(row).
  int goff[LOADS];  // byte offsets from the tile base
#pragma unroll
  for (int j = 0; j < LOADS; ++j) {
    const int r = wave * RPW + j * ROWS_PER_LOAD + lane / CPR;
    goff[j] = 2 * (r * rs + 8 * ((lane % CPR) ^ swz<D>(r)));
  }
  // buffer loads with the LDS flag: the tile base is a wave-uniform descriptor, so the
  // per-tile address update is scalar work; reads past the tile return zero
  auto dload = [&](const bf16* src_tile, bf16* dst_tile) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < LOADS; ++j)
      buffer_load_lds16(src_tile, kBN * rs * 2, dst_tile + (wave_u * RPW + j * ROWS_PER_LOAD) * D, goff[j]);
  };
  auto load_k = [&](int it, auto Bc) __attribute__((always_inline)) { dload(kbase + (long long)it * kBN * rs, kbuf(Bc)); };
  auto load_v = [&](int it, auto Bc) __attribute__((always_inline)) { dload(vbase + (long long)it * kBN * rs, vbuf(Bc)); };

  // ---- per-lane LDS read offsets (elements), fixed across tiles ----------------------
  // row reads of K: row 32 mt + swap_bits23(l32), logical chunk 2 kk + hi
  const int krow = swap_bits23(l32);
  int koff[NKK];
#pragma unroll
  for (int kk = 0; kk < NKK; ++kk) koff[kk] = krow * D + 8 * ((2 * kk + hi) ^ swz<D>(krow));
  // transpose reads of V: rows 16 kb + 8 hi + 4 r + li / 4, dims 32 dt + 16 (g & 1) + 4 (li & 3)
  const int g16 = lane >> 4, li = lane & 15;
  int voff[2][NDT];
#pragma unroll
  for (int r = 0; r < 2; ++r)
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) {
      const int row = 8 * hi + 4 * r + (li >> 2);
      const int d = 32 * dt + 16 * (g16 & 1) + 4 * (li & 3);
      voff[r][dt] = row * D + 8 * ((d >> 3) ^ swz<D>(row)) + (d & 7);
    }

  // S^T = K Q^T for the 64 keys of K buffer `buf` x this wave's 32 queries
  auto scores = [&](const bf16* kt, f32x16* sacc) __attribute__((always_inline)) {
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
      sacc[mt] = mfma32(*(const bf16x8*)(kt + 32 * mt * D + koff[0]), qreg[0], minit);
#pragma unroll
      for (int kk = 1; kk < NKK; ++kk)
        sacc[mt] = mfma32(*(const bf16x8*)(kt + 32 * mt * D + koff[kk]), qreg[kk], sacc[mt]);
    }
  };

  // ---- pipeline: K runs one tile ahead of V ------------------------------------------
  // While tile it is processed, LDS holds K tiles it, it+1 and V tile it; loads of K tile
  // it+2 (into the buffer of K tile it) and V tile it+1 (into the buffer of V tile it-1)
  // are in flight.  One straight-line region per tile issues the scores of tile it+1 on
  // the matrix cores, the exponentials of tile it on the vector ALUs and O += V P for
  // tile it, interleaved (sched_group_barrier); the running-max decision for tile it+1
  // closes the region, so the only branch (the rare rescale) sits between tiles.
  // Lazy rescale (online softmax, log2 domain).  Each lane owns one query; the partner
  // lane l^32 holds the other half of its keys.  The running maximum is raised only
  // when a row's new scores exceed it by more than kTau, so probabilities stay below
  // 2^kTau and the rescale of the accumulator -- a wave-uniform branch -- is rare.
  // mx: this lane's maximum of the tile's s - m_eff; sc: the tile's scores (s - m_eff,
  // log2 units), shifted here to the new maximum.
  auto rescale = [&](float mx, f32x16* sc) __attribute__((always_inline)) {
    const float mx2 = pair_max(mx);
    if (__builtin_amdgcn_ballot_w64(mx2 > thr)) {
      const float m_new = fmaxf(m_run, m_eff + mx2);
      const float m_new_eff = (m_new == -INFINITY) ? 0.f : m_new;
      const float alpha = (m_run == -INFINITY) ? 0.f : fast_exp2(m_run - m_new);
      const float delta = m_new_eff - m_eff;
      l_run *= alpha;
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
        for (int i = 0; i < 16; ++i) oacc[dt][i] *= alpha;
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int i = 0; i < 16; ++i) sc[mt][i] -= delta;
      m_run = m_new;
      m_eff = m_new_eff;
      thr = (m_new == -INFINITY) ? -INFINITY : kTau;
#pragma unroll
      for (int i = 0; i < 16; ++i) minit[i] = -m_eff * isl2;
    }
  };
  auto scale_half = [&](f32x16* sc, int mt) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < 16; ++i) sc[mt][i] *= sl2;
  };
  auto decide = [&](f32x16* sc) __attribute__((always_inline)) {
    float mx = -INFINITY;
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
      for (int i = 0; i < 16; ++i) mx = fmaxf(mx, sc[mt][i]);
    rescale(mx, sc);
  };
  auto mask_half = [&](f32x16* sc, int mt, int it) __attribute__((always_inline)) {
    const int kpos0 = hs.k_pos0 + it * kBN;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int kpos = kpos0 + 32 * mt + 16 * (i >> 3) + 8 * hi + (i & 7);
      if (kpos > qpos) sc[mt][i] = -INFINITY;
    }
  };
  auto mask = [&](f32x16* sc, int it) __attribute__((always_inline)) {
    const int kpos0 = hs.k_pos0 + it * kBN;
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int kpos = kpos0 + 32 * mt + 16 * (i >> 3) + 8 * hi + (i & 7);
        if (kpos > qpos) sc[mt][i] = -INFINITY;
      }
  };
  // P = exp2(s log2e/sqrt(D) - m) in bf16 and O^T += V^T P^T for one tile
  auto softmax_pv = [&](const f32x16* sc, const bf16* vt) __attribute__((always_inline)) {
    float rsum = 0.f;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      u32x4 w;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float p0 = fast_exp2(sc[kb >> 1][8 * (kb & 1) + 2 * j]);
        const float p1 = fast_exp2(sc[kb >> 1][8 * (kb & 1) + 2 * j + 1]);
        w[j] = pack_bf16x2(p0, p1);
        rsum = dot2_bf16_ones(w[j], rsum);  // row sum of the bf16 probabilities used
      }
      const bf16x8 pb = __builtin_bit_cast(bf16x8, w);
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) {
        const bf16x4 lo = lds_read_tr16(vt + 16 * kb * D + voff[0][dt]);
        const bf16x4 up = lds_read_tr16(vt + 16 * kb * D + voff[1][dt]);
        const bf16x8 a = {lo[0], lo[1], lo[2], lo[3], up[0], up[1], up[2], up[3]};
        oacc[dt] = mfma32(a, pb, oacc[dt]);
      }
    }
    l_run += rsum;
  };

  if (nt > 0) {
    load_k(0, I0{});
    load_v(0, I0{});
    if (nt > 1) load_k(1, I1{});
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  f32x16 s_cur[2];
  if (nt > 0) {
    scores(sK0, s_cur);
    scale_half(s_cur, 0);
    scale_half(s_cur, 1);
    if (n_full == 0) mask(s_cur, 0);
    decide(s_cur);
  }
  // the first loop step reloads the buffer of K tile 0: every wave must have read it
  if (nt > 2) __syncthreads();

  // tile it with a successor; B = it & 1 at compile time, MN: tile it+1 needs the mask.
  // The region is laid out by hand in 20 steps separated by scheduling fences: step s
  // issues the LDS reads of the operands kPF steps ahead, the score MFMA s of tile it+1
  // (s < 16), the O += V P MFMA s-4 of tile it (s >= 4), and a quarter of the exponentials
  // of one 16-key group of tile it (s < 16; group g is consumed from step 4g + 4 on) or
  // part of the next row maximum (s >= 16).
  auto body_sched = [&](auto Bc, auto Mc, int it) __attribute__((always_inline)) {
    constexpr int B = decltype(Bc)::value;
    constexpr bool MN = decltype(Mc)::value;
    static_assert(NKK == 8 && NDT == 4, "hand schedule written for D = 128");
    if (it + 2 < nt) load_k(it + 2, Bc);
    load_v(it + 1, std::integral_constant<int, B ^ 1>{});
    const bf16* kt = kbuf(std::integral_constant<int, B ^ 1>{});
    const bf16* vt = vbuf(Bc);
    f32x16 s_next[2];
    bf16x8 kop[16], vop[16], pb[4];
    uint32_t w[4][4];
    float rs2[4] = {0.f, 0.f, 0.f, 0.f};
    float mxa = -INFINITY, mxb = -INFINITY;
    // score MFMA S: the two 32-key halves alternate (mt = S % 2, kk = S / 2), so that
    // consecutive score MFMAs are independent
    auto read_k = [&](auto Sc) __attribute__((always_inline)) {
      constexpr int S = decltype(Sc)::value;
      kop[S] = *(const bf16x8*)(kt + 32 * (S % 2) * D + koff[S / 2]);
    };
    auto read_v = [&](auto Sc) __attribute__((always_inline)) {
      constexpr int S = decltype(Sc)::value;  // PV MFMA S: kb = S / NDT, dt = S % NDT
      const bf16x4 lo = lds_read_tr16(vt + 16 * (S / NDT) * D + voff[0][S % NDT]);
      const bf16x4 up = lds_read_tr16(vt + 16 * (S / NDT) * D + voff[1][S % NDT]);
      vop[S] = bf16x8{lo[0], lo[1], lo[2], lo[3], up[0], up[1], up[2], up[3]};
    };
    // 21 steps.  Step S: score MFMA S (S < 16); PV MFMA S - 5 (S >= 5); the exponentials of
    // pair S (S < 16), the bf16 packing of pair S - 1 and the row-sum update of pair S - 2,
    // so that no step waits on a result of its own; the next tile's masking and maximum
    // from step 16 on (the last score MFMAs issue at steps 14 and 15).
    float pe0[16], pe1[16];
    constexpr int kPVD = 5;
    static_for<0, kPF>([&](auto Sc) __attribute__((always_inline)) { read_k(Sc); });
    static_for<0, 16 + kPVD>([&](auto Sc) __attribute__((always_inline)) {
      constexpr int S = decltype(Sc)::value;
      if constexpr (S + kPF < 16) read_k(std::integral_constant<int, S + kPF>{});
      if constexpr (S + kPF >= kPVD && S + kPF < 16 + kPVD) read_v(std::integral_constant<int, S + kPF - kPVD>{});
      if constexpr (S < 16) {
        constexpr int mt = S % 2, kk = S / 2;
        s_next[mt] = mfma32(kop[S], qreg[kk], kk == 0 ? minit : s_next[mt]);
      }
      if constexpr (S >= kPVD) {
        constexpr int q = S - kPVD, kb = q / NDT, dt = q % NDT;
        if constexpr (dt == 0) pb[kb] = __builtin_bit_cast(bf16x8, u32x4{w[kb][0], w[kb][1], w[kb][2], w[kb][3]});
        oacc[dt] = mfma32(vop[q], pb[kb], oacc[dt]);
      }
      if constexpr (S < 16) {
        constexpr int kb = S / 4, j = S % 4;
        pe0[S] = fast_exp2(s_cur[kb >> 1][8 * (kb & 1) + 2 * j]);
        pe1[S] = fast_exp2(s_cur[kb >> 1][8 * (kb & 1) + 2 * j + 1]);
      }
      if constexpr (S >= 1 && S <= 16) {
        constexpr int P = S - 1;
        w[P / 4][P % 4] = pack_bf16x2(pe0[P], pe1[P]);
      }
      if constexpr (S >= 2 && S <= 17) {
        constexpr int P = S - 2;
        rs2[P % 4] = dot2_bf16_ones(w[P / 4][P % 4], rs2[P % 4]);  // row sum of the bf16 probabilities used
      }
      if constexpr (S == 16 || S == 17) {
        if constexpr (S == 16) scale_half(s_next, 0);
        if constexpr (S == 16 && MN) mask_half(s_next, 0, it + 1);
#pragma unroll
        for (int i = 8 * (S - 16); i < 8 * (S - 15); ++i) mxa = fmaxf(mxa, s_next[0][i]);
      } else if constexpr (S >= 18) {
        if constexpr (S == 18) scale_half(s_next, 1);
        if constexpr (S == 18 && MN) mask_half(s_next, 1, it + 1);
        if constexpr (S < 20) {
#pragma unroll
          for (int i = 8 * (S - 18); i < 8 * (S - 17); ++i) mxb = fmaxf(mxb, s_next[1][i]);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    });
    l_run += (rs2[0] + rs2[1]) + (rs2[2] + rs2[3]);
    rescale(fmaxf(mxa, mxb), s_next);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // tiles it+1 (V) and it+2 (K) landed
    __syncthreads();
    s_cur[0] = s_next[0];
    s_cur[1] = s_next[1];
  };
  // other head dims: the same work, ordered by the compiler
  auto body_plain = [&](auto Bc, auto Mc, int it) __attribute__((always_inline)) {
    constexpr int B = decltype(Bc)::value;
    constexpr bool MN = decltype(Mc)::value;
    if (it + 2 < nt) load_k(it + 2, Bc);
    load_v(it + 1, std::integral_constant<int, B ^ 1>{});
    f32x16 s_next[2];
    scores(kbuf(std::integral_constant<int, B ^ 1>{}), s_next);
    scale_half(s_next, 0);
    scale_half(s_next, 1);
    softmax_pv(s_cur, vbuf(Bc));
    if (MN) mask(s_next, it + 1);
    decide(s_next);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    s_cur[0] = s_next[0];
    s_cur[1] = s_next[1];
  };
  auto body = [&](auto Bc, auto Mc, int it) __attribute__((always_inline)) {
    if constexpr (D == 128)
      body_sched(Bc, Mc, it);
    else
      body_plain(Bc, Mc, it);
  };
  // tiles [a, e) that have successors, two at a time so that B is a constant
  auto run = [&](auto Mc, int a, int e) __attribute__((always_inline)) {
    int it = a;
    if ((it & 1) && it < e) body(std::integral_constant<int, 1>{}, Mc, it++);
    for (; it + 1 < e; it += 2) {
      body(std::integral_constant<int, 0>{}, Mc, it);
      body(std::integral_constant<int, 1>{}, Mc, it + 1);
    }
    if (it < e) body(std::integral_constant<int, 0>{}, Mc, it);
  };
  if (nt > 0) {
    const int split = max(0, min(nt - 1, n_full - 1));  // from here on tile it+1 is masked
    run(std::false_type{}, 0, split);
    run(std::true_type{}, split, nt - 1);
    // last tile: no successor
    if ((nt - 1) & 1)
      softmax_pv(s_cur, sV1);
    else
      softmax_pv(s_cur, sV0);
  }

  // ---- end of step: finalise or save the running state -------------------------------
  const float l_tot = pair_sum(l_run);
  if (hs.flags & kLast) {
    const float inv = 1.f / l_tot;
    bf16* orow = (bf16*)p.o + (long long)b * p.q_bstride + (long long)qr * rs + h * D;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int d = 32 * dt + 8 * g + 4 * hi;
        u32x2 w = {pack_bf16x2(oacc[dt][4 * g] * inv, oacc[dt][4 * g + 1] * inv),
                   pack_bf16x2(oacc[dt][4 * g + 2] * inv, oacc[dt][4 * g + 3] * inv)};
        *(u32x2*)(orow + d) = w;
      }
    if (!hi) p.lse[st_row] = m_run * kLn2 + logf(l_tot);
  } else {
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const f32x4 t = {oacc[dt][4 * g], oacc[dt][4 * g + 1], oacc[dt][4 * g + 2], oacc[dt][4 * g + 3]};
        ((f32x4*)acc_tile)[((wave * NDT + dt) * 4 + g) * 64 + lane] = t;
      }
    if (!hi) {
      p.m[st_row] = m_run;
      p.l[st_row] = l_tot;
    }
  }

  // ---- send: rows 128 qt .. 128 qt + 127 of (b, h) of this host's block to the host
  // that needs the block at the next step (the ring's exchange, done by the workgroups
  // as they finish instead of by copies between the steps)
  const int fto = p.fwd.to[slot] - 1;  // destination slot, or -1
  if (fto >= 0 && p.fwd.k0 != nullptr && p.fwd.v0 != nullptr) {
    constexpr int PER = kBM * CPR / kThreads;  // 16-byte chunks per thread per operand
    const long long doff = (long long)fto * p.fwd.blk_bytes + 2 * ((long long)b * p.c * rs + h * D);
    bf16* kdst = (bf16*)((char*)p.fwd.k0 + doff);
    bf16* vdst = (bf16*)((char*)p.fwd.v0 + doff);
    u32x4 kx[PER], vx[PER];
#pragma unroll
    for (int e = 0; e < PER; ++e) {
      const int idx = e * kThreads + tid;
      const long long off = (long long)(qt * kBM + idx / CPR) * rs + 8 * (idx % CPR);
      kx[e] = *(const u32x4*)(kbase + off);
      vx[e] = *(const u32x4*)(vbase + off);
    }
#pragma unroll
    for (int e = 0; e < PER; ++e) {
      const int idx = e * kThreads + tid;
      const long long off = (long long)(qt * kBM + idx / CPR) * rs + 8 * (idx % CPR);
      *(u32x4*)(kdst + off) = kx[e];
      *(u32x4*)(vdst + off) = vx[e];
    }
  }
}

// ===================================================================================
// float32 kernel (exact float32 arithmetic, no matrix cores): one thread per query,
// 64 queries per workgroup, 32-key tiles staged in LDS.  Natural-log state.
// ===================================================================================
constexpr int kF32BM = 64, kF32BN = 32;

template <int D>
__global__ __launch_bounds__(64) void fwd_f32_kernel(const FwdStep p) {
  __shared__ float sK[kF32BN * D];
  __shared__ float sV[kF32BN * D];
  const int n_qt = p.c / kF32BM;
  const int BH = p.B * p.H;
  const int total = p.n_slots * BH * n_qt;
  const int L = blockIdx.x;
  if (L >= total) return;
  const int grp = L / n_qt, qt = L % n_qt;
  const int slot = grp / BH, bh = grp % BH;
  const int b = bh / p.H, h = bh % p.H;
  const StepHost hs = p.host[slot];
  const int t = threadIdx.x;
  const int rs = p.H * D;
  const int qr = hs.q_row0 + qt * kF32BM + t;
  const int qpos = hs.q_pos0 + qt * kF32BM + t;
  const long long st_row = (long long)bh * p.Sq + qr;

  const float* qrow = (const float*)p.q + (long long)b * p.q_bstride + (long long)qr * rs + h * D;
  const float* kbase = (const float*)hs.k + (long long)b * hs.kv_bstride + h * D;
  const float* vbase = (const float*)hs.v + (long long)b * hs.kv_bstride + h * D;
  float* accrow = p.acc + st_row * D;

  float q[D], acc[D];
  #pragma unroll
  for (int d = 0; d < D; ++d) q[d] = qrow[d];
  float m_run, l_run;
  if (hs.flags & kFirst) {
    #pragma unroll
    for (int d = 0; d < D; ++d) acc[d] = 0.f;
    m_run = -INFINITY;
    l_run = 0.f;
  } else {
    #pragma unroll
    for (int d = 0; d < D; ++d) acc[d] = accrow[d];
    m_run = p.m[st_row];
    l_run = p.l[st_row];
  }

  int nt = p.c / kF32BN;
  if (p.causal) {
    const int vis = hs.q_pos0 + qt * kF32BM + kF32BM - hs.k_pos0;
    nt = min(nt, max(0, (vis + kF32BN - 1) / kF32BN));
  }
  for (int it = 0; it < nt; ++it) {
    __syncthreads();
    for (int e = t; e < kF32BN * D; e += 64) {
      const int r = e / D, d = e % D;
      const long long off = (long long)(it * kF32BN + r) * rs + d;
      sK[e] = kbase[off];
      sV[e] = vbase[off];
    }
    __syncthreads();
    float s[kF32BN];
    float mx = -INFINITY;
    #pragma unroll
    for (int j = 0; j < kF32BN; ++j) {
      float dot = 0.f;
      #pragma unroll
      for (int d = 0; d < D; ++d) dot = fmaf(q[d], sK[j * D + d], dot);
      const int kpos = hs.k_pos0 + it * kF32BN + j;
      s[j] = (p.causal && kpos > qpos) ? -INFINITY : dot * p.scale;
      mx = fmaxf(mx, s[j]);
    }
    const float m_new = fmaxf(m_run, mx);
    const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
    const float alpha = expf(m_run - m_use);
    m_run = m_new;
    l_run *= alpha;
    #pragma unroll
    for (int d = 0; d < D; ++d) acc[d] *= alpha;
    #pragma unroll
    for (int j = 0; j < kF32BN; ++j) {
      const float pj = expf(s[j] - m_use);
      l_run += pj;
      #pragma unroll
      for (int d = 0; d < D; ++d) acc[d] = fmaf(pj, sV[j * D + d], acc[d]);
    }
  }
  if (hs.flags & kLast) {
    float* orow = (float*)p.o + (long long)b * p.q_bstride + (long long)qr * rs + h * D;
    #pragma unroll
    for (int d = 0; d < D; ++d) orow[d] = acc[d] / l_run;
    p.lse[st_row] = m_run + logf(l_run);
  } else {
    #pragma unroll
    for (int d = 0; d < D; ++d) accrow[d] = acc[d];
    p.m[st_row] = m_run;
    p.l[st_row] = l_run;
  }
}

}  // namespace

hipError_t launch_fwd_bf16(const FwdStep& s, int D, hipStream_t st) {
  const int total = s.n_slots * s.B * s.H * (s.c / kBM);
  if (total == 0) return hipSuccess;
  // a forwarding destination needs both receive bases and a slot size
  for (int n = 0; n < s.n_slots; ++n)
    if (s.fwd.to[n] != 0 && (s.fwd.to[n] < 0 || s.fwd.k0 == nullptr || s.fwd.v0 == nullptr || s.fwd.blk_bytes <= 0))
      return hipErrorInvalidValue;
  if (D == 128)
    hipLaunchKernelGGL(fwd_bf16_kernel<128>, dim3(total), dim3(kThreads), 0, st, s);
  else
    hipLaunchKernelGGL(fwd_bf16_kernel<64>, dim3(total), dim3(kThreads), 0, st, s);
  return hipGetLastError();
}

hipError_t launch_fwd_f32(const FwdStep& s, int D, hipStream_t st) {
  const int total = s.n_slots * s.B * s.H * (s.c / kF32BM);
  if (total == 0) return hipSuccess;
  if (D == 128)
    hipLaunchKernelGGL(fwd_f32_kernel<128>, dim3(total), dim3(64), 0, st, s);
  else
    hipLaunchKernelGGL(fwd_f32_kernel<64>, dim3(total), dim3(64), 0, st, s);
  return hipGetLastError();
}

}  // namespace ra
