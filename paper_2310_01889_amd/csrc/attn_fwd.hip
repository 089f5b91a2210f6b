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
// bf16 kernel: NW = 4 or 8 waves, 32 queries per wave (128 or 256 per workgroup), 64-key
// tiles.
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
constexpr float kSumMax = 65536.f;  // overflow test: a lane's row sum over a tile below this


// LDS tiles are unpadded [64 rows][D] with the 16-byte chunks of each row permuted by
// an XOR swizzle, so that every read pattern below is free of bank conflicts:
//   * row reads (A operand of S^T): 16 lanes read 16 consecutive rows at one chunk;
//   * transpose reads (V^T): 16 lanes read 4 consecutive rows x 32 contiguous bytes.
// For D = 128 (16 chunks per row): chunk c of row r lives at c ^ (4 (r & 3) + ((r >> 2) & 3));
// for D = 64 (8 chunks, two rows per 256-byte bank sweep) at c ^ s, s = (r >> 1) & 7 with
// bit 2 flipped on odd s.  Tiles are filled with direct-to-LDS loads (no registers):
// lane i of a 1 KB load lands at byte 16 i of its destination, so each lane fetches the
// logical chunk that the swizzle puts there.
template <int D, int NW>
__global__ __launch_bounds__(64 * NW, NW == 4 ? 2 : 1) void fwd_bf16_kernel(const FwdStep p) {
  constexpr int BM = 32 * NW;  // queries per workgroup (32 per wave)
  constexpr int NT = 64 * NW;  // threads per workgroup
  constexpr int NKK = D / 16;  // 16-wide reduction steps of q.k
  constexpr int NDT = D / 32;  // 32-row output tiles of O^T
  constexpr int CPR = D / 8;   // 16-byte chunks per row
  constexpr int ROWS_PER_LOAD = 64 / CPR;               // rows filled by one 1 KB wave load
  constexpr int RPW = kBN / NW;                          // tile rows each wave fills
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

  const int n_qt = p.c / BM;
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

  const int q_tile_row = hs.q_row0 + qt * BM;       // first q-space row of the workgroup
  const int qr = q_tile_row + wave * 32 + l32;       // this lane's query row
  const int qpos = hs.q_pos0 + qt * BM + wave * 32 + l32;
  const int tile_first_q = hs.q_pos0 + qt * BM;

  const bf16* qbase = (const bf16*)p.q + (long long)b * p.q_bstride + h * D;
  const bf16* kbase = (const bf16*)hs.k + (long long)b * hs.kv_bstride + h * D;
  const bf16* vbase = (const bf16*)hs.v + (long long)b * hs.kv_bstride + h * D;

  // key tiles with at least one visible key; the first n_full need no mask
  int nt = p.c / kBN, n_full = nt;
  if (p.causal) {
    const int vis = tile_first_q + BM - hs.k_pos0;  // keys visible to the last row
    nt = min(nt, max(0, (vis + kBN - 1) / kBN));
    n_full = min(nt, max(0, (tile_first_q - hs.k_pos0 + 1) / kBN));
  }

  // ---- running state -------------------------------------------------------------
  f32x16 oacc[NDT];
  float m_run, l_run;
  const long long st_row = (long long)bh * p.Sq + qr;
  float* acc_tile = p.acc + ((long long)bh * (p.Sq / BM) + q_tile_row / BM) * (BM * D);
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
  // score, fused with the subtraction of the running maximum: x = fma(q.k, sl2, -m_eff).
  const float sl2 = p.scale * kLog2e;
  bf16x8 qreg[NKK];
  {
    const bf16* qrow = qbase + (long long)qr * rs;
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) qreg[kk] = *(const bf16x8*)(qrow + 16 * kk + 8 * hi);
  }
  // Running maximum without a per-tile maximum.  m_eff = the running maximum in log2 units
  // (0 while it is still -inf); the probabilities of a tile are formed against it, and the
  // tile's exact maximum is taken -- m raised, O^T and l rescaled, the probabilities formed
  // again -- only when a lane's row sum over the tile is not below kSumMax (or not finite),
  // or while m is still -inf (thrs = -1).  Every probability that reaches the products is
  // thus at most kSumMax, which bf16 and float32 hold exactly in range; the offset cancels
  // in o and is carried in lse.
  float m_eff = (m_run == -INFINITY) ? 0.f : m_run;
  float thrs = (m_run == -INFINITY) ? -1.f : kSumMax;
  const f32x16 zero16 = {};

  // ---- direct-to-LDS staging: each wave fills RPW rows of a tile ---------------------
  // load j of wave w covers rows j * NW ROWS_PER_LOAD + w ROWS_PER_LOAD + lane / CPR; the
  // lane's physical chunk is lane % CPR, its logical (global) chunk that ^ swz(row).  With
  // rows interleaved over the waves this way, swz(row) is the same for all loads of a lane
  // (the row bits it reads do not depend on j), so every load of the lane reads at one
  // byte offset goff plus a wave-uniform j * 2 NW ROWS_PER_LOAD * rs bytes.
  static_assert(RPW == LOADS * ROWS_PER_LOAD, "each wave fills LOADS row groups");
  const int goff = 2 * ((wave * ROWS_PER_LOAD + lane / CPR) * rs +
                        8 * ((lane % CPR) ^ swz<D>(wave * ROWS_PER_LOAD + lane / CPR)));
  // buffer loads with the LDS flag: the tile base is a wave-uniform descriptor, so the
  // per-tile address update is scalar work; reads past the tile return zero
  auto dload = [&](const bf16* src_tile, bf16* dst_tile) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < LOADS; ++j)
      buffer_load_lds16_so(src_tile, kBN * rs * 2, dst_tile + (j * NW + wave_u) * ROWS_PER_LOAD * D, goff,
                           j * 2 * NW * ROWS_PER_LOAD * rs);
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

  // ---- three-stage tile pipeline -----------------------------------------------------
  // Region t (one straight-line stretch of code per tile): the score products of tile t+1
  // (into s_nx), the exponentials of tile t (from s_cur, into the packed probabilities w)
  // and O^T += V^T P^T of tile t-1 (from pprev), interleaved step by step; the overflow
  // test of tile t closes the region, so that the only branch (the rare exact path) sits
  // between regions and tile t's probabilities are known good before tile t+1's region
  // multiplies them into O^T.  K runs one tile ahead of the scores, V one tile behind.
  // Region t reads K(t+1) and V(t-1) from buffer (t+1) % 2 and loads K(t+2), V(t) into
  // buffer t % 2.
  constexpr int NS = 2 * NKK;    // score products per tile (two 32-key halves)
  constexpr int NP = 4 * NDT;    // PV products per tile (four 16-key groups)
  constexpr int NSTEP = NS + NP;
  constexpr int PF = 2;          // operand reads issued this many steps ahead
  static_assert(NS == NP, "as many score as PV products per tile");
  f32x16 s_cur[2], s_nx[2];      // raw q.k of tiles t and t+1 (masked keys -inf)
  bf16x8 pprev[4];               // P^T of tile t-1, four 16-key groups
  float l_tile = 0.f;            // this lane's row sum of tile t's probabilities

  auto mask_tile = [&](f32x16* sc, int it) __attribute__((always_inline)) {
    const int kpos0 = hs.k_pos0 + it * kBN;
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int kpos = kpos0 + 32 * mt + 16 * (i >> 3) + 8 * hi + (i & 7);
        if (kpos > qpos) sc[mt][i] = -INFINITY;
      }
  };
  // probabilities of pair u (keys 2u, 2u+1 of this lane's 32) of a tile, packed bf16
  auto expo_pair = [&](const f32x16* sc, int u) __attribute__((always_inline)) -> uint32_t {
    const int kb = u / 4, jj = u % 4, i0 = 8 * (kb & 1) + 2 * jj;
    return pack_bf16x2(fast_exp2(fmaf(sc[kb >> 1][i0], sl2, -m_eff)), fast_exp2(fmaf(sc[kb >> 1][i0 + 1], sl2, -m_eff)));
  };
  // exact path of a tile whose probabilities failed the test: its maximum, the rescale of
  // the state, the probabilities again (w, l_tile)
  auto exact = [&](const f32x16* sc, uint32_t* w) __attribute__((always_inline)) {
    float mx = -INFINITY;
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
      for (int i = 0; i < 16; ++i) mx = fmaxf(mx, sc[mt][i]);
    const float mx2 = pair_max(mx) * sl2;  // masked keys -inf; every scale positive
    const float m_new = fmaxf(m_run, mx2);
    const float alpha = (m_run == -INFINITY) ? 0.f : fast_exp2(m_run - m_new);
    l_run *= alpha;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int i = 0; i < 16; ++i) oacc[dt][i] *= alpha;
    m_run = m_new;
    m_eff = (m_new == -INFINITY) ? 0.f : m_new;
    thrs = (m_new == -INFINITY) ? -1.f : kSumMax;
    float r0 = 0.f, r1 = 0.f;
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      w[u] = expo_pair(sc, u);
      if (u & 1) r1 = dot2_bf16_ones(w[u], r1); else r0 = dot2_bf16_ones(w[u], r0);
    }
    l_tile = r0 + r1;
  };
  // end of region: the test, then the tile's probabilities become pprev
  auto close_tile = [&](const f32x16* sc, uint32_t* w) __attribute__((always_inline)) {
    if (__builtin_amdgcn_ballot_w64(!(l_tile < thrs))) exact(sc, w);
    l_run += l_tile;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) pprev[kb] = __builtin_bit_cast(bf16x8, u32x4{w[4 * kb], w[4 * kb + 1], w[4 * kb + 2], w[4 * kb + 3]});
  };

  // Region t.  Bc = t % 2 (buffer loaded), NX: tile t+1 exists, PV: tile t-1 exists, MC:
  // tile t needs the causal mask.  Step s issues MFMA s -- the PV products of tile t-1 in
  // the first half of the region, the score products of tile t+1 in the second, so that
  // the probabilities of tile t-1 and the scores of tile t+1 are never live together --,
  // operand reads PF steps ahead, and the vector work of pair u = s * 16 / NSTEP of tile t:
  // its exponentials at that step, its packing one step later, its row-sum term two steps
  // later.
  auto region = [&](auto Bc, auto NXc, auto PVc, auto MCc, int it, bool RTMASK = false) __attribute__((always_inline)) {
    constexpr int B = decltype(Bc)::value;
    constexpr bool NX = decltype(NXc)::value, PV = decltype(PVc)::value, MC = decltype(MCc)::value;
    if (NX && it + 2 < nt) load_k(it + 2, Bc);
    load_v(it, Bc);  // read by region t+1 or, after the last region, by the final products
    const bf16* kt = kbuf(std::integral_constant<int, B ^ 1>{});
    const bf16* vt = vbuf(std::integral_constant<int, B ^ 1>{});
    if constexpr (MC) mask_tile(s_cur, it);
    if constexpr (!MC) {
      if (RTMASK && it >= n_full) mask_tile(s_cur, it);
    }
    bf16x8 kop[NS], vop[NP];
    uint32_t w[16];
    float pe[16][2];
    float rs2[4] = {0.f, 0.f, 0.f, 0.f};
    auto fetch = [&](auto Sc) __attribute__((always_inline)) {
      constexpr int S = decltype(Sc)::value;
      if constexpr (S >= NP) {
        constexpr int I = S - NP;  // score product I: key half I % 2, dims 16 (I / 2)..
        if constexpr (NX) kop[I] = *(const bf16x8*)(kt + 32 * (I % 2) * D + koff[I / 2]);
      } else {
        constexpr int Q = S;  // PV product Q: keys 16 (Q / NDT).., dims 32 (Q % NDT)..
        if constexpr (PV) {
          const bf16x4 lo = lds_read_tr16(vt + 16 * (Q / NDT) * D + voff[0][Q % NDT]);
          const bf16x4 up = lds_read_tr16(vt + 16 * (Q / NDT) * D + voff[1][Q % NDT]);
          vop[Q] = bf16x8{lo[0], lo[1], lo[2], lo[3], up[0], up[1], up[2], up[3]};
        }
      }
    };
    constexpr int UPS = NSTEP / 16;  // steps per probability pair
    static_for<0, PF>([&](auto Sc) __attribute__((always_inline)) { fetch(Sc); });
    static_for<0, NSTEP + 2 * UPS>([&](auto Sc) __attribute__((always_inline)) {
      constexpr int S = decltype(Sc)::value;
      if constexpr (S + PF < NSTEP) fetch(std::integral_constant<int, S + PF>{});
      if constexpr (S < NSTEP && S >= NP) {
        constexpr int I = S - NP, mt = I % 2, kk = I / 2;
        if constexpr (NX) s_nx[mt] = mfma32(kop[I], qreg[kk], kk == 0 ? zero16 : s_nx[mt]);
      } else if constexpr (S < NP) {
        constexpr int Q = S;
        if constexpr (PV) oacc[Q % NDT] = mfma32(vop[Q], pprev[Q / NDT], oacc[Q % NDT]);
      }
      if constexpr (S % UPS == 0 && S / UPS < 16) {
        constexpr int u = S / UPS, kb = u / 4, jj = u % 4, i0 = 8 * (kb & 1) + 2 * jj;
        pe[u][0] = fast_exp2(fmaf(s_cur[kb >> 1][i0], sl2, -m_eff));
        pe[u][1] = fast_exp2(fmaf(s_cur[kb >> 1][i0 + 1], sl2, -m_eff));
      }
      if constexpr (S % UPS == 0 && S / UPS >= 1 && S / UPS <= 16) {
        constexpr int u = S / UPS - 1;
        w[u] = pack_bf16x2(pe[u][0], pe[u][1]);
      }
      if constexpr (S % UPS == 0 && S / UPS >= 2 && S / UPS <= 17) {
        constexpr int u = S / UPS - 2;
        rs2[u % 4] = dot2_bf16_ones(w[u], rs2[u % 4]);  // row sum of the bf16 probabilities used
      }
      __builtin_amdgcn_sched_barrier(0);
    });
    l_tile = (rs2[0] + rs2[1]) + (rs2[2] + rs2[3]);
    close_tile(s_cur, w);
    if constexpr (NX) {
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // K(t+2) and V(t) landed
      __syncthreads();
      s_cur[0] = s_nx[0];
      s_cur[1] = s_nx[1];
    }
  };

  // regions [a, e) that have a successor and a predecessor, two at a time so that the
  // buffer parity is a constant; MC: their tiles need the mask
  auto run = [&](auto MCc, int a, int e) __attribute__((always_inline)) {
    int it = a;
    if ((it & 1) && it < e) region(std::integral_constant<int, 1>{}, std::true_type{}, std::true_type{}, MCc, it++);
    for (; it + 1 < e; it += 2) {
      region(std::integral_constant<int, 0>{}, std::true_type{}, std::true_type{}, MCc, it);
      region(std::integral_constant<int, 1>{}, std::true_type{}, std::true_type{}, MCc, it + 1);
    }
    if (it < e) region(std::integral_constant<int, 0>{}, std::true_type{}, std::true_type{}, MCc, it);
  };
  // the last region (no successor): one instance for any parity, mask and predecessor,
  // its two buffers chosen at run time (the compiler then waits for the in-flight load of
  // V(t) before reading V(t-1) from the other buffer: once per workgroup)
  auto last = [&](int it) __attribute__((always_inline)) {
    if (it >= n_full) mask_tile(s_cur, it);
    bf16* vld = (it & 1) ? sV1 : sV0;
    const bf16* vt = (it & 1) ? sV0 : sV1;
    dload(vbase + (long long)it * kBN * rs, vld);  // V(t) for the final products
    uint32_t w[16];
    float r0 = 0.f, r1 = 0.f;
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      w[u] = expo_pair(s_cur, u);
      if (u & 1) r1 = dot2_bf16_ones(w[u], r1); else r0 = dot2_bf16_ones(w[u], r0);
    }
    if (it > 0) {
#pragma unroll
      for (int q = 0; q < NP; ++q) {
        const bf16x4 lo = lds_read_tr16(vt + 16 * (q / NDT) * D + voff[0][q % NDT]);
        const bf16x4 up = lds_read_tr16(vt + 16 * (q / NDT) * D + voff[1][q % NDT]);
        oacc[q % NDT] = mfma32(bf16x8{lo[0], lo[1], lo[2], lo[3], up[0], up[1], up[2], up[3]}, pprev[q / NDT], oacc[q % NDT]);
      }
    }
    l_tile = r0 + r1;
    close_tile(s_cur, w);
  };

  if (nt > 0) {
    // K(0) and K(1); the scores of tile 0
    load_k(0, std::integral_constant<int, 0>{});
    if (nt > 1) load_k(1, std::integral_constant<int, 1>{});
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
      s_cur[mt] = mfma32(*(const bf16x8*)(sK0 + 32 * mt * D + koff[0]), qreg[0], zero16);
#pragma unroll
      for (int kk = 1; kk < NKK; ++kk) s_cur[mt] = mfma32(*(const bf16x8*)(sK0 + 32 * mt * D + koff[kk]), qreg[kk], s_cur[mt]);
    }
    // region 0 loads K(2) into the buffer of K(0): every wave must have read it
    if (nt > 2) __syncthreads();
    if (nt > 1) {
      // region 0: no predecessor
      region(std::integral_constant<int, 0>{}, std::true_type{}, std::false_type{}, std::false_type{}, 0, true);
      const int split = max(1, min(nt - 1, n_full));  // regions from here on mask their tile
      run(std::false_type{}, 1, split);
      run(std::true_type{}, split, nt - 1);
    }
    last(nt - 1);
    // O^T += V^T P^T of the last tile, from V(nt-1) in buffer (nt-1) % 2
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    const bf16* vt = ((nt - 1) & 1) ? sV1 : sV0;
#pragma unroll
    for (int q = 0; q < NP; ++q) {
      const bf16x4 lo = lds_read_tr16(vt + 16 * (q / NDT) * D + voff[0][q % NDT]);
      const bf16x4 up = lds_read_tr16(vt + 16 * (q / NDT) * D + voff[1][q % NDT]);
      oacc[q % NDT] = mfma32(bf16x8{lo[0], lo[1], lo[2], lo[3], up[0], up[1], up[2], up[3]}, pprev[q / NDT], oacc[q % NDT]);
    }
  }

  // ---- end of step: finalise or save the running state -------------------------------
  // The per-lane indices are recomputed here from an opaque copy of the thread index, so
  // that none of them is kept live (or spilled) across the tile loop.
  int tid_e = threadIdx.x;
  asm volatile("" : "+v"(tid_e));
  const int lane_e = tid_e & 63, wave_e = tid_e >> 6, hi_e = lane_e >> 5;
  const int qr_e = q_tile_row + wave_e * 32 + (lane_e & 31);
  const long long st_row_e = (long long)bh * p.Sq + qr_e;
  const float l_tot = pair_sum(l_run);
  if (hs.flags & kLast) {
    const float inv = 1.f / l_tot;
    bf16* orow = (bf16*)p.o + (long long)b * p.q_bstride + (long long)qr_e * rs + h * D;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int d = 32 * dt + 8 * g + 4 * hi_e;
        u32x2 w = {pack_bf16x2(oacc[dt][4 * g] * inv, oacc[dt][4 * g + 1] * inv),
                   pack_bf16x2(oacc[dt][4 * g + 2] * inv, oacc[dt][4 * g + 3] * inv)};
        *(u32x2*)(orow + d) = w;
      }
    if (!hi_e) p.lse[st_row_e] = m_run * kLn2 + logf(l_tot);
  } else {
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const f32x4 t = {oacc[dt][4 * g], oacc[dt][4 * g + 1], oacc[dt][4 * g + 2], oacc[dt][4 * g + 3]};
        ((f32x4*)acc_tile)[((wave_e * NDT + dt) * 4 + g) * 64 + lane_e] = t;
      }
    if (!hi_e) {
      p.m[st_row_e] = m_run;
      p.l[st_row_e] = l_tot;
    }
  }

  // ---- send: rows 128 qt .. 128 qt + 127 of (b, h) of this host's block to the host
  // that needs the block at the next step (the ring's exchange, done by the workgroups
  // as they finish instead of by copies between the steps)
  const int fto = p.fwd.to[slot] - 1;  // destination slot, or -1
  if (fto >= 0 && p.fwd.k0 != nullptr && p.fwd.v0 != nullptr) {
    constexpr int PER = BM * CPR / NT;  // 16-byte chunks per thread per operand
    const long long doff = (long long)fto * p.fwd.blk_bytes + 2 * ((long long)b * p.c * rs + h * D);
    bf16* kdst = (bf16*)((char*)p.fwd.k0 + doff);
    bf16* vdst = (bf16*)((char*)p.fwd.v0 + doff);
    u32x4 kx[PER], vx[PER];
#pragma unroll
    for (int e = 0; e < PER; ++e) {
      const int idx = e * NT + tid_e;
      const long long off = (long long)(qt * BM + idx / CPR) * rs + 8 * (idx % CPR);
      kx[e] = *(const u32x4*)(kbase + off);
      vx[e] = *(const u32x4*)(vbase + off);
    }
#pragma unroll
    for (int e = 0; e < PER; ++e) {
      const int idx = e * NT + tid_e;
      const long long off = (long long)(qt * BM + idx / CPR) * rs + 8 * (idx % CPR);
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

// Long blocks (D = 128, at least 16384 keys, a multiple of 256) run the eight-wave kernel:
// 256 queries per workgroup, so each key/value tile is loaded once for twice the queries
// (one workgroup per CU instead of two; at 4096-8192 keys the longer start and end of each
// workgroup outweigh the saved loads).  The choice depends only on (D, c), so every step
// of a call uses the same kernel and the float32 state keeps one layout.
static bool fwd_bf16_wide(int D, int c) { return D == 128 && c % 256 == 0 && c >= 16384; }

hipError_t launch_fwd_bf16(const FwdStep& s, int D, hipStream_t st) {
  const int total = s.n_slots * s.B * s.H * (s.c / kBM);
  if (total == 0) return hipSuccess;
  const bool wide = fwd_bf16_wide(D, s.c);
  // a forwarding destination needs both receive bases and a slot size
  for (int n = 0; n < s.n_slots; ++n)
    if (s.fwd.to[n] != 0 && (s.fwd.to[n] < 0 || s.fwd.k0 == nullptr || s.fwd.v0 == nullptr || s.fwd.blk_bytes <= 0))
      return hipErrorInvalidValue;
  if (wide)
    hipLaunchKernelGGL((fwd_bf16_kernel<128, 8>), dim3(total / 2), dim3(512), 0, st, s);
  else if (D == 128)
    hipLaunchKernelGGL((fwd_bf16_kernel<128, 4>), dim3(total), dim3(kThreads), 0, st, s);
  else
    hipLaunchKernelGGL((fwd_bf16_kernel<64, 4>), dim3(total), dim3(kThreads), 0, st, s);
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
