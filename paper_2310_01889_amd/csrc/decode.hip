// Ring decode for gfx950: a few query tokens against a long key/value cache.
//
// The paper's appendix on the inference requirement applies ring attention to
// autoregressive decoding: the cache of S tokens stays split in n_hosts blocks of
// c = S / n_hosts tokens over the ring, the Tq newest tokens (the queries, one per
// generated token, at positions S - Tq .. S - 1 of the last host's block) see the blocks
// pass by in ring order -- the last host's own block first, then its predecessors'
// (Section 3) -- and each block is folded into the queries' running maximum, numerator
// and denominator (the online-softmax recurrence of Section 2).
//
// On one GPU every block is resident, so one launch computes the partial state of every
// block at once, each block split into chunks of `kch` keys for parallelism (one wave per
// (batch, head, chunk)): the step is a read of the whole cache, bound by HBM bandwidth.
// A second launch combines the partial states of each (batch, head, query) in ring
// order, block by block and, inside a block, chunk by chunk, and writes o and lse.
#include <mutex>

#include "ra_common.h"
#include "ra_runtime.h"
#include "ringattn.h"

namespace ra {
namespace {

constexpr int kDecKT = 32;      // keys per LDS tile
constexpr int kDecMaxQ = 32;    // query slots per wave
constexpr float kDecTau = 8.f;  // lazy-rescale threshold (log2 units)

struct DecodeArgs {
  const bf16* q;     // [B, Tq, H, D]
  const bf16* k;     // [B, S, H, D]
  const bf16* v;     // [B, S, H, D]
  float* part_acc;   // [B*H, nch, Tq, D]   unnormalised partial outputs
  float* part_m;     // [B*H, nch, Tq]      partial maxima (log2 units of the scaled scores)
  float* part_l;     // [B*H, nch, Tq]      partial denominators
  int B, H, S, Tq, kch, nch, causal;
  float scale;
};

// One wave: the partial state of all Tq queries (lane l % 32 = query slot) over the kch
// keys of one chunk.  The arithmetic per 32-key tile is that of the forward step kernel:
// S^T = K Q^T on the matrix cores (K rows from LDS with bits 2 and 3 of the row index
// swapped, Q as stored in registers, accumulators starting at minus the running maximum
// over the scale, which is applied in float32 before the maximum), lazy online softmax, O^T += V^T P^T with V^T read from LDS by
// the transpose read.  Tiles are double buffered: direct-to-LDS loads of tile it+1 are
// in flight while tile it is processed.  Lanes of slots >= Tq compute on zero queries
// and store nothing.
template <int D>
__global__ __launch_bounds__(64) void decode_partial_kernel(const DecodeArgs a) {
  constexpr int NKK = D / 16, NDT = D / 32, CPR = D / 8;
  constexpr int ROWS_PER_LOAD = 64 / CPR;        // rows filled by one 1 KB wave load
  constexpr int LOADS = kDecKT / ROWS_PER_LOAD;  // loads per operand tile
  constexpr int TILE = kDecKT * D;
  // separate objects per buffer: reads of one are known not to alias loads into the other
  __shared__ __attribute__((aligned(1024))) bf16 sK0[TILE];
  __shared__ __attribute__((aligned(1024))) bf16 sK1[TILE];
  __shared__ __attribute__((aligned(1024))) bf16 sV0[TILE];
  __shared__ __attribute__((aligned(1024))) bf16 sV1[TILE];
  auto pick = [](auto Bc, auto* x, auto* y) __attribute__((always_inline)) {
    if constexpr (decltype(Bc)::value == 0) return x; else return y;
  };

  const int ch = blockIdx.x % a.nch, bh = blockIdx.x / a.nch;
  const int b = bh / a.H, h = bh % a.H;
  const int lane = threadIdx.x, l32 = lane & 31, hi = lane >> 5;
  const int rs = a.H * D;
  const int t = l32;                   // query slot
  const int qpos = a.S - a.Tq + t;     // its global position (slots >= Tq: past the cache)
  const int k0 = ch * a.kch;
  const int nt = a.kch / kDecKT;

  // scores in log2 units: sl2 q.k, the products exact in float32 (the queries stay as
  // stored), the scale applied in float32
  const float sl2 = a.scale * kLog2e;
  const float isl2 = 1.f / sl2;
  bf16x8 qreg[NKK];
  {
    const bf16* qrow = a.q + ((long long)b * a.Tq + min(t, a.Tq - 1)) * rs + h * D;
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) {
      const bf16x8 x = *(const bf16x8*)(qrow + 16 * kk + 8 * hi);
#pragma unroll
      for (int e = 0; e < 8; ++e) qreg[kk][e] = t < a.Tq ? x[e] : (bf16)0.f;
    }
  }

  f32x16 oacc[NDT];
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
    for (int i = 0; i < 16; ++i) oacc[dt][i] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;
  float m_eff = 0.f, thr = -INFINITY;  // see the forward step kernel
  f32x16 minit;
#pragma unroll
  for (int i = 0; i < 16; ++i) minit[i] = 0.f;

  // direct-to-LDS staging of one 32-row tile by this wave
  int goff[LOADS];
#pragma unroll
  for (int j = 0; j < LOADS; ++j) {
    const int r = j * ROWS_PER_LOAD + lane / CPR;
    goff[j] = 2 * (r * rs + 8 * ((lane % CPR) ^ swz<D>(r)));
  }
  const bf16* kbase = a.k + ((long long)b * a.S + k0) * rs + h * D;
  const bf16* vbase = a.v + ((long long)b * a.S + k0) * rs + h * D;
  auto load_tile = [&](int it, auto Bc) __attribute__((always_inline)) {
    const long long off = (long long)it * kDecKT * rs;
#pragma unroll
    for (int j = 0; j < LOADS; ++j) {
      buffer_load_lds16(kbase + off, kDecKT * rs * 2, pick(Bc, sK0, sK1) + j * ROWS_PER_LOAD * D, goff[j]);
      buffer_load_lds16(vbase + off, kDecKT * rs * 2, pick(Bc, sV0, sV1) + j * ROWS_PER_LOAD * D, goff[j]);
    }
  };

  const int krow = swap_bits23(l32);
  int koff[NKK];
#pragma unroll
  for (int kk = 0; kk < NKK; ++kk) koff[kk] = krow * D + 8 * ((2 * kk + hi) ^ swz<D>(krow));
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

  auto tile = [&](auto Bc, int it) __attribute__((always_inline)) {
    // the previous tile's LDS reads have all returned before its buffer is refilled
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    if (it + 1 < nt) {
      load_tile(it + 1, std::integral_constant<int, decltype(Bc)::value ^ 1>{});
      asm volatile("s_waitcnt vmcnt(%0)" ::"n"(2 * LOADS) : "memory");  // tile it landed
    } else {
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    }
    const bf16* kt = pick(Bc, sK0, sK1);
    const bf16* vt = pick(Bc, sV0, sV1);
    f32x16 s = mfma32(*(const bf16x8*)(kt + koff[0]), qreg[0], minit);
#pragma unroll
    for (int kk = 1; kk < NKK; ++kk) s = mfma32(*(const bf16x8*)(kt + koff[kk]), qreg[kk], s);
#pragma unroll
    for (int i = 0; i < 16; ++i) s[i] *= sl2;  // s - m_eff, log2 units
    const int kpos0 = k0 + it * kDecKT;
    if (a.causal && kpos0 + kDecKT - 1 > a.S - a.Tq) {
#pragma unroll
      for (int i = 0; i < 16; ++i)
        if (kpos0 + 16 * (i >> 3) + 8 * hi + (i & 7) > qpos) s[i] = -INFINITY;
    }
    // lazy rescale: raise the running maximum only when a score exceeds it by kDecTau
    float mx = -INFINITY;
#pragma unroll
    for (int i = 0; i < 16; ++i) mx = fmaxf(mx, s[i]);
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
      for (int i = 0; i < 16; ++i) s[i] -= delta;
      m_run = m_new;
      m_eff = m_new_eff;
      thr = (m_new == -INFINITY) ? -INFINITY : kDecTau;
#pragma unroll
      for (int i = 0; i < 16; ++i) minit[i] = -m_eff * isl2;
    }
    // P (bf16) and O^T += V^T P^T, one 16-key group at a time
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      u32x4 w;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        w[j] = pack_bf16x2(fast_exp2(s[8 * kb + 2 * j]), fast_exp2(s[8 * kb + 2 * j + 1]));
        l_run = dot2_bf16_ones(w[j], l_run);
      }
      const bf16x8 pb = __builtin_bit_cast(bf16x8, w);
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) {
        const bf16x4 lo = lds_read_tr16(vt + 16 * kb * D + voff[0][dt]);
        const bf16x4 up = lds_read_tr16(vt + 16 * kb * D + voff[1][dt]);
        oacc[dt] = mfma32(bf16x8{lo[0], lo[1], lo[2], lo[3], up[0], up[1], up[2], up[3]}, pb, oacc[dt]);
      }
    }
  };

  load_tile(0, std::integral_constant<int, 0>{});
  int it = 0;
  for (; it + 1 < nt; it += 2) {
    tile(std::integral_constant<int, 0>{}, it);
    tile(std::integral_constant<int, 1>{}, it + 1);
  }
  if (it < nt) tile(std::integral_constant<int, 0>{}, it);

  // partial state of the chunk for the valid query slots
  const float l_tot = pair_sum(l_run);
  if (t < a.Tq) {
    const long long row = ((long long)bh * a.nch + ch) * a.Tq + t;
    float* acc = a.part_acc + row * D;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int g = 0; g < 4; ++g)
        *(f32x4*)(acc + 32 * dt + 8 * g + 4 * hi) =
            f32x4{oacc[dt][4 * g], oacc[dt][4 * g + 1], oacc[dt][4 * g + 2], oacc[dt][4 * g + 3]};
    if (!hi) {
      a.part_m[row] = m_run;
      a.part_l[row] = l_tot;
    }
  }
}

struct MergeArgs {
  const float* part_acc;
  const float* part_m;
  const float* part_l;
  bf16* o;      // [B, Tq, H, D]
  float* lse;   // [B, H, Tq]
  int B, H, Tq, nch, n_hosts;
};

// One workgroup of 4 waves per (batch, head, query): combine the chunk partial states in
// ring order -- blocks n_hosts-1, n_hosts-2, ..., 0, chunks of a block in order.  All
// partials are present, so instead of carrying a running maximum the sum is taken relative
// to the overall maximum M (found first, in any order):
//   o = sum_c acc_c 2^(m_c - M) / sum_c l_c 2^(m_c - M),  lse = (M ln 2) + ln(denominator),
// which is the online-softmax fold of the same partials without its sequential
// dependence.  Wave w sums the w-th quarter of the ring-ordered sequence of chunks, in
// order; the four quarter sums are then added in order.  (A single wave walking every
// chunk was bound by the latency of its dependent loads.)
constexpr int kMergeWaves = 4;

template <int D>
__global__ __launch_bounds__(64 * kMergeWaves) void decode_merge_kernel(const MergeArgs a) {
  constexpr int E = D / 64;  // dims per lane
  __shared__ float s_max[kMergeWaves];
  __shared__ float s_part[kMergeWaves][D + 1];
  const int t = blockIdx.x % a.Tq, bh = blockIdx.x / a.Tq;
  const int b = bh / a.H, h = bh % a.H;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int cpb = a.nch / a.n_hosts;  // chunks per block
  const long long base = (long long)bh * a.nch;
  float mx = -INFINITY;
  for (int c = tid; c < a.nch; c += 64 * kMergeWaves) mx = fmaxf(mx, a.part_m[(base + c) * a.Tq + t]);
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
  if (lane == 0) s_max[wave] = mx;
  __syncthreads();
#pragma unroll
  for (int w = 0; w < kMergeWaves; ++w) mx = fmaxf(mx, s_max[w]);
  // sequence position q (0 .. nch-1) of the ring order is chunk (n_hosts-1-q/cpb)*cpb + q%cpb
  const int q0 = (int)((long long)a.nch * wave / kMergeWaves);
  const int q1 = (int)((long long)a.nch * (wave + 1) / kMergeWaves);
  float l = 0.f, acc[E];
#pragma unroll
  for (int e = 0; e < E; ++e) acc[e] = 0.f;
#pragma unroll 4
  for (int q = q0; q < q1; ++q) {
    const int chunk = (a.n_hosts - 1 - q / cpb) * cpb + q % cpb;
    const long long row = (base + chunk) * a.Tq + t;
    const float mc = a.part_m[row];
    const float w = (mc == -INFINITY) ? 0.f : exp2f(mc - mx);
    l = fmaf(a.part_l[row], w, l);
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] = fmaf(a.part_acc[row * D + lane + 64 * e], w, acc[e]);
  }
#pragma unroll
  for (int e = 0; e < E; ++e) s_part[wave][lane + 64 * e] = acc[e];
  if (lane == 0) s_part[wave][D] = l;
  __syncthreads();
  if (wave != 0) return;
  float lt = 0.f, at[E];
#pragma unroll
  for (int e = 0; e < E; ++e) at[e] = 0.f;
#pragma unroll
  for (int w = 0; w < kMergeWaves; ++w) {
    lt += s_part[w][D];
#pragma unroll
    for (int e = 0; e < E; ++e) at[e] += s_part[w][lane + 64 * e];
  }
  const float inv = 1.f / lt;
  bf16* orow = a.o + ((long long)b * a.Tq + t) * a.H * D + h * D;
#pragma unroll
  for (int e = 0; e < E; ++e) orow[lane + 64 * e] = (bf16)(at[e] * inv);
  if (lane == 0) a.lse[(long long)bh * a.Tq + t] = mx * kLn2 + logf(lt);
}

// Keys per chunk: the whole block, halved while the launch has fewer than 4096
// workgroups (16 per compute unit) and the half stays a multiple of 32.
int pick_chunk(int B, int H, int S, int c) {
  int kch = c;
  while (kch % 64 == 0 && (long long)B * H * (S / kch) < 4096) kch /= 2;
  return kch;
}

}  // namespace
}  // namespace ra

using namespace ra;

// Argument checks shared by both decode entry points.
static int decode_validate(const void* q, const void* k_cache, const void* v_cache, const void* o, const float* lse,
                           int B, int H, int S, int D, int Tq, int n_hosts, int causal) {
  if (!q || !k_cache || !v_cache || !o || !lse) return set_err(RA_EINVAL, "null pointer argument");
  if (int e = check_aligned({q, k_cache, v_cache, o}, {lse})) return e;
  if (B <= 0 || H <= 0 || S <= 0 || D <= 0 || Tq <= 0 || n_hosts <= 0)
    return set_err(RA_EINVAL, "sizes must be positive (B=%d H=%d S=%d D=%d Tq=%d n_hosts=%d)", B, H, S, D, Tq,
                   n_hosts);
  if (causal != 0 && causal != 1) return set_err(RA_EINVAL, "causal must be 0 or 1 (got %d)", causal);
  if (Tq > S) return set_err(RA_EINVAL, "Tq=%d exceeds the cache length S=%d", Tq, S);
  if (Tq > kDecMaxQ) return set_err(RA_EUNSUPPORTED, "Tq=%d exceeds %d query tokens", Tq, kDecMaxQ);
  if (D != 64 && D != 128) return set_err(RA_EUNSUPPORTED, "head dim D=%d not supported (64 or 128)", D);
  if (n_hosts > 64) return set_err(RA_EUNSUPPORTED, "n_hosts=%d exceeds 64", n_hosts);
  if (S % n_hosts) return set_err(RA_EUNSUPPORTED, "S=%d is not a multiple of n_hosts=%d", S, n_hosts);
  if ((S / n_hosts) % kDecKT)
    return set_err(RA_EUNSUPPORTED, "block S/n_hosts=%d is not a multiple of %d", S / n_hosts, kDecKT);
  if ((long long)B * S * H * D >= (1ll << 31))
    return set_err(RA_EUNSUPPORTED, "B*S*H*D = %lld elements exceeds 2^31-1", (long long)B * S * H * D);
  return RA_OK;
}

// Both launches of a decode call, the chunk partial states in `part` (rows * (D + 2) floats
// for rows = B * H * nch * Tq, every entry written by the first launch before the second
// reads it).
static int decode_launch(const void* q, const void* k_cache, const void* v_cache, void* o, float* lse, int B, int H,
                         int S, int D, int Tq, int n_hosts, int causal, int kch, float* part, hipStream_t stream) {
  const int nch = S / kch;
  const long long rows = (long long)B * H * nch * Tq;
  DecodeArgs da;
  da.q = (const bf16*)q;
  da.k = (const bf16*)k_cache;
  da.v = (const bf16*)v_cache;
  da.part_acc = part;
  da.part_m = da.part_acc + rows * D;
  da.part_l = da.part_m + rows;
  da.B = B;
  da.H = H;
  da.S = S;
  da.Tq = Tq;
  da.kch = kch;
  da.nch = nch;
  da.causal = causal;
  da.scale = 1.f / sqrtf((float)D);
  const int grid = B * H * nch;
  RA_HIP(timed_launch(RA_KERNEL_DECODE, stream, [&] {
    if (D == 128)
      hipLaunchKernelGGL(decode_partial_kernel<128>, dim3(grid), dim3(64), 0, stream, da);
    else
      hipLaunchKernelGGL(decode_partial_kernel<64>, dim3(grid), dim3(64), 0, stream, da);
    return hipGetLastError();
  }));
  MergeArgs ma{da.part_acc, da.part_m, da.part_l, (bf16*)o, lse, B, H, Tq, nch, n_hosts};
  if (D == 128)
    hipLaunchKernelGGL(decode_merge_kernel<128>, dim3(B * H * Tq), dim3(64 * kMergeWaves), 0, stream, ma);
  else
    hipLaunchKernelGGL(decode_merge_kernel<64>, dim3(B * H * Tq), dim3(64 * kMergeWaves), 0, stream, ma);
  RA_HIP(hipGetLastError());
  return RA_OK;
}

extern "C" int ring_attn_decode(const void* q, const void* k_cache, const void* v_cache, void* o, float* lse, int B,
                                int H, int S, int D, int Tq, int n_hosts, int causal, hipStream_t stream) {
  g_err.clear();
  int rc = decode_validate(q, k_cache, v_cache, o, lse, B, H, S, D, Tq, n_hosts, causal);
  if (rc) return rc;
  const int kch = pick_chunk(B, H, S, S / n_hosts);
  const long long rows = (long long)B * H * (S / kch) * Tq;
  CallResources R(stream);
  if ((rc = R.alloc((size_t)rows * (D + 2) * sizeof(float)))) return rc;
  return decode_launch(q, k_cache, v_cache, o, lse, B, H, S, D, Tq, n_hosts, causal, kch, (float*)R.ws, stream);
}

// ---------------------------------------------------------------------------------
// Decode without allocation.  The chunk partial states live in a fixed device array of
// kScratchFloats floats that every device the library runs on holds until the process
// ends.  In host code `scratch` names a host-side stand-in, not device memory: the device
// address of each device's copy is looked up once per device, with that device current,
// and only that address is handed to the kernels.
// ---------------------------------------------------------------------------------
constexpr long long kScratchFloats = 8ll << 20;  // 32 MiB
static __device__ __align__(256) float scratch[kScratchFloats];

namespace {
std::mutex g_scratch_mu;
float* g_scratch_ptr[64];

int scratch_ptr(float** out) {
  int dev = 0;
  RA_HIP(hipGetDevice(&dev));
  if (dev < 0 || dev >= 64) return set_err(RA_EHIP, "device index %d out of range", dev);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    RA_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (!p) return set_err(RA_EHIP, "hipGetSymbolAddress returned a null address for the decode scratch");
    g_scratch_ptr[dev] = (float*)p;
  }
  *out = g_scratch_ptr[dev];
  return RA_OK;
}
}  // namespace

extern "C" int ring_attn_decode_noalloc(const void* q, const void* k_cache, const void* v_cache, void* o, float* lse,
                                        int B, int H, int S, int D, int Tq, int n_hosts, int causal,
                                        hipStream_t stream) {
  g_err.clear();
  int rc = decode_validate(q, k_cache, v_cache, o, lse, B, H, S, D, Tq, n_hosts, causal);
  if (rc) return rc;
  const int kch = pick_chunk(B, H, S, S / n_hosts);
  const long long need = (long long)B * H * (S / kch) * Tq * (D + 2);
  if (need > kScratchFloats)
    return set_err(RA_EUNSUPPORTED,
                   "partial state of %lld floats (B*H*(S/%d)*Tq*(D+2)) exceeds the %lld-float scratch of "
                   "ring_attn_decode_noalloc",
                   need, kch, kScratchFloats);
  float* part = nullptr;
  if ((rc = scratch_ptr(&part))) return rc;
  return decode_launch(q, k_cache, v_cache, o, lse, B, H, S, D, Tq, n_hosts, causal, kch, part, stream);
}
