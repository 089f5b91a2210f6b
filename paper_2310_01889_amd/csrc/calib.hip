// Calibration kernel (not part of the method): the rate at which the chip sustains bf16
// 32x32x16 matrix-core products when nothing else competes, as the measured reference
// beside the published peak in the benchmark's roofline.
#include "ra_common.h"
#include "ra_runtime.h"
#include "ringattn.h"

namespace ra {
namespace {

constexpr int kProbeBlocks = 512, kProbeThreads = 256;  // 2 waves per SIMD on 256 CUs

// Integer mixing function (the "lowbias32" hash of C. Wellons' hash-prospector) for the
// random operand bits.
__device__ __forceinline__ uint32_t mix32(uint32_t x) {
  x ^= x >> 16;
  x *= 0x7feb352dU;
  x ^= x >> 15;
  x *= 0x846ca68bU;
  x ^= x >> 16;
  return x;
}
// Two bf16 values from 32 random bits: random sign and 7-bit mantissa, exponent chosen
// among 2^-1 .. 2^2 (magnitudes in [0.5, 8), the range of unit-variance data).
__device__ __forceinline__ uint32_t random_bf16_pair(uint32_t h) {
  const uint32_t lo = (h & 0x807fu) | ((((h >> 7) & 3u) + 126u) << 7);
  const uint32_t hi = ((h >> 16) & 0x807fu) | ((((h >> 23) & 3u) + 126u) << 7);
  return (lo & 0xffffu) | (hi << 16);
}

// Each wave runs `iters` rounds of 8 products on each of 4 independent accumulator chains
// (the chains keep the matrix pipeline full), then writes one value derived from the
// accumulators so that the products are not optimised away.  RAND = false: the same two
// operands in every product (few bits toggle: the matrix cores' headline rate); RAND =
// true: eight random operand pairs per lane in rotation, so the operands change from one
// product to the next as they do on real data (more switching power: the clock the board
// sustains is lower).
template <bool RAND>
__global__ __launch_bounds__(kProbeThreads) void mfma_probe_kernel(float* sink, int iters) {
  constexpr int NOP = RAND ? 8 : 1;
  bf16x8 a[NOP], b[NOP];
  const uint32_t seed = (blockIdx.x * kProbeThreads + threadIdx.x) * 977u;
#pragma unroll
  for (int j = 0; j < NOP; ++j) {
    if constexpr (RAND) {
      u32x4 ua, ub;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        ua[e] = random_bf16_pair(mix32(seed + 64 * j + e));
        ub[e] = random_bf16_pair(mix32(seed + 64 * j + 32 + e));
      }
      a[j] = __builtin_bit_cast(bf16x8, ua);
      b[j] = __builtin_bit_cast(bf16x8, ub);
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        a[j][i] = (bf16)(1e-3f * (float)(threadIdx.x + i));
        b[j][i] = (bf16)(1e-3f * (float)i);
      }
    }
  }
  f32x16 c[4];
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int i = 0; i < 16; ++i) c[j][i] = 0.f;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int r = 0; r < 8; ++r)
#pragma unroll
      for (int j = 0; j < 4; ++j) c[j] = mfma32(a[(r + j) % NOP], b[(3 * r + j) % NOP], c[j]);
  }
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int i = 0; i < 16; ++i) s += c[j][i];
  const int wave = (blockIdx.x * kProbeThreads + threadIdx.x) >> 6;
  if ((threadIdx.x & 63) == 0) sink[wave] = s;
}

}  // namespace
}  // namespace ra

using namespace ra;

extern "C" int ring_attn_mfma_probe(int iters, int random_operands, float* sink, hipStream_t stream) {
  g_err.clear();
  if (!sink) return set_err(RA_EINVAL, "null pointer argument");
  if (iters < 1 || iters > (1 << 20)) return set_err(RA_EINVAL, "iters=%d outside [1, 2^20]", iters);
  if (random_operands != 0 && random_operands != 1) return set_err(RA_EINVAL, "random_operands=%d not 0 or 1", random_operands);
  if (random_operands)
    hipLaunchKernelGGL(mfma_probe_kernel<true>, dim3(kProbeBlocks), dim3(kProbeThreads), 0, stream, sink, iters);
  else
    hipLaunchKernelGGL(mfma_probe_kernel<false>, dim3(kProbeBlocks), dim3(kProbeThreads), 0, stream, sink, iters);
  RA_HIP(hipGetLastError());
  return RA_OK;
}
