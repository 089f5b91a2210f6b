// Calibration kernel (not part of the method): the rate at which the chip sustains bf16
// 32x32x16 matrix-core products when nothing else competes, as the measured reference
// beside the published peak in the benchmark's roofline.
#include "ra_common.h"
#include "ra_runtime.h"
#include "ringattn.h"

namespace ra {
namespace {

constexpr int kProbeBlocks = 512, kProbeThreads = 256;  // 2 waves per SIMD on 256 CUs

// Each wave runs `iters` rounds of 8 products on each of 4 independent accumulator chains
// (the chains keep the matrix pipeline full), then writes one value derived from the
// accumulators so that the products are not optimised away.
__global__ __launch_bounds__(kProbeThreads) void mfma_probe_kernel(float* sink, int iters) {
  bf16x8 a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = (bf16)(1e-3f * (float)(threadIdx.x + i));
    b[i] = (bf16)(1e-3f * (float)i);
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
      for (int j = 0; j < 4; ++j) c[j] = mfma32(a, b, c[j]);
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

extern "C" int ring_attn_mfma_probe(int iters, float* sink, hipStream_t stream) {
  g_err.clear();
  if (!sink) return set_err(RA_EINVAL, "null pointer argument");
  if (iters < 1 || iters > (1 << 20)) return set_err(RA_EINVAL, "iters=%d outside [1, 2^20]", iters);
  hipLaunchKernelGGL(mfma_probe_kernel, dim3(kProbeBlocks), dim3(kProbeThreads), 0, stream, sink, iters);
  RA_HIP(hipGetLastError());
  return RA_OK;
}
