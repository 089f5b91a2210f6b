// Interface of the bf16 GEMM kernel family and the column-sum reduction.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>

namespace ra {

enum GemmEpilogue {
  EPI_BF16 = 0,           // C = acc (+ bias[n]) (+ residual[m][n]), stored bf16
  EPI_ACT_BF16 = 1,       // C = act(acc + bias[n]) (+ residual), stored bf16
  EPI_ACT_STORE_H = 2,    // aux_f32 = acc + bias (pre-activation, float32); C = act(aux_f32), bf16
  EPI_ACT_GRAD_BF16 = 3,  // C = acc * act'(aux_f32[m][n]), stored bf16
  EPI_F32 = 4,            // C = acc (or C += acc if accumulate), float32
  EPI_GLU_BF16 = 5,       // C = silu(aux_f32[m][n]) * acc, bf16; aux2_f32 = acc if aux2_f32 != null
  EPI_GLU_GRAD = 6        // with u = aux_f32, w = aux2_f32: C = acc * w * silu'(u), C2 = acc * silu(u) (bf16)
};

struct GemmArgs {
  const void* A;          // bf16, [M][lda] (or [K][lda] when transposed)
  const void* B;          // bf16, [K][ldb] (or [N][ldb] when transposed)
  void* C;                // bf16 or float32 [M][ldc]
  const void* bias;       // bf16 [N] or null
  const void* residual;   // bf16 [M][ldc] or null
  float* aux_f32;         // float32 [M][ldc]: pre-activation (written or read)
  float* aux2_f32;        // float32 [M][ldc]: second gate input of the GLU epilogues
  void* C2;               // bf16 [M][ldc]: second output of EPI_GLU_GRAD
  long long lda, ldb, ldc;
  int M, N, K, act, accumulate;
};

// ta: A stored as [K][M]; tb: B stored as [N][K].  M % 256, N % 256, K % 64 must be 0.
hipError_t launch_gemm(const GemmArgs& g, bool ta, bool tb, int epi, hipStream_t st);
int gemm_tile_m();
int gemm_tile_n();
int gemm_tile_k();

// out[n] (+)= sum_m x[m][n] for bf16 x [M][N]; part: colsum_workspace_floats(N) floats.
hipError_t launch_colsum_bf16(const void* x, float* part, float* out, int M, int N, int accumulate,
                              hipStream_t st);
size_t colsum_workspace_floats(int N);

// out = bf16(a + b) elementwise for float32 a and bf16 b (n elements).
hipError_t launch_add_cast_bf16(const float* a, const void* b, void* out, long long n, hipStream_t st);

}  // namespace ra
