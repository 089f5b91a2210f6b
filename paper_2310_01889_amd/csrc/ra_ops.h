// Internal host-side building blocks shared by the C-ABI translation units.
#pragma once

#include <hip/hip_runtime.h>

#include "ra_gemm.h"

namespace ra {

// Validation of a row-blocked product [T, d_in] x [d_in, d_out]; sets the error text.
int check_gemm_dims(int T, int d_in, int d_out, int block);
// One GEMM launch (timed when kernel timing is enabled); RA_OK or an ra_status.
int gemm(const GemmArgs& g, bool ta, bool tb, int epi, hipStream_t st);

// Row-blocked products (bf16 operands, blocks of `block` rows):
//   proj:    y (bf16) = x w (+ residual)
//   wgrad:   dw (f32, overwritten) = x^T dy, accumulated over the row blocks
//   dgrad32: dx32 (f32) = dy w^T, or += when accumulate
int proj(const void* x, const void* w, const void* residual, void* y, int T, int din, int dout, int block,
         hipStream_t st);
int wgrad(const void* x, const void* dy, float* dw, int T, int din, int dout, int block, hipStream_t st);
int dgrad32(const void* dy, const void* w, float* dx32, int accumulate, int T, int din, int dout, int block,
            hipStream_t st);

// Blockwise FFN forward: y = act(x W1 + b1) W2 + b2 (+ residual); arguments validated.
int ffn_forward(const void* x, const void* w1, const void* b1, const void* w2, const void* b2, const void* residual,
                void* y, int T, int d_model, int d_ff, int block, int act, hipStream_t stream);
// Blockwise FFN backward; dx = dy_ffn (+ dx_residual).  Weight gradients overwritten.
int ffn_backward(const void* x, const void* w1, const void* b1, const void* w2, const void* dy, const void* dx_residual,
                 void* dx, float* dw1, float* db1, float* dw2, float* db2, int T, int d_model, int d_ff, int block,
                 int act, hipStream_t stream);

}  // namespace ra
