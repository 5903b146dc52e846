// Host-side launchers of the HIP kernels (all asynchronous on `s`).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace ckpt {

enum { GEMM_EPI_STORE = 0, GEMM_EPI_ADD = 1, GEMM_EPI_MLPFWD = 2 };

// C = epilogue(op(A) op(B)); see gemm_f32.hip for the operand conventions.
void gemm_f32(hipStream_t s, int M, int N, int K, const float *A, int lda, bool ta, const float *B,
              int ldb, bool tb, float *C, int ldc, int epi, const float *D = nullptr, int ldd = 0,
              const float *bias = nullptr, float *Z = nullptr, int ldz = 0);

// Residual-MLP backward prologue: dr = g * [z > 0]; db[n] = sum_m dr[m, n]
// (fixed summation order).  [rows, cols] row-major.
void mlp_relu_bwd(hipStream_t s, int rows, int cols, const float *g, const float *z, float *dr,
                  float *db);

// Mean-squared-error head: loss_out[0] = sum((y-t)^2)/count, g = 2 (y-t)/count.
void mse_head(hipStream_t s, int64_t count, const float *y, const float *t, float *g,
              float *loss_out);

// Copy one f32 scalar (device to device) -- used to publish the loss.
void copy_scalar(hipStream_t s, const float *src, float *dst);

}  // namespace ckpt
