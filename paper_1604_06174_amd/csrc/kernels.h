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

// ---- 3x3 convolutions (conv.hip) ----
enum { CONV_FWD = 0, CONV_DGRAD = 1 };
enum { CONV_EPI_STORE = 0, CONV_EPI_STATS = 1, CONV_EPI_MASK = 2, CONV_EPI_SC1 = 3, CONV_EPI_SC2 = 4 };

// Y[N,H,W,J] = conv of X[N,Hx,Wx,C] (FWD: stride S; DGRAD: gradient of a
// stride-S forward conv, X = dy).  Epilogue operands: MASK E0 = mask tensor
// shaped like Y; SC1 E0 = g, E1 = y shaped like Y; SC2 E0 = g, E1 = y of dims
// [N, Eh, Ew, Ec].  STATS writes [blocks][2][J] float64 channel sums.
void conv3x3(hipStream_t s, int mode, int S, int epi, const float *X, const float *Wt, float *Y,
             int N, int H, int W, int Hx, int Wx, int C, int J, const float *E0 = nullptr,
             const float *E1 = nullptr, int Eh = 0, int Ew = 0, int Ec = 0,
             double *stats = nullptr);
int conv3x3_blocks(int mode, int S, int N, int H, int W, int C, int J);
int conv3x3_wgrad_blocks(int S, int N, int H, int W, int C, int J);
bool conv3x3_supported(int mode, int S, int H, int W, int C, int J);
// dW[J,3,3,C] of a stride-S forward conv with input X[N,Hx,Wx,C] and output
// gradient DY[N,H,W,J]; part holds conv3x3_wgrad_blocks * J*9*C floats.
void conv3x3_wgrad(hipStream_t s, int S, const float *X, const float *DY, float *part, float *dW,
                   int N, int H, int W, int Hx, int Wx, int C, int J);

// ---- batch norm and the classifier head (bn.hip) ----
enum { BN_RES_NONE = 0, BN_RES_ID = 1, BN_RES_A = 2 };
int bn_partial_blocks(int64_t P, int J);
// st[0..J) = mean, st[J..2J) = rstd from conv STATS partials over m values.
void bn_finalize_fwd(hipStream_t s, const double *part, int nb, int J, int64_t m, float *st);
// Y = relu(gamma (C - mean) rstd + beta [+ shortcut(X)]) over P pixels x J.
void bn_apply(hipStream_t s, int res, int64_t P, int J, const float *Cv, const float *st,
              const float *gamma, const float *beta, const float *X, int H, int W, int Cx, float *Y);
// ds = Ym ? g [Ym > 0] : g; writes dgamma, dbeta and D = dL/dC.
void bn_backward(hipStream_t s, int64_t P, int J, const float *G, const float *Ym, const float *Cv,
                 const float *st, const float *gamma, double *part, float *sums, float *dgamma,
                 float *dbeta, float *D);
void pool_fc_ce_head(hipStream_t s, int N, int HW, int C, int K, const float *X, const float *Wf,
                     const float *bf, const int *labels, float *pooled, float *dlog, float *lossn,
                     float *G, float *dW, float *db, float *loss);

// ---- bf16 GEMM (gemm_bf16.hip) ----
// C[M,N] fp32 = op(A) op(B) (+ bias | + D).  A is bf16, or fp32 rounded to
// bf16 on load (a_fp32); B is bf16.  ak / bk: the operand is stored with k
// contiguous (A[m*lda + k], B[n*ldb + k]); otherwise A[k*lda + m], B[k*ldb + n].
void gemm_bf16(hipStream_t s, int M, int N, int K, const void *A, bool a_fp32, int lda, bool ak,
               const void *B, int ldb, bool bk, float *C, int ldc, int epi, const float *D = nullptr,
               int ldd = 0, const float *bias = nullptr);

// ---- LSTM step kernels (lstm.hip) ----
void transpose_bf16(hipStream_t s, int R, int C, const float *src, void *dst);  // dst[c][r]
void cvt_bf16(hipStream_t s, int64_t n, const float *src, void *dst);
void lstm_fwd_point(hipStream_t s, int B, int H, const float *z, const float *c_prev, float *gates,
                    void *h_out, float *c_out);
void softmax_ce_rows(hipStream_t s, int rows, int V, const float *logits, const int *labels,
                     float scale, float *dlog, float *loss_rows);
void head_bwd_prep(hipStream_t s, int B, int V, const float *dlog, void *dl_bf, float *db_o, bool first);
void lstm_bwd_point(hipStream_t s, int B, int H, const float *dh, const float *dc_in, const float *gates,
                    const float *c_t, const float *c_prev, const void *h_prev, const void *h_t, void *dz,
                    float *dc_prev, void *hp_copy, void *hc_copy, float *db, bool first);
void loss_reduce(hipStream_t s, int64_t rows, const float *v, float scale, float *loss);
void fill_f32(hipStream_t s, int64_t n, float *p, float v);

}  // namespace ckpt
