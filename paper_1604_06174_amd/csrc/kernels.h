// Host-side launchers of the HIP kernels (all asynchronous on `s`).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace ckpt {

// relu(gamma (x - mean) rstd + beta) with one explicit rounding sequence, so
// that every kernel that forms a batch-norm + ReLU output (the apply kernel,
// and the convolutions that form it on the fly from the convolution output
// and its statistics) produces the same bits.
__device__ __forceinline__ float bn_relu(float x, float mean, float rstd, float g, float b) {
  return fmaxf(__builtin_fmaf(g, (x - mean) * rstd, b), 0.f);
}

// GEMM_EPI_BNBWD (bf16 GEMM, k-contiguous bf16 A, n-contiguous B, one k
// split, ldc == N): the product is the gradient G that reaches a batch norm's
// output through a ReLU; the epilogue stores ds = [Ym > 0] G into C and
// writes, per row tile of the GEMM, the float64 column sums of ds and of
// ds * xhat, xhat = (Cv - mean) * rstd, block-major [row tile][2][N] (the
// batch-norm backward's partial sums, so only its finalize and element pass
// remain).
// GEMM_EPI_ROWSOFTMAX (bf16 GEMM, k-contiguous dense A and B, one k split,
// ldc == N, N % 4 == 0): C = product + bias[n]; per row m and column tile t
// (gemm_bf16_col_blocks(M, N) tiles) rstat[(m * tiles + t) * 2] = the row's
// maximum over the tile's columns and the sum of exp(C - maximum) over them.
enum { GEMM_EPI_STORE = 0, GEMM_EPI_ADD = 1, GEMM_EPI_MLPFWD = 2, GEMM_EPI_BF16STATS = 3, GEMM_EPI_ADDMASK = 4,
       GEMM_EPI_BIAS = 5, GEMM_EPI_BNBWD = 6, GEMM_EPI_ROWSOFTMAX = 7 };

// C = epilogue(op(A) op(B)); see gemm_f32.hip for the operand conventions.
void gemm_f32(hipStream_t s, int M, int N, int K, const float *A, int lda, bool ta, const float *B,
              int ldb, bool tb, float *C, int ldc, int epi, const float *D = nullptr, int ldd = 0,
              const float *bias = nullptr, float *Z = nullptr, int ldz = 0);

// Residual-MLP backward prologue: dr = g * [z > 0]; db[n] = sum_m dr[m, n]
// (fixed summation order).  [rows, cols] row-major.
// dr = g * [z > 0] and db = column sums of dr (rows in a fixed order); pdb is
// workspace of mlp_relu_row_blocks(rows) * cols floats.
int mlp_relu_row_blocks(int rows);
void mlp_relu_bwd(hipStream_t s, int rows, int cols, const float *g, const float *z, float *dr,
                  float *db, float *pdb);

// Mean-squared-error head: loss_out[0] = sum((y-t)^2)/count, g = 2 (y-t)/count.
void mse_head(hipStream_t s, int64_t count, const float *y, const float *t, float *g,
              float *loss_out);

// Copy one f32 scalar (device to device) -- used to publish the loss.
void copy_scalar(hipStream_t s, const float *src, float *dst);
// column sums of g [rows, cols] in the same order as mlp_relu_bwd's
void mlp_colsum(hipStream_t s, int rows, int cols, const float *g, float *db, float *pdb);
// elementwise operators of node-level graphs (outputs may alias inputs)
void ew_relu(hipStream_t s, int64_t n, const float *x, float *y);                  // y = max(x, 0)
void ew_add(hipStream_t s, int64_t n, const float *a, const float *b, float *y);   // y = a + b
void ew_relu_bwd(hipStream_t s, int64_t n, const float *dy, const float *y, float *dx);  // dy [y > 0]
void ew_copy(hipStream_t s, int64_t n, const float *x, float *y);

// ---- 3x3 convolutions (conv.hip) ----
enum { CONV_FWD = 0, CONV_DGRAD = 1 };
enum { CONV_EPI_STORE = 0, CONV_EPI_STATS = 1, CONV_EPI_MASK = 2, CONV_EPI_SC1 = 3, CONV_EPI_SC2 = 4,
       CONV_EPI_MASKSTATS = 5 };

// Y[N,H,W,J] = conv of X[N,Hx,Wx,C] (FWD: stride S; DGRAD: gradient of a
// stride-S forward conv, X = dy).  Epilogue operands: MASK E0 = mask tensor
// shaped like Y; SC1 E0 = g, E1 = y shaped like Y; SC2 E0 = g, E1 = y of dims
// [N, Eh, Ew, Ec].  STATS writes [2][J][blocks] float64 channel sums.
// Optional batch-norm + ReLU transform (tst = mean | rstd, tg = gamma,
// tb = beta): FWD applies bn_relu to every in-image input value (channel c);
// DGRAD with MASK takes the mask as bn_relu(E0) (channel j) instead of E0.
// MASKSTATS (DGRAD, transform required): MASK with the mask bn_relu(E0), and
// per-workgroup float64 sums of ds and ds * xhat per channel, ds = the masked
// output, xhat = (E0 - mean) rstd: the partial sums of the batch-norm backward
// of E0's batch norm, stored like STATS ([2][J][blocks]).
// rout (stride-1 FWD with the transform, C a multiple of 4): the transformed
// input [N,Hx,Wx,C] is also stored, every element once.
void conv3x3(hipStream_t s, int mode, int S, int epi, const float *X, const float *Wt, float *Y,
             int N, int H, int W, int Hx, int Wx, int C, int J, const float *E0 = nullptr,
             const float *E1 = nullptr, int Eh = 0, int Ew = 0, int Ec = 0,
             double *stats = nullptr, const float *tst = nullptr, const float *tg = nullptr,
             const float *tb = nullptr, float *rout = nullptr);
int conv3x3_blocks(int mode, int S, int N, int H, int W, int C, int J);
int conv3x3_wgrad_blocks(int S, int N, int H, int W, int C, int J);
bool conv3x3_supported(int mode, int S, int H, int W, int C, int J);
// dW[J,3,3,C] of a stride-S forward conv with input X[N,Hx,Wx,C] and output
// gradient DY[N,H,W,J]; part holds conv3x3_wgrad_blocks * J*9*C floats.
// Optional input transform bn_relu (tst, tg, tb) as for the forward.
void conv3x3_wgrad(hipStream_t s, int S, const float *X, const float *DY, float *part, float *dW,
                   int N, int H, int W, int Hx, int Wx, int C, int J, const float *tst = nullptr,
                   const float *tg = nullptr, const float *tb = nullptr);

// ---- batch norm and the classifier head (bn.hip) ----
enum { BN_RES_NONE = 0, BN_RES_ID = 1, BN_RES_A = 2 };
int bn_partial_blocks(int64_t P, int J);
// st[0..J) = mean, st[J..2J) = rstd from the partial sums (sum v, sum v^2) of
// nb workgroups over m values, stored channel-major ([2][J][nb]: conv STATS)
// or block-major ([nb][2][J]: bf16 GEMM BF16STATS).
void bn_finalize_fwd(hipStream_t s, const double *part, int nb, int J, int64_t m, float *st,
                     bool channel_major);
// Y = relu(gamma (C - mean) rstd + beta [+ shortcut(X)]) over P pixels x J.
void bn_apply(hipStream_t s, int res, int64_t P, int J, const float *Cv, const float *st,
              const float *gamma, const float *beta, const float *X, int H, int W, int Cx, float *Y);
// ds = Ym ? g [Ym > 0] : g; writes dgamma, dbeta and D = dL/dC.
void bn_backward(hipStream_t s, int64_t P, int J, const float *G, const float *Ym, const float *Cv,
                 const float *st, const float *gamma, double *part, float *sums, float *dgamma,
                 float *dbeta, float *D);
// the element pass alone, D = dL/dC from the finalized sums (bn_finalize_bwd)
void bn_backward_apply(hipStream_t s, int64_t P, int J, const float *G, const float *Ym,
                       const float *Cv, const float *st, const float *gamma, const float *sums,
                       float *D);
void pool_fc_ce_head(hipStream_t s, int N, int HW, int C, int K, const float *X, const float *Wf,
                     const float *bf, const int *labels, float *pooled, float *dlog, float *lossn,
                     float *G, float *dW, float *db, float *loss);
// the same head over a bf16 X, for wide classifiers: the two products on the
// fp32 GEMM; dpool = N x C floats of workspace
void pool_fc_ce_head_bf16(hipStream_t s, int N, int HW, int C, int K, const void *X, const float *Wf,
                          const float *bf, const int *labels, float *pooled, float *dlog,
                          float *lossn, float *dpool, float *G, float *dW, float *db, float *loss);
// Standalone forms for node-level graphs (NHWC fp32, J a multiple of 4):
// st = mean | rstd of X [P, J] (part: bn_partial_blocks(P, J) * 2 * J
// doubles); Y = gamma (X - mean) rstd + beta; the option-A shortcut Y [N, H,
// W, J] of X [N, 2H, 2W, Cx] and its backward DX [N, 2H, 2W, Cx]; global
// average pool Y [N, C] of X [N, HW, C] and its backward; softmax
// cross-entropy rows of logits L [N, K]: G = the mean loss's gradient with
// respect to L, lossn = each row's loss, loss = their mean.
void bn_stats(hipStream_t s, int64_t P, int J, const float *X, double *part, float *st);
void bn_norm(hipStream_t s, int64_t P, int J, const float *X, const float *st, const float *gamma,
             const float *beta, float *Y);
void shortcut_a(hipStream_t s, int N, int H, int W, int J, int Cx, const float *X, float *Y);
void shortcut_a_bwd(hipStream_t s, int N, int H, int W, int J, int Cx, const float *DY, float *DX);
void avgpool(hipStream_t s, int N, int HW, int C, const float *X, float *Y);
void avgpool_bwd(hipStream_t s, int N, int HW, int C, const float *DY, float *DX);
void softmax_ce_rows(hipStream_t s, int N, int K, const float *L, const int *labels, float *G,
                     float *lossn, float *loss);
// sums[0..J) = mean(ds), sums[J..2J) = mean(ds xhat), dgamma, dbeta from the
// backward partials (sum ds, sum ds xhat) of nb workgroups over m values, in
// either layout (fp32 backward partials: channel-major; bf16: block-major)
void bn_finalize_bwd(hipStream_t s, const double *part, int nb, int J, int64_t m, float *sums,
                     float *dgamma, float *dbeta, bool channel_major);

// ---- bf16 batch norm, stem im2col and max pool (bneck.hip) ----
enum { BNB_RES_NONE = 0, BNB_RES_ID = 1, BNB_RES_BN = 2 };
// Y = bf16(relu(gamma (C - mean) rstd + beta [+ X | + gp (X - meanp) rstdp + bp]))
// over P pixels x J channels (bf16 NHWC; st / stp = mean | rstd).
void bnb_apply(hipStream_t s, int res, int64_t P, int J, const void *Cv, const float *st,
               const float *gamma, const float *beta, const void *X, const float *stp,
               const float *gp, const float *bp, void *Y);
int bnb_partial_blocks(int64_t P, int J);
// D (bf16) = dL/dC of the batch norm with ds = [Ym > 0] G (Ym may be null);
// writes dgamma, dbeta.  part: bnb_partial_blocks * 2J doubles; sums: 2J floats.
void bnb_backward(hipStream_t s, int64_t P, int J, const float *G, const void *Ym, const void *Cv,
                  const float *st, const float *gamma, double *part, float *sums, float *dgamma,
                  float *dbeta, void *D);
// The partial sums and finalize of bnb_backward alone (sums, dgamma, dbeta),
// without its element pass.
void bnb_backward_sums(hipStream_t s, int64_t P, int J, const float *G, const void *Ym, const void *Cv,
                       const float *st, double *part, float *sums, float *dgamma, float *dbeta);
// The element pass of bnb_backward alone, given the finalized sums (2J floats:
// mean of ds, mean of ds * xhat); Ym may be null (G already masked).
void bnb_backward_apply(hipStream_t s, int64_t P, int J, const float *G, const void *Ym,
                        const void *Cv, const float *st, const float *gamma, const float *sums,
                        void *D);
// col [N*Ho*Wo, KP] bf16 = 7x7 / stride 2 / pad 3 patches of X [N, H, W, 3]
// in the first 147 columns, zero past them (KP = 147, or a multiple of 8
// above it: 16-byte chunks, and a GEMM row pitch that takes the direct loop)
void im2col7(hipStream_t s, int N, int H, int W, int Ho, int Wo, int KP, const void *X, void *col);
// dst [R, KP] bf16 = src [R, C] fp32 rounded, zero past column C
void cvt_pad_rows(hipStream_t s, int R, int C, int KP, const float *src, void *dst);
// 3x3 / stride 2 / pad 1 max pool of R [N, H, W, C] into Y [N, Ho, Wo, C] (bf16)
void maxpool_fwd(hipStream_t s, int N, int H, int W, int C, int Ho, int Wo, const void *R, void *Y);
// dR (fp32) = gradient of the max pool: each window's G goes to its first
// maximum.  arg (N Ho Wo C bytes) or null: two passes (each window's
// first-maximum tap, then the gather per input pixel) or one (every input
// pixel scans the windows that hold it); the same bits.
void maxpool_bwd(hipStream_t s, int N, int H, int W, int C, int Ho, int Wo, const float *G,
                 const void *R, const void *Y, float *dR, void *arg);

// ---- bf16 GEMM (gemm_bf16.hip, gemm_bf16_conv.hip) ----
// C[M,N] fp32 = op(A) op(B) (+ bias | + D).  A is bf16, or fp32 rounded to
// bf16 on load (a_fp32); B is bf16.  ak / bk: the operand is stored with k
// contiguous (A[m*lda + k], B[n*ldb + k]); otherwise A[k*lda + m], B[k*ldb + n].
void gemm_bf16(hipStream_t s, int M, int N, int K, const void *A, bool a_fp32, int lda, bool ak,
               const void *B, int ldb, bool bk, float *C, int ldc, int epi, const float *D = nullptr,
               int ldd = 0, const float *bias = nullptr);
// Options: splits > 1 = split-K, C receives splits partial [M, ldc] products
// (STORE); ADDMASK: C = acc + (mask > 0 ? D : 0), mask bf16 shaped like D;
// BF16STATS: Cb (bf16, ldc) = round(acc) and stats[row block][2][N] float64
// sums of the rounded values and squares (row blocks: gemm_bf16_row_blocks).
struct GemmX {
  int splits = 1;
  const void *mask = nullptr;  // ADDMASK, BNBWD
  void *Cb = nullptr;          // BF16STATS
  double *stats = nullptr;     // BF16STATS, BNBWD
  const void *cv = nullptr;    // BNBWD: the batch norm's input (bf16, [M, N])
  const float *bst = nullptr;  // BNBWD: its mean [N] and 1/std [N]
  float *rstat = nullptr;      // ROWSOFTMAX: [M][column tiles][2]
  // BF16STATS with Rb set (a bottleneck unit's re-run, its statistics known):
  // also Rb = bf16(relu(bn(bf16 product) [+ Xr])), bn = act_g ((c - mean)
  // rstd) + act_b with act_st = mean [N] | 1/std [N]; Xr a bf16 residual laid
  // out as Cb, or null (the element pass's bits, see bnb_act.h)
  void *Rb = nullptr;
  const void *Xr = nullptr;
  const float *act_st = nullptr, *act_g = nullptr, *act_b = nullptr;
};
void gemm_bf16x(hipStream_t s, int M, int N, int K, const void *A, bool a_fp32, int lda, bool ak,
                const void *B, int ldb, bool bk, float *C, int ldc, int epi, const float *D,
                int ldd, const float *bias, const GemmX &x);
// nb products of the ROWSOFTMAX form at once (k-contiguous bf16 A [M, K] and
// B [N, K], ldc = N): product z reads A + z bstrA and writes C + z bstrC and
// its row statistics at rstat + z bstrR (at least M * gemm_bf16_col_blocks(M,
// N) * 2 floats apart); every product's bits are those of its own launch.
void gemm_bf16_rowsoftmax_batched(hipStream_t s, int nb, int M, int N, int K, const void *A, int lda,
                                  int64_t bstrA, const void *B, int ldb, float *C, int64_t bstrC,
                                  const float *bias, float *rstat, int64_t bstrR);
int gemm_bf16_row_blocks(int M, int N);
int gemm_bf16_col_blocks(int M, int N);
int gemm_bf16_tiles(int M, int N);
// Split-K for short, wide products: gemm_bf16_part writes `splits` partial
// [M, N] products (contiguous slices) of op(A) op(B) over consecutive k
// ranges; sum_slices adds nslices such slices in order, then D and bias:
// C = sum_z part[z] (+ D) (+ bias[n]).  N must be a multiple of 4.
// (splits chosen so that about `target` workgroups run, at least 128 k each)
int gemm_bf16_splits(int M, int N, int K, int target = 512);
void gemm_bf16_part(hipStream_t s, int M, int N, int K, const void *A, bool a_fp32, int lda, bool ak,
                    const void *B, int ldb, bool bk, float *part, int splits);
void sum_slices(hipStream_t s, const float *part, int nslices, int M, int N, float *C, int ldc,
                const float *D = nullptr, int ldd = 0, const float *bias = nullptr);
// k per split of gemm_bf16_part over K with `splits` splits
int gemm_bf16_kper(int K, int splits);
// gemm_bf16_part of [A1 | A2] (bf16, k contiguous, K1 + K2 columns) times B
// ([N, ldb] bf16, k contiguous over K1 + K2): one launch, `splits` partial
// [M, N] products over consecutive k ranges.  K1, K2, lda1, lda2 and ldb
// multiples of 8.
void gemm_bf16_part_cat(hipStream_t s, int M, int N, int K1, const void *A1, int lda1, int K2,
                        const void *A2, int lda2, const void *B, int ldb, float *part, int splits);
// out[e] = sum_b part[b*E + e], b in a fixed order
void sum_partials(hipStream_t s, const float *part, int nb, int E, float *out);

// Convolution of NHWC bf16 tensors as implicit GEMM: input [N, H, W, Ci],
// output [N, Ho, Wo, Co], weights [Co, R, R, Ci] (bf16), stride S in {1, 2},
// padding P; Ci and Co powers of two, at least 8.
struct ConvGeo {
  int N, H, W, Ci, Ho, Wo, Co, R, S, P;
};
bool conv_bf16_supported(const ConvGeo &g);
// Yb = bf16(conv(X, Wt)); stats[row block][2][Co] as for BF16STATS (none when
// stats is null)
// (row blocks: gemm_bf16_row_blocks(N*Ho*Wo, Co)).
// act (optional): the batch-norm apply output of the BF16STATS epilogue
// (GemmX::Rb, act_st, act_g, act_b; no residual)
void conv_bf16_fwd(hipStream_t s, const ConvGeo &g, const void *X, const void *Wt, void *Yb,
                   double *stats, const GemmX *act = nullptr);
// DX [N, H, W, Ci] fp32 = data gradient of DY [N, Ho, Wo, Co] (bf16) through
// Wt; epi STORE, ADD (+ D), ADDMASK (+ D where mask > 0) or BNBWD (mask, Cv,
// bst and stats as for gemm_bf16x; stats gets gemm_bf16_row_blocks(M, Ci)
// row tiles, M = N*H*W), D, mask and Cv shaped like DX.
void conv_bf16_dgrad(hipStream_t s, const ConvGeo &g, const void *DY, const void *Wt, float *DX,
                     int epi, const float *D = nullptr, const void *mask = nullptr,
                     const void *Cv = nullptr, const float *bst = nullptr, double *stats = nullptr);
// dW [Co, R, R, Ci] fp32 = weight gradient from X (bf16 input) and DY (bf16
// output gradient); split-K over the N*Ho*Wo pixels with `splits` partials
// in part (splits * Co*R*R*Ci floats), added in a fixed order.
void conv_bf16_wgrad(hipStream_t s, const ConvGeo &g, const void *X, const void *DY, float *part,
                     int splits, float *dW);

// ---- LSTM step kernels (lstm.hip) ----
// dst[c * ld + r] = bf16(src[r * C + c]) (ld = R when 0)
void transpose_bf16(hipStream_t s, int R, int C, const float *src, void *dst, int ld = 0);
void cvt_bf16(hipStream_t s, int64_t n, const float *src, void *dst);
// dst (bf16, row stride ld) = src [R][C] fp32
void cvt_bf16_rows(hipStream_t s, int R, int C, const float *src, void *dst, int ld);
// Split-K inputs: zpart / lpart / dhpart hold ns partial slices of the
// product, added in slice order before the bias (or the incoming dh), exactly
// as sum_slices would.
void lstm_fwd_point(hipStream_t s, int B, int H, const float *zpart, int ns, const float *bias,
                    const float *c_prev, float *gates, void *h_out, float *c_out);
// Softmax cross-entropy rows: loss_rows[r] = logsumexp(l[r]) - l[r][label],
// dlog = (softmax - onehot) * scale, from the logits [rows, V] (bias
// included) and the per row and column tile (max, sum of exp) pairs that
// GEMM_EPI_ROWSOFTMAX wrote (nt tiles per row); V % 4 == 0.
void softmax_ce_tiles(hipStream_t s, int rows, int V, const float *logits, int nt, const float *rstat,
                      const int *labels, float scale, float *dlog, float *loss_rows);
// the same over nunits units at once, in place (dlog over the logits): unit u's
// logits at logits + u ul, statistics at rstat + u ur, labels and loss rows at
// + u rows
void softmax_ce_tiles_batched(hipStream_t s, int nunits, int rows, int V, float *logits, int64_t ul, int nt,
                              const float *rstat, int64_t ur, const int *labels, float scale,
                              float *loss_rows);
void head_bwd_prep(hipStream_t s, int B, int V, const float *dlog, void *dl_bf, float *db_o, bool first);
// dbp receives ceil(B/4) records [4H] of bias-gradient column sums (one per
// block of 4 batch rows); db_chunk adds a run of such records into db.
// dh = the ns split-K slices [B, H] of the product that forms it, in order.
void lstm_bwd_point(hipStream_t s, int B, int H, const float *dhpart, int ns, const float *dc_in,
                    const float *gates, const float *c_t, const float *c_prev, const void *h_prev,
                    const void *h_t, void *dz, float *dc_prev, void *hp_copy, void *hc_copy,
                    float *dbp);
void db_chunk(hipStream_t s, int N, int nrec, const float *rec, float *db, bool first);
void loss_reduce(hipStream_t s, int64_t rows, const float *v, float scale, float *loss);
void fill_f32(hipStream_t s, int64_t n, float *p, float v);

}  // namespace ckpt
