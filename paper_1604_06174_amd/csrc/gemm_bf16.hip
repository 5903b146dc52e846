// Dense bf16 GEMM entry points (kernel and conventions in gemm_bf16_kernel.h).
#include "gemm_bf16_kernel.h"

namespace ckpt {

using namespace gb;

namespace {

Args make_args(int M, int N, int K, const void *A, int lda, const void *B, int ldb, float *C, int ldc,
               const float *D, int ldd, const float *bias, const GemmX &x) {
  const int splits = x.splits < 1 ? 1 : x.splits;
  int kper = ((K + splits - 1) / splits + KS - 1) / KS * KS;
  if (kper < KS) kper = KS;
  Args a{};
  a.M = M; a.N = N; a.K = K;
  a.A = A; a.lda = lda;
  a.B = static_cast<const __bf16 *>(B); a.ldb = ldb;
  a.C = C; a.ldc = ldc; a.D = D; a.ldd = ldd; a.bias = bias;
  a.Ym = static_cast<const __bf16 *>(x.mask);
  a.Cb = static_cast<__bf16 *>(x.Cb);
  a.stats = x.stats;
  a.kper = kper;
  return a;
}

}  // namespace

void gemm_bf16x(hipStream_t s, int M, int N, int K, const void *A, bool a_fp32, int lda, bool ak,
                const void *B, int ldb, bool bk, float *C, int ldc, int epi, const float *D, int ldd,
                const float *bias, const GemmX &x) {
  if (M <= 0 || N <= 0) return;
  const int splits = x.splits < 1 ? 1 : x.splits;
  const Args a = make_args(M, N, K, A, lda, B, ldb, C, ldc, D, ldd, bias, x);
#define CKPT_GB(AK_, BK_)                                                            \
  if (ak == AK_ && bk == BK_) {                                                      \
    if (a_fp32) pick_tile<AK_, BK_, float, G_DENSE, G_DENSE>(a, epi, splits, s);     \
    else pick_tile<AK_, BK_, __bf16, G_DENSE, G_DENSE>(a, epi, splits, s);           \
    return;                                                                          \
  }
  CKPT_GB(true, true)
  CKPT_GB(true, false)
  CKPT_GB(false, true)
  CKPT_GB(false, false)
#undef CKPT_GB
}

void gemm_bf16(hipStream_t s, int M, int N, int K, const void *A, bool a_fp32, int lda, bool ak,
               const void *B, int ldb, bool bk, float *C, int ldc, int epi, const float *D, int ldd,
               const float *bias) {
  gemm_bf16x(s, M, N, K, A, a_fp32, lda, ak, B, ldb, bk, C, ldc, epi, D, ldd, bias, GemmX{});
}

int gemm_bf16_row_blocks(int M, int N) {
  const Tile t = tile_of(M, N);
  return (M + t.BM - 1) / t.BM;
}

int gemm_bf16_tiles(int M, int N) {
  const Tile t = tile_of(M, N);
  return ((M + t.BM - 1) / t.BM) * ((N + t.BN - 1) / t.BN);
}

}  // namespace ckpt
