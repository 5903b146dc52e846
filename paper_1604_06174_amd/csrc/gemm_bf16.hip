// Dense bf16 GEMM entry points (kernel and conventions in gemm_bf16_kernel.h).
#include <algorithm>

#include "common.h"
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
  a.Cv = static_cast<const __bf16 *>(x.cv);
  a.bst = x.bst;
  a.rstat = x.rstat;
  a.Rb = static_cast<__bf16 *>(x.Rb);
  a.Xr = static_cast<const __bf16 *>(x.Xr);
  a.ast = x.act_st;
  a.ag = x.act_g;
  a.ab = x.act_b;
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
  const bool safe = !a_fp32 && safe8(a, ak, bk);
  if (epi == GEMM_EPI_BNBWD &&
      (!ak || bk || !safe || splits != 1 || ldc != N || !x.mask || !x.cv || !x.bst || !x.stats))
    fail(CKPT_E_INVALID, "gemm_bf16x: BNBWD takes k-contiguous bf16 A, n-contiguous B, one split, "
                         "ldc == N and the mask, input, statistics and partial buffers");
  if (x.Rb && (epi != GEMM_EPI_BF16STATS || !x.act_st || !x.act_g || !x.act_b))
    fail(CKPT_E_INVALID, "gemm_bf16x: the batch-norm apply output goes with BF16STATS and needs the "
                         "statistics, gamma and beta");
  if (epi == GEMM_EPI_ROWSOFTMAX &&
      (!ak || !bk || !safe || splits != 1 || ldc != N || N % 4 != 0 || !bias || !x.rstat))
    fail(CKPT_E_INVALID, "gemm_bf16x: ROWSOFTMAX takes k-contiguous bf16 A and B, one split, "
                         "ldc == N, N % 4 == 0, a bias and the row-statistics buffer");
#define CKPT_GB(AK_, BK_)                                                                  \
  if (ak == AK_ && bk == BK_) {                                                            \
    if (a_fp32) pick_tile<AK_, BK_, float, G_DENSE, G_DENSE, false>(a, epi, splits, s);    \
    else if (safe) pick_tile<AK_, BK_, __bf16, G_DENSE, G_DENSE, true>(a, epi, splits, s); \
    else pick_tile<AK_, BK_, __bf16, G_DENSE, G_DENSE, false>(a, epi, splits, s);          \
    return;                                                                                \
  }
  CKPT_GB(true, true)
  CKPT_GB(true, false)
  CKPT_GB(false, true)
  CKPT_GB(false, false)
#undef CKPT_GB
}

void gemm_bf16_rowsoftmax_batched(hipStream_t s, int nb, int M, int N, int K, const void *A, int lda,
                                  int64_t bstrA, const void *B, int ldb, float *C, int64_t bstrC,
                                  const float *bias, float *rstat, int64_t bstrR) {
  if (nb <= 0 || M <= 0 || N <= 0) return;
  if (K % 8 || lda % 8 || ldb % 8 || N % 4 || bstrA % 8 || bstrC % 4 || !bias || !rstat ||
      bstrR < int64_t(M) * gemm_bf16_col_blocks(M, N) * 2)
    fail(CKPT_E_INVALID, "gemm_bf16_rowsoftmax_batched: k extents, strides and tile statistics");
  GemmX x;
  x.rstat = rstat;
  Args a = make_args(M, N, K, A, lda, B, ldb, C, N, nullptr, 0, bias, x);
  a.nbatch = nb;
  a.bstrA = bstrA;
  a.bstrC = bstrC;
  a.bstrR = bstrR;
  pick_tile<true, true, __bf16, G_DENSE, G_DENSE, true>(a, GEMM_EPI_ROWSOFTMAX, nb, s);
}

void gemm_bf16(hipStream_t s, int M, int N, int K, const void *A, bool a_fp32, int lda, bool ak,
               const void *B, int ldb, bool bk, float *C, int ldc, int epi, const float *D, int ldd,
               const float *bias) {
  gemm_bf16x(s, M, N, K, A, a_fp32, lda, ak, B, ldb, bk, C, ldc, epi, D, ldd, bias, GemmX{});
}

namespace {

// C[m, n] = sum over z = 0..ns-1 (in order) of part[z][m][n] (+ D[m, n]) (+ bias[n]);
// four consecutive columns per thread (N % 4 == 0).
__global__ __launch_bounds__(256) void k_sum_slices(const float *__restrict__ part, int ns, int M,
                                                    int N, float *__restrict__ C, int ldc,
                                                    const float *__restrict__ D, int ldd,
                                                    const float *__restrict__ bias) {
  const int NQ = N / 4;
  const int64_t e = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (e >= int64_t(M) * NQ) return;
  const int m = int(e / NQ), n = int(e % NQ) * 4;
  const size_t slice = size_t(M) * N, o = size_t(m) * N + n;
  float4 acc = *reinterpret_cast<const float4 *>(part + o);
  for (int z = 1; z < ns; ++z) {
    const float4 v = *reinterpret_cast<const float4 *>(part + z * slice + o);
    acc.x += v.x; acc.y += v.y; acc.z += v.z; acc.w += v.w;
  }
  if (D) {
    const float *d = D + size_t(m) * ldd + n;
    acc.x += d[0]; acc.y += d[1]; acc.z += d[2]; acc.w += d[3];
  }
  if (bias) {
    acc.x += bias[n]; acc.y += bias[n + 1]; acc.z += bias[n + 2]; acc.w += bias[n + 3];
  }
  float *c = C + size_t(m) * ldc + n;
  c[0] = acc.x; c[1] = acc.y; c[2] = acc.z; c[3] = acc.w;
}

}  // namespace

int gemm_bf16_splits(int M, int N, int K, int target) {
  const int tiles = gemm_bf16_tiles(M, N);
  int s = (target + tiles - 1) / tiles;
  s = std::min(s, std::max(1, K / 128));  // at least 128 k per split
  return std::max(s, 1);
}

void gemm_bf16_part(hipStream_t s, int M, int N, int K, const void *A, bool a_fp32, int lda, bool ak,
                    const void *B, int ldb, bool bk, float *part, int splits) {
  GemmX x;
  x.splits = splits;
  gemm_bf16x(s, M, N, K, A, a_fp32, lda, ak, B, ldb, bk, part, N, GEMM_EPI_STORE, nullptr, 0,
             nullptr, x);
}

int gemm_bf16_kper(int K, int splits) {
  if (splits < 1) splits = 1;
  const int kper = ((K + splits - 1) / splits + KS - 1) / KS * KS;
  return kper < KS ? KS : kper;
}

void gemm_bf16_part_cat(hipStream_t s, int M, int N, int K1, const void *A1, int lda1, int K2,
                        const void *A2, int lda2, const void *B, int ldb, float *part, int splits) {
  if (M <= 0 || N <= 0) return;
  if (K1 % 8 || K2 % 8 || lda1 % 8 || lda2 % 8 || ldb % 8)
    fail(CKPT_E_UNSUPPORTED, "gemm_bf16_part_cat: k extents and strides must be multiples of 8");
  GemmX x;
  x.splits = splits;
  Args a = make_args(M, N, K1 + K2, A1, lda1, B, ldb, part, N, nullptr, 0, nullptr, x);
  a.A2 = static_cast<const __bf16 *>(A2);
  a.lda2 = lda2;
  a.K1 = K1;
  pick_tile<true, true, __bf16, GA_CAT, G_DENSE, true>(a, GEMM_EPI_STORE, x.splits, s);
}

void sum_slices(hipStream_t s, const float *part, int nslices, int M, int N, float *C, int ldc,
                const float *D, int ldd, const float *bias) {
  const int64_t e = int64_t(M) * (N / 4);
  hipLaunchKernelGGL(k_sum_slices, dim3(unsigned((e + 255) / 256)), dim3(256), 0, s, part, nslices,
                     M, N, C, ldc, D, ldd, bias);
}

int gemm_bf16_row_blocks(int M, int N) {
  const Tile t = tile_of(M, N);
  return (M + t.BM - 1) / t.BM;
}

int gemm_bf16_col_blocks(int M, int N) {
  const Tile t = tile_of(M, N);
  return (N + t.BN - 1) / t.BN;
}

int gemm_bf16_tiles(int M, int N) {
  const Tile t = tile_of(M, N);
  return ((M + t.BM - 1) / t.BM) * ((N + t.BN - 1) / t.BN);
}

}  // namespace ckpt
