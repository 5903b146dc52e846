// bf16 GEMM with fp32 accumulation on CDNA4 matrix cores (v_mfma_f32_16x16x32_bf16).
//
//   C[M,N] (fp32) = epilogue( sum_k A(m,k) B(k,n) )
//   A(m,k) = AK ? A[m*lda + k] : A[k*lda + m]     (AK: k contiguous)
//   B(k,n) = BK ? B[n*ldb + k] : B[k*ldb + n]     (BK: k contiguous)
// A is bf16, or fp32 rounded to bf16 (nearest even) as it is loaded; B is bf16.
//
// Block = 256 threads = 4 wavefronts in a WM x WN grid; each wavefront owns a
// (BM/WM) x (BN/WN) tile of 16x16 accumulators.  K advances in slices of 32
// through double-buffered LDS stored k-contiguous ([m][k] and [n][k]), so
// every lane reads its MFMA operand (8 consecutive k of one row) as one
// 16-byte LDS load.  Operands stored the other way round are transposed while
// they are written to LDS.  Every output element is reduced over K in one
// fixed order (bit-reproducible).
//
// Epilogues: STORE C = acc (+ bias[n]); ADD C = acc + D (D may alias C).
#include <hip/hip_runtime.h>

#include <type_traits>

#include "kernels.h"

namespace ckpt {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

namespace {

constexpr int KS = 32;      // k per LDS slice
constexpr int KP = KS + 8;  // padded row (bf16 elements): 80-byte rows

struct GbArgs {
  int M, N, K;
  const void *A;
  int lda;
  const __bf16 *B;
  int ldb;
  float *C;
  int ldc;
  const float *D;
  int ldd;
  const float *bias;
};

__device__ __forceinline__ __bf16 to_bf16(float x) { return (__bf16)x; }

// 8 consecutive elements of row `row` starting at column `col` of a
// row-major [rows, cols] matrix of T, zero outside, as bf16.
template <typename T>
__device__ __forceinline__ void ld8(__bf16 r[8], const T *base, int row, int col, int rows, int cols,
                                    int ld) {
  const bool inrow = row < rows;
  const T *p = base + size_t(row) * ld + col;
  if (inrow && col + 7 < cols && (ld % 8 == 0)) {
    if constexpr (std::is_same<T, float>::value) {
      const float4 a = *reinterpret_cast<const float4 *>(p);
      const float4 b = *reinterpret_cast<const float4 *>(p + 4);
      r[0] = to_bf16(a.x); r[1] = to_bf16(a.y); r[2] = to_bf16(a.z); r[3] = to_bf16(a.w);
      r[4] = to_bf16(b.x); r[5] = to_bf16(b.y); r[6] = to_bf16(b.z); r[7] = to_bf16(b.w);
    } else {
      const bf16x8 v = *reinterpret_cast<const bf16x8 *>(p);
#pragma unroll
      for (int u = 0; u < 8; ++u) r[u] = v[u];
    }
  } else {
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      if (inrow && col + u < cols) {
        if constexpr (std::is_same<T, float>::value) r[u] = to_bf16(p[u]);
        else r[u] = p[u];
      } else {
        r[u] = (__bf16)0.f;
      }
    }
  }
}

template <int BM, int BN, int WM, int WN, bool AK, bool BK, typename TA, int EPI>
__global__ __launch_bounds__(256) void k_gemm_bf16(GbArgs p) {
  constexpr int TM = BM / WM / 16, TN = BN / WN / 16;  // 16x16 tiles per wavefront
  static_assert(WM * WN == 4 && TM >= 1 && TN >= 1, "wave grid");
  constexpr int CHA = BM * KS / 8, CHB = BN * KS / 8;  // 8-element chunks per slice
  constexpr int PA = (CHA + 255) / 256, PB = (CHB + 255) / 256;
  __shared__ __align__(16) __bf16 As[2][BM][KP];
  __shared__ __align__(16) __bf16 Bs[2][BN][KP];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int i16 = lane & 15, q = lane >> 4;
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
  const int wm = (wave / WN) * (BM / WM), wn = (wave % WN) * (BN / WN);
  const TA *A = static_cast<const TA *>(p.A);

  __bf16 ra[PA][8], rb[PB][8];
  auto gload = [&](int k0) {
#pragma unroll
    for (int c = 0; c < PA; ++c) {
      const int e = tid + c * 256;
      if (e < CHA) {
        if (AK) {  // chunk = 8 k of one m
          const int mr = e / (KS / 8), kc = (e % (KS / 8)) * 8;
          ld8<TA>(ra[c], A, m0 + mr, k0 + kc, p.M, p.K, p.lda);
        } else {   // chunk = 8 m of one k
          const int kr = e / (BM / 8), mc = (e % (BM / 8)) * 8;
          ld8<TA>(ra[c], A, k0 + kr, m0 + mc, p.K, p.M, p.lda);
        }
      }
    }
#pragma unroll
    for (int c = 0; c < PB; ++c) {
      const int e = tid + c * 256;
      if (e < CHB) {
        if (BK) {
          const int nr = e / (KS / 8), kc = (e % (KS / 8)) * 8;
          ld8<__bf16>(rb[c], p.B, n0 + nr, k0 + kc, p.N, p.K, p.ldb);
        } else {
          const int kr = e / (BN / 8), nc = (e % (BN / 8)) * 8;
          ld8<__bf16>(rb[c], p.B, k0 + kr, n0 + nc, p.K, p.N, p.ldb);
        }
      }
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int c = 0; c < PA; ++c) {
      const int e = tid + c * 256;
      if (e < CHA) {
        if (AK) {
          const int mr = e / (KS / 8), kc = (e % (KS / 8)) * 8;
          bf16x8 v;
#pragma unroll
          for (int u = 0; u < 8; ++u) v[u] = ra[c][u];
          *reinterpret_cast<bf16x8 *>(&As[buf][mr][kc]) = v;
        } else {
          const int kr = e / (BM / 8), mc = (e % (BM / 8)) * 8;
#pragma unroll
          for (int u = 0; u < 8; ++u) As[buf][mc + u][kr] = ra[c][u];
        }
      }
    }
#pragma unroll
    for (int c = 0; c < PB; ++c) {
      const int e = tid + c * 256;
      if (e < CHB) {
        if (BK) {
          const int nr = e / (KS / 8), kc = (e % (KS / 8)) * 8;
          bf16x8 v;
#pragma unroll
          for (int u = 0; u < 8; ++u) v[u] = rb[c][u];
          *reinterpret_cast<bf16x8 *>(&Bs[buf][nr][kc]) = v;
        } else {
          const int kr = e / (BN / 8), nc = (e % (BN / 8)) * 8;
#pragma unroll
          for (int u = 0; u < 8; ++u) Bs[buf][nc + u][kr] = rb[c][u];
        }
      }
    }
  };

  floatx4 acc[TM][TN];
#pragma unroll
  for (int a = 0; a < TM; ++a)
#pragma unroll
    for (int b = 0; b < TN; ++b) acc[a][b] = floatx4{0.f, 0.f, 0.f, 0.f};

  const int nk = (p.K + KS - 1) / KS;
  gload(0);
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    sstore(buf);
    __syncthreads();
    if (kt + 1 < nk) gload((kt + 1) * KS);
    bf16x8 av[TM], bv[TN];
#pragma unroll
    for (int a = 0; a < TM; ++a) av[a] = *reinterpret_cast<const bf16x8 *>(&As[buf][wm + a * 16 + i16][8 * q]);
#pragma unroll
    for (int b = 0; b < TN; ++b) bv[b] = *reinterpret_cast<const bf16x8 *>(&Bs[buf][wn + b * 16 + i16][8 * q]);
#pragma unroll
    for (int a = 0; a < TM; ++a)
#pragma unroll
      for (int b = 0; b < TN; ++b)
        acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[a], bv[b], acc[a][b], 0, 0, 0);
  }

#pragma unroll
  for (int a = 0; a < TM; ++a)
#pragma unroll
    for (int b = 0; b < TN; ++b)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = m0 + wm + a * 16 + 4 * q + r, n = n0 + wn + b * 16 + i16;
        if (m < p.M && n < p.N) {
          float v = acc[a][b][r];
          if (EPI == GEMM_EPI_ADD) v += p.D[size_t(m) * p.ldd + n];
          else if (p.bias) v += p.bias[n];
          p.C[size_t(m) * p.ldc + n] = v;
        }
      }
}

template <int BM, int BN, int WM, int WN, bool AK, bool BK, typename TA>
void launch_b(const GbArgs &a, int epi, hipStream_t s) {
  dim3 grid((a.N + BN - 1) / BN, (a.M + BM - 1) / BM);
  if (epi == GEMM_EPI_ADD)
    hipLaunchKernelGGL((k_gemm_bf16<BM, BN, WM, WN, AK, BK, TA, GEMM_EPI_ADD>), grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL((k_gemm_bf16<BM, BN, WM, WN, AK, BK, TA, GEMM_EPI_STORE>), grid, dim3(256), 0, s, a);
}

template <bool AK, bool BK, typename TA>
void pick_tile(const GbArgs &a, int epi, hipStream_t s) {
  const long big = long((a.M + 127) / 128) * ((a.N + 127) / 128);
  if (a.M >= 256 && big >= 128) {
    launch_b<128, 128, 2, 2, AK, BK, TA>(a, epi, s);
  } else if (long((a.M + 63) / 64) * ((a.N + 63) / 64) >= 64) {
    launch_b<64, 64, 2, 2, AK, BK, TA>(a, epi, s);
  } else {
    launch_b<64, 32, 4, 1, AK, BK, TA>(a, epi, s);
  }
}

}  // namespace

void gemm_bf16(hipStream_t s, int M, int N, int K, const void *A, bool a_fp32, int lda, bool ak,
               const void *B, int ldb, bool bk, float *C, int ldc, int epi, const float *D, int ldd,
               const float *bias) {
  if (M <= 0 || N <= 0) return;
  GbArgs a{M, N, K, A, lda, static_cast<const __bf16 *>(B), ldb, C, ldc, D, ldd, bias};
#define CKPT_GB(AK_, BK_)                                                 \
  if (ak == AK_ && bk == BK_) {                                           \
    if (a_fp32) pick_tile<AK_, BK_, float>(a, epi, s);                    \
    else pick_tile<AK_, BK_, __bf16>(a, epi, s);                          \
    return;                                                               \
  }
  CKPT_GB(true, true)
  CKPT_GB(true, false)
  CKPT_GB(false, true)
  CKPT_GB(false, false)
#undef CKPT_GB
}

}  // namespace ckpt
