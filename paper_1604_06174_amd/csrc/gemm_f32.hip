// fp32 GEMM on CDNA4 matrix cores (v_mfma_f32_32x32x2f32 / 16x16x4f32).
//
//   C[M,N] = epilogue( op(A)[M,K] * op(B)[K,N] )
//   op(A)(m,k) = TA ? A[k*lda + m] : A[m*lda + k]
//   op(B)(k,n) = TB ? B[n*ldb + k] : B[k*ldb + n]
//
// Block = 256 threads = 4 wavefronts in a 2x2 grid; each wavefront owns a
// WT x WT output tile (WT = 32 -> one 32x32x2 MFMA accumulator, WT = 16 -> one
// 16x16x4 accumulator); block tile (2 WT) x (2 WT), K staged through LDS in
// slices of 16 with double buffering (global loads of slice k+1 are in flight
// while slice k is multiplied).  Every output element is reduced over K in one
// fixed order, so results do not depend on the launch or on buffer addresses.
//
// Epilogues:
//   STORE    C = acc
//   ADD      C = acc + D                      (backward: dx = dy + dr W^T)
//   MLPFWD   Z = acc + bias;  C = A + relu(Z) (residual block y = x + relu(xW+b);
//                                               requires !TA and K == N)
#include <hip/hip_runtime.h>

#include <type_traits>

#include "kernels.h"

namespace ckpt {

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

namespace {

constexpr int BK = 16;
constexpr int PAD = 4;

struct GemmArgs {
  int M, N, K;
  const float *A;
  int lda;
  const float *B;
  int ldb;
  float *C;
  int ldc;
  const float *D;  // ADD
  int ldd;
  const float *bias;  // MLPFWD
  float *Z;           // MLPFWD
  int ldz;
  int vecA, vecB;  // float4 loads allowed (leading dims and bases 16-byte aligned)
};

// Load 4 consecutive elements of a row-major [rows, cols] matrix, zero outside.
__device__ __forceinline__ void ld4(float r[4], const float *base, int row, int col, int rows,
                                    int cols, int ld, int vec) {
  if (vec && row < rows && col + 3 < cols) {
    float4 v = *reinterpret_cast<const float4 *>(base + size_t(row) * ld + col);
    r[0] = v.x; r[1] = v.y; r[2] = v.z; r[3] = v.w;
  } else {
#pragma unroll
    for (int j = 0; j < 4; ++j)
      r[j] = (row < rows && col + j < cols) ? base[size_t(row) * ld + col + j] : 0.f;
  }
}

template <int WT, bool TA, bool TB, int EPI>
__global__ __launch_bounds__(256) void k_gemm_f32(GemmArgs p) {
  constexpr int BMN = 2 * WT;                 // block tile side
  constexpr int CH_A = BMN * BK / 4;          // float4 chunks per operand slice
  __shared__ float As[2][BK][BMN + PAD];
  __shared__ float Bs[2][BK][BMN + PAD];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int m0 = blockIdx.y * BMN, n0 = blockIdx.x * BMN;
  const int wm = (wave >> 1) * WT, wn = (wave & 1) * WT;

  float ra[4], rb[4];
  auto gload = [&](int k0) {
    if (tid < CH_A) {
      if (!TA) {  // A row-major [M,K]: chunk = 4 k's of one row
        int mr = tid / (BK / 4), kc = (tid % (BK / 4)) * 4;
        ld4(ra, p.A, m0 + mr, k0 + kc, p.M, p.K, p.lda, p.vecA);
      } else {    // A stored [K,M]: chunk = 4 m's of one k
        int kr = tid / (BMN / 4), mc = (tid % (BMN / 4)) * 4;
        ld4(ra, p.A, k0 + kr, m0 + mc, p.K, p.M, p.lda, p.vecA);
      }
      if (!TB) {  // B row-major [K,N]
        int kr = tid / (BMN / 4), nc = (tid % (BMN / 4)) * 4;
        ld4(rb, p.B, k0 + kr, n0 + nc, p.K, p.N, p.ldb, p.vecB);
      } else {    // B stored [N,K]
        int nr = tid / (BK / 4), kc = (tid % (BK / 4)) * 4;
        ld4(rb, p.B, n0 + nr, k0 + kc, p.N, p.K, p.ldb, p.vecB);
      }
    }
  };
  auto sstore = [&](int buf) {
    if (tid < CH_A) {
      if (!TA) {
        int mr = tid / (BK / 4), kc = (tid % (BK / 4)) * 4;
#pragma unroll
        for (int j = 0; j < 4; ++j) As[buf][kc + j][mr] = ra[j];
      } else {
        int kr = tid / (BMN / 4), mc = (tid % (BMN / 4)) * 4;
#pragma unroll
        for (int j = 0; j < 4; ++j) As[buf][kr][mc + j] = ra[j];
      }
      if (!TB) {
        int kr = tid / (BMN / 4), nc = (tid % (BMN / 4)) * 4;
#pragma unroll
        for (int j = 0; j < 4; ++j) Bs[buf][kr][nc + j] = rb[j];
      } else {
        int nr = tid / (BK / 4), kc = (tid % (BK / 4)) * 4;
#pragma unroll
        for (int j = 0; j < 4; ++j) Bs[buf][kc + j][nr] = rb[j];
      }
    }
  };

  using acc_t = typename std::conditional<WT == 32, floatx16, floatx4>::type;
  acc_t acc;
#pragma unroll
  for (int r = 0; r < (WT == 32 ? 16 : 4); ++r) acc[r] = 0.f;

  const int nk = (p.K + BK - 1) / BK;
  gload(0);
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    sstore(buf);
    __syncthreads();
    if (kt + 1 < nk) gload((kt + 1) * BK);
    if constexpr (WT == 32) {
#pragma unroll
      for (int kk = 0; kk < BK; kk += 2) {
        float a = As[buf][kk + (lane >> 5)][wm + (lane & 31)];
        float b = Bs[buf][kk + (lane >> 5)][wn + (lane & 31)];
        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, acc, 0, 0, 0);
      }
    } else {
#pragma unroll
      for (int kk = 0; kk < BK; kk += 4) {
        float a = As[buf][kk + (lane >> 4)][wm + (lane & 15)];
        float b = Bs[buf][kk + (lane >> 4)][wn + (lane & 15)];
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, acc, 0, 0, 0);
      }
    }
  }

  // epilogue: accumulator register r of this lane holds element (row, col)
#pragma unroll
  for (int r = 0; r < (WT == 32 ? 16 : 4); ++r) {
    int row, col;
    if (WT == 32) {
      row = 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
      col = lane & 31;
    } else {
      row = 4 * (lane >> 4) + r;
      col = lane & 15;
    }
    const int m = m0 + wm + row, n = n0 + wn + col;
    if (m < p.M && n < p.N) {
      float v = acc[r];
      if (EPI == GEMM_EPI_STORE) {
        p.C[size_t(m) * p.ldc + n] = v;
      } else if (EPI == GEMM_EPI_ADD) {
        p.C[size_t(m) * p.ldc + n] = v + p.D[size_t(m) * p.ldd + n];
      } else {  // MLPFWD
        float z = v + p.bias[n];
        p.Z[size_t(m) * p.ldz + n] = z;
        p.C[size_t(m) * p.ldc + n] = p.A[size_t(m) * p.lda + n] + fmaxf(z, 0.f);
      }
    }
  }
}

template <int WT, bool TA, bool TB, int EPI>
void launch(const GemmArgs &a, hipStream_t s) {
  dim3 grid((a.N + 2 * WT - 1) / (2 * WT), (a.M + 2 * WT - 1) / (2 * WT));
  hipLaunchKernelGGL((k_gemm_f32<WT, TA, TB, EPI>), grid, dim3(256), 0, s, a);
}

template <int WT>
void dispatch(const GemmArgs &a, bool ta, bool tb, int epi, hipStream_t s) {
  if (epi == GEMM_EPI_MLPFWD) {
    launch<WT, false, false, GEMM_EPI_MLPFWD>(a, s);
    return;
  }
#define CKPT_GEMM_CASE(TA_, TB_)                                        \
  if (ta == TA_ && tb == TB_) {                                         \
    if (epi == GEMM_EPI_STORE) launch<WT, TA_, TB_, GEMM_EPI_STORE>(a, s); \
    else launch<WT, TA_, TB_, GEMM_EPI_ADD>(a, s);                       \
    return;                                                             \
  }
  CKPT_GEMM_CASE(false, false)
  CKPT_GEMM_CASE(false, true)
  CKPT_GEMM_CASE(true, false)
  CKPT_GEMM_CASE(true, true)
#undef CKPT_GEMM_CASE
}

inline bool al16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

}  // namespace

void gemm_f32(hipStream_t s, int M, int N, int K, const float *A, int lda, bool ta, const float *B,
              int ldb, bool tb, float *C, int ldc, int epi, const float *D, int ldd,
              const float *bias, float *Z, int ldz) {
  if (M <= 0 || N <= 0) return;
  GemmArgs a{M, N, K, A, lda, B, ldb, C, ldc, D, ldd, bias, Z, ldz, 0, 0};
  a.vecA = (lda % 4 == 0) && al16(A);
  a.vecB = (ldb % 4 == 0) && al16(B);
  // 64x64 block tiles when they alone give at least one block per compute
  // unit; 32x32 tiles otherwise, so that small GEMMs still spread out.
  long tiles64 = long((M + 63) / 64) * ((N + 63) / 64);
  if (tiles64 >= 256)
    dispatch<32>(a, ta, tb, epi, s);
  else
    dispatch<16>(a, ta, tb, epi, s);
}

}  // namespace ckpt
