// fp32 GEMM on CDNA4 matrix cores (v_mfma_f32_32x32x2f32).
//
//   C[M,N] = epilogue( op(A)[M,K] * op(B)[K,N] )
//   op(A)(m,k) = TA ? A[k*lda + m] : A[m*lda + k]
//   op(B)(k,n) = TB ? B[n*ldb + k] : B[k*ldb + n]
//
// Block = 256 threads = 4 wavefronts; each wavefront owns a 32 x 32 output
// tile (one 32x32x2 accumulator, 16 floats per lane).  Two shapes:
//   KS = 1  block tile 64 x 64, waves in a 2 x 2 grid, K slices of 32;
//   KS = 4  block tile 32 x 32, the four waves split every K slice of 128
//           into quarters and their accumulators are added in LDS in wave
//           order ((w0 + w1) + w2) + w3 -- four times the waves for GEMMs
//           whose output has few 64 x 64 tiles.
// Operand slices are staged through LDS k-contiguous ([m][k] and [n][k],
// rows padded by 4 floats), double-buffered, with the global loads of the
// next two slices in flight during the current slice's MFMAs.  Within a
// wave's 32-wide k range, MFMA j takes k = 16 h + j in lane half h (h = lane / 32) for both
// operands -- a fixed permutation of the reduction, so each lane reads 16
// consecutive floats (four 16-byte LDS reads) per operand.  Every output
// element is reduced over K in one order fixed by the shape alone.
//
// Epilogues:
//   STORE    C = acc
//   ADD      C = acc + D                      (backward: dx = dy + dr W^T)
//   MLPFWD   Z = acc + bias;  C = A + relu(Z) (residual block y = x + relu(xW+b);
//                                               requires !TA and K == N)
//   BIAS     C = acc + bias
#include <hip/hip_runtime.h>

#include "common.h"
#include "kernel_args.h"
#include "kernels.h"
#include "launch.h"

namespace ckpt {

typedef float floatx16 __attribute__((ext_vector_type(16)));

namespace {

constexpr int PAD = 4;


// 4 KB of zeros in device memory: an element outside its operand is loaded
// from here (16 bytes per thread, spread over many cache lines), so no loaded
// value is masked afterwards and nothing waits for a load before it is
// written to LDS a slice later.
static __device__ __align__(16) const float g_zero_area[1024] = {};
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(1))) const f32x4 global_f32x4;
typedef __attribute__((address_space(1))) const float global_float;

// 4 consecutive elements of a row-major [rows, cols] matrix, zero outside.
// Branch-free (an outside address is replaced by the zero chunk), so the loads
// of a slice stay in flight together; the pointers are cast to the global
// address space so that the loads are global loads.  VEC: one 16-byte load;
// needs ld and cols multiples of 4 and a 16-byte aligned base, so a chunk is
// either wholly inside or wholly outside.
template <bool VEC>
__device__ __forceinline__ float4 ld4(const float *base, int row, int col, int rows, int cols,
                                      int ld) {
  if (VEC) {
    const bool ok = (row < rows) & (col < cols);
    const float *z = g_zero_area + 4 * (threadIdx.x & 255);
    const f32x4 v = *(global_f32x4 *)(ok ? base + size_t(row) * ld + col : z);
    return make_float4(v.x, v.y, v.z, v.w);
  }
  float r[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const bool ok = (row < rows) & (col + j < cols);
    r[j] = *(global_float *)(ok ? base + size_t(row) * ld + col + j : g_zero_area + 4 * (threadIdx.x & 255));
  }
  return make_float4(r[0], r[1], r[2], r[3]);
}

template <int KS, bool TA, bool TB, int EPI, bool VEC>
__global__ __launch_bounds__(256) void k_gemm_f32(GemmArgs p) {
  constexpr int BM = KS == 1 ? 64 : 32, BN = BM;  // block tile
  constexpr int BK = 32 * KS;                      // k slice
  constexpr int LD = BK + PAD;                     // LDS row stride (floats)
  constexpr int NCH = BM * BK / 4 / 256;           // float4 chunks per thread per operand
  static_assert(NCH * 256 * 4 == BM * BK, "tile / thread mismatch");
  __shared__ __attribute__((aligned(16))) float smem[2 * (BM + BN) * LD];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // Workgroups reach the eight XCDs (one L2 each) in turn; the linear id is
  // remapped so that each XCD takes a contiguous run of tiles, m fastest: an
  // XCD then reads a few column tiles of B (plus A) instead of all of B.
  int tm, tn;
  {
    const int G = gridDim.x * gridDim.y, id = blockIdx.x + gridDim.x * blockIdx.y;
    const int q8 = G / 8, r8 = G % 8, x8 = id % 8;
    const int L = x8 * q8 + (x8 < r8 ? x8 : r8) + id / 8;
    tm = L % gridDim.y;
    tn = L / gridDim.y;
  }
  const int m0 = tm * BM, n0 = tn * BN;
  const int kw = KS == 1 ? 0 : wave;                         // k quarter of this wave
  const int wm = KS == 1 ? (wave >> 1) * 32 : 0, wn = KS == 1 ? (wave & 1) * 32 : 0;

  auto gload = [&](float4 (&ra)[NCH], float4 (&rb)[NCH], int k0) {
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      const int ch = tid + 256 * c;
      if (!TA) {  // A row-major [M,K]: a chunk is 4 k's of one row
        ra[c] = ld4<VEC>(p.A, m0 + ch / (BK / 4), k0 + (ch % (BK / 4)) * 4, p.M, p.K, p.lda);
      } else {    // A stored [K,M]: a chunk is 4 m's of one k
        ra[c] = ld4<VEC>(p.A, k0 + ch / (BM / 4), m0 + (ch % (BM / 4)) * 4, p.K, p.M, p.lda);
      }
      if (TB) {   // B stored [N,K]: 4 k's of one n
        rb[c] = ld4<VEC>(p.B, n0 + ch / (BK / 4), k0 + (ch % (BK / 4)) * 4, p.N, p.K, p.ldb);
      } else {    // B row-major [K,N]: 4 n's of one k
        rb[c] = ld4<VEC>(p.B, k0 + ch / (BN / 4), n0 + (ch % (BN / 4)) * 4, p.K, p.N, p.ldb);
      }
    }
  };
  auto sstore = [&](const float4 (&ra)[NCH], const float4 (&rb)[NCH], int buf) {
    float *As = smem + buf * (BM + BN) * LD, *Bs = As + BM * LD;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      const int ch = tid + 256 * c;
      if (!TA) {
        *reinterpret_cast<float4 *>(As + (ch / (BK / 4)) * LD + (ch % (BK / 4)) * 4) = ra[c];
      } else {
        const int k = ch / (BM / 4), m = (ch % (BM / 4)) * 4;
        As[(m + 0) * LD + k] = ra[c].x;
        As[(m + 1) * LD + k] = ra[c].y;
        As[(m + 2) * LD + k] = ra[c].z;
        As[(m + 3) * LD + k] = ra[c].w;
      }
      if (TB) {
        *reinterpret_cast<float4 *>(Bs + (ch / (BK / 4)) * LD + (ch % (BK / 4)) * 4) = rb[c];
      } else {
        const int k = ch / (BN / 4), n = (ch % (BN / 4)) * 4;
        Bs[(n + 0) * LD + k] = rb[c].x;
        Bs[(n + 1) * LD + k] = rb[c].y;
        Bs[(n + 2) * LD + k] = rb[c].z;
        Bs[(n + 3) * LD + k] = rb[c].w;
      }
    }
  };

  floatx16 acc;
#pragma unroll
  for (int r = 0; r < 16; ++r) acc[r] = 0.f;

  const int h = lane >> 5, l32 = lane & 31;
  auto compute = [&](int buf) {
    const float *As = smem + buf * (BM + BN) * LD, *Bs = As + BM * LD;
    const float *pa = As + (wm + l32) * LD + kw * 32 + h * 16;
    const float *pb = Bs + (wn + l32) * LD + kw * 32 + h * 16;
    float4 a4[4], b4[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      a4[q] = *reinterpret_cast<const float4 *>(pa + 4 * q);
      b4[q] = *reinterpret_cast<const float4 *>(pb + 4 * q);
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a4[q].x, b4[q].x, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a4[q].y, b4[q].y, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a4[q].z, b4[q].z, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a4[q].w, b4[q].w, acc, 0, 0, 0);
    }
  };

  // slices kt+1 and kt+2 are in flight in registers while slice kt is
  // multiplied out of LDS buffer kt & 1.  The loop body has no branches (a
  // branch there makes the compiler wait for every load at each iteration):
  // it runs while two more slices follow, and the last one or two slices are
  // multiplied after it.
  const int nk = (p.K + BK - 1) / BK;
  // k origin of slice s; a slice past K re-reads the last one (real,
  // spread-out addresses; it is never multiplied)
  auto kslice = [&](int s) { return max(0, min(s, nk - 1)) * BK; };
  float4 ra0[NCH], rb0[NCH], ra1[NCH], rb1[NCH];
  gload(ra0, rb0, kslice(0));
  gload(ra1, rb1, kslice(1));
  sstore(ra0, rb0, 0);
  __syncthreads();
  int kt = 0;
  for (; kt + 2 < nk; kt += 2) {
    gload(ra0, rb0, kslice(kt + 2));
    compute(0);
    sstore(ra1, rb1, 1);
    __syncthreads();
    gload(ra1, rb1, kslice(kt + 3));
    compute(1);
    sstore(ra0, rb0, 0);
    __syncthreads();
  }
  compute(0);  // slice kt
  if (kt + 1 < nk) {
    sstore(ra1, rb1, 1);
    __syncthreads();
    compute(1);
  }

  // accumulator register r of a lane holds element (row, col) of its 32x32 tile
  auto rc = [&](int r, int &row, int &col) {
    row = 8 * (r >> 2) + 4 * h + (r & 3);
    col = l32;
  };
  auto emit = [&](int m, int n, float v) {
    if (m < p.M && n < p.N) {
      if (EPI == GEMM_EPI_STORE) {
        p.C[size_t(m) * p.ldc + n] = v;
      } else if (EPI == GEMM_EPI_ADD) {
        p.C[size_t(m) * p.ldc + n] = v + p.D[size_t(m) * p.ldd + n];
      } else if (EPI == GEMM_EPI_BIAS) {
        p.C[size_t(m) * p.ldc + n] = v + p.bias[n];
      } else {  // MLPFWD
        const float z = v + p.bias[n];
        p.Z[size_t(m) * p.ldz + n] = z;
        p.C[size_t(m) * p.ldc + n] = p.A[size_t(m) * p.lda + n] + fmaxf(z, 0.f);
      }
    }
  };
  if (KS == 1) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      int row, col;
      rc(r, row, col);
      emit(m0 + wm + row, n0 + wn + col, acc[r]);
    }
  } else {
    // the four k quarters, added in wave order (the last loop iteration's
    // barrier has retired every read of the staging buffers)
    float *red = smem;  // [4][32][33]
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      int row, col;
      rc(r, row, col);
      red[(wave * 32 + row) * 33 + col] = acc[r];
    }
    __syncthreads();
#pragma unroll
    for (int e = tid; e < 32 * 32; e += 256) {
      const int row = e >> 5, col = e & 31;
      const float v = ((red[row * 33 + col] + red[(32 + row) * 33 + col]) + red[(64 + row) * 33 + col]) +
                      red[(96 + row) * 33 + col];
      emit(m0 + row, n0 + col, v);
    }
  }
}

template <int KS, bool TA, bool TB, int EPI>
void launch(const GemmArgs &a, bool vec, hipStream_t s) {
  constexpr int T = KS == 1 ? 64 : 32;
  dim3 grid((a.N + T - 1) / T, (a.M + T - 1) / T);
  if (vec)
    launch_timed((k_gemm_f32<KS, TA, TB, EPI, true>), grid, dim3(256), 0, s, a);
  else
    launch_timed((k_gemm_f32<KS, TA, TB, EPI, false>), grid, dim3(256), 0, s, a);
}

template <int KS>
void dispatch(const GemmArgs &a, bool ta, bool tb, int epi, bool vec, hipStream_t s) {
  if (epi == GEMM_EPI_MLPFWD) {
    launch<KS, false, false, GEMM_EPI_MLPFWD>(a, vec, s);
    return;
  }
  if (epi == GEMM_EPI_BIAS) {
    if (ta || tb) fail(CKPT_E_UNSUPPORTED, "gemm_f32: the bias epilogue takes untransposed operands");
    launch<KS, false, false, GEMM_EPI_BIAS>(a, vec, s);
    return;
  }
#define CKPT_GEMM_CASE(TA_, TB_)                                               \
  if (ta == TA_ && tb == TB_) {                                                \
    if (epi == GEMM_EPI_STORE) launch<KS, TA_, TB_, GEMM_EPI_STORE>(a, vec, s); \
    else launch<KS, TA_, TB_, GEMM_EPI_ADD>(a, vec, s);                         \
    return;                                                                    \
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
  GemmArgs a{M, N, K, A, lda, B, ldb, C, ldc, D, ldd, bias, Z, ldz};
  // 16-byte operand loads when every contiguous extent and leading dimension
  // is a multiple of 4 floats and both bases are 16-byte aligned
  const bool vec = lda % 4 == 0 && ldb % 4 == 0 && al16(A) && al16(B) &&
                   (ta ? M : K) % 4 == 0 && (tb ? K : N) % 4 == 0;
  // 64x64 tiles when they alone give a block per compute unit; otherwise
  // 32x32 tiles with the k range split over the block's four waves
  const long tiles64 = long((M + 63) / 64) * ((N + 63) / 64);
  if (tiles64 >= 256)
    dispatch<1>(a, ta, tb, epi, vec, s);
  else
    dispatch<4>(a, ta, tb, epi, vec, s);
}

}  // namespace ckpt
