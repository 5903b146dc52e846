// bf16 GEMM with fp32 accumulation on CDNA4 matrix cores (v_mfma_f32_16x16x32_bf16),
// shared by the dense instantiations (gemm_bf16.hip) and the implicit-GEMM
// convolution instantiations (gemm_bf16_conv.hip).
//
//   C[M,N] (fp32) = epilogue( sum_k A(m,k) B(k,n) )
//   dense A(m,k) = AK ? A[m*lda + k] : A[k*lda + m]     (AK: k contiguous)
//   dense B(k,n) = BK ? B[n*ldb + k] : B[k*ldb + n]     (BK: k contiguous)
// A is bf16, or fp32 rounded to bf16 (nearest even) as it is loaded; B is bf16.
//
// Gather modes read a convolution operand straight from an NHWC bf16 tensor
// (implicit GEMM), 8 channels (16 bytes) per load; geometry g: input H x W,
// output Ho x Wo, kernel R x R, stride S (1 or 2), padding P, C channels of
// the gathered tensor (a power of two, at least 8):
//   GA_FWD    A(m, k): m = (n, ho, wo), k = (kh, kw, ci)
//             -> x[n, ho*S + kh - P, wo*S + kw - P, ci]        (forward)
//   GA_DGRAD  A(m, k): m = (n, h, w), k = (kh, kw, co)
//             -> dy[n, t/S, u/S, co], t = h + P - kh, u = w + P - kw,
//                zero unless S divides t and u            (data gradient)
//   GB_WGRAD  B(k, n): k = (n, ho, wo), n = (kh, kw, ci)
//             -> x[n, ho*S + kh - P, wo*S + kw - P, ci]        (weight gradient)
//   GB_WDGRAD B(k, n): k = (kh, kw, co), n = ci -> W[co, kh, kw, ci]  (the
//             forward weights [Co, R, R, Ci] read as the data gradient's B)
// Out-of-image taps read zero.
//
// Block = 256 threads = 4 wavefronts in a WM x WN grid; each wavefront owns a
// (BM/WM) x (BN/WN) tile of 16x16 accumulators.  K advances in slices of 32
// through double-buffered LDS stored k-contiguous ([m][k] and [n][k]), so
// every lane reads its MFMA operand (8 consecutive k of one row) as one
// 16-byte LDS load.  Operands stored the other way round are transposed while
// they are written to LDS.  Every output element is reduced over K in one
// fixed order (bit-reproducible).
//
// Epilogues: STORE C = acc (+ bias[n]); ADD C = acc + D (D may alias C);
// ADDMASK C = acc + (Ym > 0 ? D : 0) with Ym bf16 shaped like D;
// BF16STATS Cb = bf16(acc) and, per workgroup row of tiles, float64 sums of
// the rounded values and their squares per column (batch-norm statistics:
// stats[blockIdx.y][2][N]).  Split-K (gridDim.z > 1): workgroup z reduces the
// k range [z*kper, (z+1)*kper) and stores its partial product to
// C + z*M*ldc (STORE only); the partials are then added in z order.
#pragma once

#include <hip/hip_runtime.h>

#include <type_traits>

#include "kernels.h"

namespace ckpt {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

namespace gb {

constexpr int KS = 32;      // k per LDS slice
constexpr int KP = KS + 8;  // padded row (bf16 elements): 80-byte rows

enum { G_DENSE = 0, GA_FWD = 1, GA_DGRAD = 2, GB_WGRAD = 3, GB_WDGRAD = 4 };

struct Args {
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
  const __bf16 *Ym;  // ADDMASK mask
  __bf16 *Cb;        // BF16STATS output
  double *stats;     // BF16STATS partial sums
  int kper;          // split-K: k per workgroup (multiple of 32)
  // gather geometry
  int H, W, Ho, Wo, R, S, P, cshift;
  float inv_wo, inv_ho;
};

__device__ __forceinline__ __bf16 to_bf16(float x) { return (__bf16)x; }

__device__ __forceinline__ void zero8(__bf16 r[8]) {
#pragma unroll
  for (int u = 0; u < 8; ++u) r[u] = (__bf16)0.f;
}

__device__ __forceinline__ void vload8(__bf16 r[8], const __bf16 *p) {
  const bf16x8 v = *reinterpret_cast<const bf16x8 *>(p);
#pragma unroll
  for (int u = 0; u < 8; ++u) r[u] = v[u];
}

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
      vload8(r, p);
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

// q = x / d for 0 <= x < 2^24 (float estimate, then corrected)
__device__ __forceinline__ int divq(int x, int d, float inv) {
  int q = int(float(x) * inv);
  int r = x - q * d;
  if (r < 0) { --q; r += d; }
  if (r >= d) ++q;
  return q;
}

// kernel tap (kh, kw) of tap index t = kh*R + kw, R in {1, 3} or general
__device__ __forceinline__ void tap_hw(int t, int R, int &kh, int &kw) {
  kh = R == 1 ? 0 : (R == 3 ? (t * 11) >> 5 : t / R);
  kw = t - kh * R;
}

// Per-chunk row state of the A gathers: the output (GA_FWD) or input
// (GA_DGRAD) pixel of the chunk's row m, fixed for the whole k loop.
struct RowPix {
  int img, y, x;  // image, row, column
  bool ok;
};

__device__ __forceinline__ RowPix row_pixel(const Args &p, int m, int h, int w) {
  RowPix r;
  r.ok = m < p.M;
  const int mm = r.ok ? m : 0;
  const int t = divq(mm, w, 1.0f / float(w));
  r.x = mm - t * w;
  r.img = divq(t, h, 1.0f / float(h));
  r.y = t - r.img * h;
  return r;
}

template <int GA>
__device__ __forceinline__ void gatherA(__bf16 r[8], const Args &p, const __bf16 *A, const RowPix &rp,
                                        int k, int kend) {
  if (!rp.ok || k >= kend) { zero8(r); return; }
  const int C = 1 << p.cshift;
  const int tap = k >> p.cshift, ch = k & (C - 1);
  int kh, kw;
  tap_hw(tap, p.R, kh, kw);
  if constexpr (GA == GA_FWD) {
    const int hi = rp.y * p.S + kh - p.P, wi = rp.x * p.S + kw - p.P;
    if (hi < 0 || hi >= p.H || wi < 0 || wi >= p.W) { zero8(r); return; }
    vload8(r, A + ((size_t(rp.img) * p.H + hi) * p.W + wi) * C + ch);
  } else {
    const int t = rp.y + p.P - kh, u = rp.x + p.P - kw;
    const int sm = p.S - 1;  // S in {1, 2}
    if (t < 0 || u < 0 || (t & sm) || (u & sm)) { zero8(r); return; }
    const int ho = t >> sm, wo = u >> sm;
    if (ho >= p.Ho || wo >= p.Wo) { zero8(r); return; }
    vload8(r, A + ((size_t(rp.img) * p.Ho + ho) * p.Wo + wo) * C + ch);
  }
}

// Per-chunk column state of GB_WGRAD: the tap and channel of column n.
struct ColTap {
  int kh, kw, ch;
  bool ok;
};

__device__ __forceinline__ ColTap col_tap(const Args &p, int n) {
  ColTap c;
  c.ok = n < p.N;
  const int C = 1 << p.cshift;
  const int t = (c.ok ? n : 0) >> p.cshift;
  c.ch = (c.ok ? n : 0) & (C - 1);
  tap_hw(t, p.R, c.kh, c.kw);
  return c;
}

__device__ __forceinline__ void gatherB_wgrad(__bf16 r[8], const Args &p, const ColTap &ct, int k,
                                              int kend) {
  if (!ct.ok || k >= kend) { zero8(r); return; }
  const int t = divq(k, p.Wo, p.inv_wo);
  const int wo = k - t * p.Wo;
  const int img = divq(t, p.Ho, p.inv_ho);
  const int ho = t - img * p.Ho;
  const int hi = ho * p.S + ct.kh - p.P, wi = wo * p.S + ct.kw - p.P;
  if (hi < 0 || hi >= p.H || wi < 0 || wi >= p.W) { zero8(r); return; }
  vload8(r, p.B + ((size_t(img) * p.H + hi) * p.W + wi) * (size_t(1) << p.cshift) + ct.ch);
}

__device__ __forceinline__ void gatherB_wdgrad(__bf16 r[8], const Args &p, int k, int n, int kend) {
  if (k >= kend || n >= p.N) { zero8(r); return; }
  const int Co = 1 << p.cshift;
  const int tap = k >> p.cshift, co = k & (Co - 1);
  vload8(r, p.B + (size_t(co) * p.R * p.R + tap) * p.N + n);
}

template <int BM, int BN, int WM, int WN, bool AK, bool BK, typename TA, int EPI, int GA, int GB>
__global__ __launch_bounds__(256) void k_gemm_bf16(Args p) {
  constexpr int TM = BM / WM / 16, TN = BN / WN / 16;  // 16x16 tiles per wavefront
  static_assert(WM * WN == 4 && TM >= 1 && TN >= 1, "wave grid");
  static_assert(GA == G_DENSE || (AK && std::is_same<TA, __bf16>::value), "A gathers are k-contiguous bf16");
  static_assert(GB == G_DENSE || !BK, "B gathers are n-contiguous");
  constexpr int CHA = BM * KS / 8, CHB = BN * KS / 8;  // 8-element chunks per slice
  constexpr int PA = (CHA + 255) / 256, PB = (CHB + 255) / 256;
  __shared__ __align__(16) __bf16 As[2][BM][KP];
  __shared__ __align__(16) __bf16 Bs[2][BN][KP];
  static_assert(EPI != GEMM_EPI_BF16STATS || WM * 4 * 2 * BN * 8 <= int(sizeof(As)), "stats scratch");

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int i16 = lane & 15, q = lane >> 4;
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
  const int kbeg = blockIdx.z * p.kper;
  const int kend = min(p.K, kbeg + p.kper);
  const int wm = (wave / WN) * (BM / WM), wn = (wave % WN) * (BN / WN);
  const TA *A = static_cast<const TA *>(p.A);

  // fixed per-chunk gather state
  RowPix rpix[GA != G_DENSE ? PA : 1];
  ColTap ctap[GB == GB_WGRAD ? PB : 1];
  if constexpr (GA != G_DENSE) {
#pragma unroll
    for (int c = 0; c < PA; ++c) {
      const int e = min(tid + c * 256, CHA - 1);
      const int m = m0 + e / (KS / 8);
      rpix[c] = GA == GA_FWD ? row_pixel(p, m, p.Ho, p.Wo) : row_pixel(p, m, p.H, p.W);
    }
  }
  if constexpr (GB == GB_WGRAD) {
#pragma unroll
    for (int c = 0; c < PB; ++c) {
      const int e = min(tid + c * 256, CHB - 1);
      ctap[c] = col_tap(p, n0 + (e % (BN / 8)) * 8);
    }
  }

  __bf16 ra[PA][8], rb[PB][8];
  auto gload = [&](int k0) {
#pragma unroll
    for (int c = 0; c < PA; ++c) {
      const int e = tid + c * 256;
      if (e < CHA) {
        if (AK) {  // chunk = 8 k of one m
          const int mr = e / (KS / 8), kc = (e % (KS / 8)) * 8;
          if constexpr (GA != G_DENSE)
            gatherA<GA>(ra[c], p, reinterpret_cast<const __bf16 *>(A), rpix[c], k0 + kc, kend);
          else
            ld8<TA>(ra[c], A, m0 + mr, k0 + kc, p.M, kend, p.lda);
        } else {   // chunk = 8 m of one k
          const int kr = e / (BM / 8), mc = (e % (BM / 8)) * 8;
          ld8<TA>(ra[c], A, k0 + kr, m0 + mc, kend, p.M, p.lda);
        }
      }
    }
#pragma unroll
    for (int c = 0; c < PB; ++c) {
      const int e = tid + c * 256;
      if (e < CHB) {
        if (BK) {
          const int nr = e / (KS / 8), kc = (e % (KS / 8)) * 8;
          ld8<__bf16>(rb[c], p.B, n0 + nr, k0 + kc, p.N, kend, p.ldb);
        } else {
          const int kr = e / (BN / 8), nc = (e % (BN / 8)) * 8;
          if constexpr (GB == GB_WGRAD)
            gatherB_wgrad(rb[c], p, ctap[c], k0 + kr, kend);
          else if constexpr (GB == GB_WDGRAD)
            gatherB_wdgrad(rb[c], p, k0 + kr, n0 + nc, kend);
          else
            ld8<__bf16>(rb[c], p.B, k0 + kr, n0 + nc, kend, p.N, p.ldb);
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

  const int nk = kend > kbeg ? (kend - kbeg + KS - 1) / KS : 0;
  if (nk > 0) gload(kbeg);
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    sstore(buf);
    __syncthreads();
    if (kt + 1 < nk) gload(kbeg + (kt + 1) * KS);
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

  if constexpr (EPI == GEMM_EPI_BF16STATS) {
    // per column: sums over this wavefront's rows, then over the lane groups
    // and the WM wavefronts sharing the column, in a fixed order
    double s1[TN], s2[TN];
#pragma unroll
    for (int b = 0; b < TN; ++b) s1[b] = s2[b] = 0.0;
#pragma unroll
    for (int a = 0; a < TM; ++a)
#pragma unroll
      for (int b = 0; b < TN; ++b)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int m = m0 + wm + a * 16 + 4 * q + r, n = n0 + wn + b * 16 + i16;
          if (m < p.M && n < p.N) {
            const __bf16 h = (__bf16)acc[a][b][r];
            p.Cb[size_t(m) * p.ldc + n] = h;
            const double v = double(float(h));
            s1[b] += v;
            s2[b] += v * v;
          }
        }
    __syncthreads();
    double *red = reinterpret_cast<double *>(&As[0][0][0]);  // [WM*4][2][BN]
    const int wr = wave / WN;
#pragma unroll
    for (int b = 0; b < TN; ++b) {
      const int col = wn + b * 16 + i16;
      red[((wr * 4 + q) * 2 + 0) * BN + col] = s1[b];
      red[((wr * 4 + q) * 2 + 1) * BN + col] = s2[b];
    }
    __syncthreads();
    if (tid < 2 * BN) {
      const int which = tid / BN, col = tid % BN;
      double t = 0.0;
      for (int k = 0; k < WM * 4; ++k) t += red[(k * 2 + which) * BN + col];
      if (n0 + col < p.N) p.stats[(size_t(blockIdx.y) * 2 + which) * p.N + n0 + col] = t;
    }
  } else {
    float *Cz = p.C + size_t(blockIdx.z) * p.M * p.ldc;
#pragma unroll
    for (int a = 0; a < TM; ++a)
#pragma unroll
      for (int b = 0; b < TN; ++b)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int m = m0 + wm + a * 16 + 4 * q + r, n = n0 + wn + b * 16 + i16;
          if (m < p.M && n < p.N) {
            float v = acc[a][b][r];
            if (EPI == GEMM_EPI_ADD) {
              v += p.D[size_t(m) * p.ldd + n];
            } else if (EPI == GEMM_EPI_ADDMASK) {
              const size_t o = size_t(m) * p.ldd + n;
              if (float(p.Ym[o]) > 0.f) v += p.D[o];
            } else if (p.bias) {
              v += p.bias[n];
            }
            Cz[size_t(m) * p.ldc + n] = v;
          }
        }
  }
}

// Tile by shape: 128x128 when that alone fills the GPU, else 64x64, else 64x32.
struct Tile {
  int BM, BN;
};

inline Tile tile_of(int M, int N) {
  const long big = long((M + 127) / 128) * ((N + 127) / 128);
  if (M >= 256 && big >= 128) return {128, 128};
  if (long((M + 63) / 64) * ((N + 63) / 64) >= 64) return {64, 64};
  return {64, 32};
}

template <int BM, int BN, int WM, int WN, bool AK, bool BK, typename TA, int GA, int GB>
void launch_epi(const Args &a, int epi, int splits, hipStream_t s) {
  dim3 grid((a.N + BN - 1) / BN, (a.M + BM - 1) / BM, splits);
  if (epi == GEMM_EPI_ADD) {
    hipLaunchKernelGGL((k_gemm_bf16<BM, BN, WM, WN, AK, BK, TA, GEMM_EPI_ADD, GA, GB>), grid, dim3(256), 0, s, a);
    return;
  }
  if constexpr (std::is_same<TA, __bf16>::value) {
    if (epi == GEMM_EPI_ADDMASK) {
      hipLaunchKernelGGL((k_gemm_bf16<BM, BN, WM, WN, AK, BK, TA, GEMM_EPI_ADDMASK, GA, GB>), grid, dim3(256), 0, s, a);
      return;
    }
    if (epi == GEMM_EPI_BF16STATS) {
      hipLaunchKernelGGL((k_gemm_bf16<BM, BN, WM, WN, AK, BK, TA, GEMM_EPI_BF16STATS, GA, GB>), grid, dim3(256), 0, s, a);
      return;
    }
  }
  hipLaunchKernelGGL((k_gemm_bf16<BM, BN, WM, WN, AK, BK, TA, GEMM_EPI_STORE, GA, GB>), grid, dim3(256), 0, s, a);
}

template <bool AK, bool BK, typename TA, int GA, int GB>
void pick_tile(const Args &a, int epi, int splits, hipStream_t s) {
  const Tile t = tile_of(a.M, a.N);
  if (t.BM == 128) launch_epi<128, 128, 2, 2, AK, BK, TA, GA, GB>(a, epi, splits, s);
  else if (t.BN == 64) launch_epi<64, 64, 2, 2, AK, BK, TA, GA, GB>(a, epi, splits, s);
  else launch_epi<64, 32, 4, 1, AK, BK, TA, GA, GB>(a, epi, splits, s);
}

}  // namespace gb
}  // namespace ckpt
