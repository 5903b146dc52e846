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
//   GA_CAT    A(m, k) = A[m, k] for k < K1, A2[m, k - K1] after: two
//             k-contiguous bf16 operands side by side along k
//   GA_FWDT, GA_DGRADT  GA_FWD and GA_DGRAD (the latter with S = 1) when C
//             and the k range per workgroup are multiples of the k slice and
//             R * R <= 32: each slice then lies in one tap, so the tap and its
//             offset are the same for the whole workgroup, and a chunk's
//             source is its row's fixed address plus that offset, or zero
//             when the tap is outside the image (a per-row mask of taps)
//             (direct loop only)
// Out-of-image taps read zero.
//
// Block = 4 or 8 wavefronts (256 or 512 threads) in a WM x WN grid; each wavefront owns a
// (BM/WM) x (BN/WN) tile of 16x16 accumulators.  K advances in slices of 64
// (two 32-deep MFMA steps): straight from global memory into a ring of two
// or three LDS stages (the direct loop), or through registers two slices
// ahead into double-buffered LDS.  A k-contiguous operand is stored [row][k], so every lane
// reads its MFMA operand (8 consecutive k of one row) as one 16-byte LDS
// load; a k-major operand stays k-major in LDS and reaches the matrix cores
// through gfx950's transposing LDS read.  Every output element is reduced
// over K in one fixed order (bit-reproducible).
//
// Epilogues: STORE C = acc (+ bias[n]); ADD C = acc + D (D may alias C);
// ADDMASK C = acc + (Ym > 0 ? D : 0) with Ym bf16 shaped like D;
// BF16STATS Cb = bf16(acc) and, per workgroup row of tiles, float64 sums of
// the rounded values and their squares per column (batch-norm statistics:
// stats[m tile][2][N], block-major; none when stats is null; with Rb also the
// batch norm + ReLU of the rounded values); BNBWD C = (Ym > 0) acc and the
// column sums of C and C * (Cv - mean) / std (a batch norm's backward sums);
// ROWSOFTMAX C = acc + bias and each row's (max, sum of exp) per column tile.
// Split-K (gridDim.z > 1): workgroup z reduces the
// k range [z*kper, (z+1)*kper) and stores its partial product to
// C + z*M*ldc (STORE only); the partials are then added in z order.
#pragma once

#include <hip/hip_runtime.h>

#include <type_traits>
#include <utility>

#include "bnb_act.h"
#include "kernels.h"
#include "launch.h"

namespace ckpt {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

namespace gb {

constexpr int cmax(int a, int b) { return a > b ? a : b; }
// do three direct-loop stages of a BM x BN tile (plus an epilogue scratch
// larger than one A stage) leave room for two workgroups per compute unit?
constexpr bool direct_three_stages(int BM, int BN, int epi_scratch) {
  return 3 * (BM + BN) * 64 * 2 + (epi_scratch <= BM * 64 * 2 ? 0 : epi_scratch) <= 80 * 1024;
}

constexpr int KS = 64;      // k per LDS slice: two 32-deep MFMA steps
constexpr int KP = KS + 8;  // padded row (bf16 elements): 144-byte rows

enum { G_DENSE = 0, GA_FWD = 1, GA_DGRAD = 2, GB_WGRAD = 3, GB_WDGRAD = 4, GA_CAT = 5, GA_FWDT = 6,
       GA_DGRADT = 7 };

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
  const __bf16 *Ym;  // ADDMASK / BNBWD mask
  __bf16 *Cb;        // BF16STATS output
  double *stats;     // BF16STATS / BNBWD partial sums
  const __bf16 *Cv;  // BNBWD: the batch norm's input, [M, N]
  const float *bst;  // BNBWD: its mean [N] and 1/std [N]
  float *rstat;      // ROWSOFTMAX: per row and column tile, (max, sum of exp(x - max))
  // BF16STATS with Rb: also Rb = bf16(relu(ag ((Cb - ast[n]) ast[N + n]) + ab
  // [+ Xr])) (the bottleneck units' batch-norm apply, bnb_act.h)
  __bf16 *Rb;
  const __bf16 *Xr;
  const float *ast, *ag, *ab;
  int kper;          // split-K: k per workgroup (multiple of 32)
  // gather geometry
  int H, W, Ho, Wo, R, S, P, cshift;
  int rmagic;  // ceil(2^16 / R): t / R = (t * rmagic) >> 16 for the tap indices used
  const __bf16 *A2;  // GA_CAT: the second operand, from k = K1 on
  int lda2, K1;
  float inv_wo, inv_ho;
  // batched products (nbatch > 0, one k split): workgroup z computes product
  // z, whose A, C and row statistics start bstrA, bstrC and bstrR elements
  // after product z - 1's (B is shared)
  int nbatch;
  int64_t bstrA, bstrC, bstrR;
};

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// A staged operand chunk: 8 bf16 in four dwords, kept as one vector so that
// its global load stays in flight until the chunk is written to LDS.
__device__ __forceinline__ u32x4 zero_chunk() { return u32x4{0u, 0u, 0u, 0u}; }

// 4 KB of zeros in device memory: a chunk outside its operand is loaded from
// here (16 bytes per thread of the workgroup, so the zero loads spread over
// many cache lines instead of all meeting on one).  No loaded value then needs
// masking, so nothing waits for a load before the chunk is written to LDS a
// slice later (a mask applied right after the load made the compiler wait for
// every load of the iteration at the end of each k-loop iteration).
static __device__ __align__(16) const unsigned g_zero_area[1024] = {};

// 16-byte load of p when ok, else of the thread's zero chunk: no branch around
// the load.  The pointer is cast to the global address space so that the load
// is a global (not flat) load, counted by the vector-memory counter only.
typedef __attribute__((address_space(1))) const u32x4 global_u32x4;
__device__ __forceinline__ u32x4 masked16(const void *p, bool ok) {
  const void *z = g_zero_area + 4 * (threadIdx.x & 255);
  return *(global_u32x4 *)(ok ? p : z);
}

__device__ __forceinline__ unsigned pack2(float lo, float hi) {
  const __bf16 a = (__bf16)lo, b = (__bf16)hi;
  return unsigned(__builtin_bit_cast(unsigned short, a)) |
         (unsigned(__builtin_bit_cast(unsigned short, b)) << 16);
}

// 8 consecutive elements of row `row` from column `col` of a row-major
// [rows, cols] matrix of T, zero outside, as bf16.  SAFE: cols and ld are
// multiples of 8 (T = bf16), so a chunk is wholly inside or outside.
template <bool SAFE, typename T>
__device__ __forceinline__ u32x4 ld8(const T *base, int row, int col, int rows, int cols, int ld) {
  if constexpr (SAFE) {
    return masked16(base + size_t(row) * ld + col, (row < rows) & (col < cols));
  } else {
    const bool inrow = row < rows;
    const T *p = base + size_t(row) * ld + col;
    float f[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) f[u] = (inrow && col + u < cols) ? float(p[u]) : 0.f;
    return u32x4{pack2(f[0], f[1]), pack2(f[2], f[3]), pack2(f[4], f[5]), pack2(f[6], f[7])};
  }
}

// MFMA operand (8 consecutive k of one row) from a k-major LDS tile with the
// transposing read: within each 16-lane group, lane 4t + s points at k-row t
// (then t + 4, `step` bytes further) and columns 4s..4s+3 of the group's 16
// rows, and lane i receives column i of k-rows 0..3 (then 4..7).
typedef short short4v __attribute__((ext_vector_type(4)));
__device__ __forceinline__ bf16x8 tr_operand(const unsigned char *p, int step) {
  typedef __attribute__((address_space(3))) short4v lds_short4;
  const short4v lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_short4 *)(p));
  const short4v hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_short4 *)(p + step));
  typedef short short8v __attribute__((ext_vector_type(8)));
  const short8v v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  return __builtin_bit_cast(bf16x8, v);
}

// q = x / d for 0 <= x < 2^24 (float estimate, then corrected)
__device__ __forceinline__ int divq(int x, int d, float inv) {
  int q = int(float(x) * inv);
  int r = x - q * d;
  if (r < 0) { --q; r += d; }
  if (r >= d) ++q;
  return q;
}

// kernel tap (kh, kw) of tap index t = kh*R + kw by a multiply and shift
// (exact while t (R - 1) < 2^16), so the gathers stay free of branches and the
// compiler keeps counting their loads across the k loop
__device__ __forceinline__ void tap_hw(int t, const Args &p, int &kh, int &kw) {
  kh = (t * p.rmagic) >> 16;
  kw = t - kh * p.R;
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
__device__ __forceinline__ u32x4 gatherA(const Args &p, const __bf16 *A, const RowPix &rp, int k, int kend) {
  const int C = 1 << p.cshift;
  const int tap = k >> p.cshift, ch = k & (C - 1);
  int kh, kw;
  tap_hw(tap, p, kh, kw);
  if constexpr (GA == GA_FWD) {
    const int hi = rp.y * p.S + kh - p.P, wi = rp.x * p.S + kw - p.P;
    const bool ok = rp.ok & (k < kend) & (hi >= 0) & (hi < p.H) & (wi >= 0) & (wi < p.W);
    return masked16(A + ((size_t(rp.img) * p.H + hi) * p.W + wi) * C + ch, ok);
  } else {
    const int t = rp.y + p.P - kh, u = rp.x + p.P - kw;
    const int sm = p.S - 1;  // S in {1, 2}
    const int ho = t >> sm, wo = u >> sm;
    const bool ok = rp.ok & (k < kend) & (t >= 0) & (u >= 0) & !(t & sm) & !(u & sm) & (ho < p.Ho) &
                    (wo < p.Wo);
    return masked16(A + ((size_t(rp.img) * p.Ho + ho) * p.Wo + wo) * C + ch, ok);
  }
}

// The same gathers as addresses for the direct global -> LDS loads: the
// chunk's source, or the thread's zero slot when it lies outside.
__device__ __forceinline__ const void *src16(const void *p, bool ok) {
  return ok ? p : static_cast<const void *>(g_zero_area + 4 * (threadIdx.x & 255));
}

template <int GA>
__device__ __forceinline__ const void *gatherA_src(const Args &p, const __bf16 *A, const RowPix &rp, int k,
                                                   int kend) {
  const int C = 1 << p.cshift;
  const int tap = k >> p.cshift, ch = k & (C - 1);
  int kh, kw;
  tap_hw(tap, p, kh, kw);
  if constexpr (GA == GA_FWD) {
    const int hi = rp.y * p.S + kh - p.P, wi = rp.x * p.S + kw - p.P;
    const bool ok = rp.ok & (k < kend) & (hi >= 0) & (hi < p.H) & (wi >= 0) & (wi < p.W);
    return src16(A + ((size_t(rp.img) * p.H + hi) * p.W + wi) * C + ch, ok);
  } else {
    const int t = rp.y + p.P - kh, u = rp.x + p.P - kw;
    const int sm = p.S - 1;
    const int ho = t >> sm, wo = u >> sm;
    const bool ok = rp.ok & (k < kend) & (t >= 0) & (u >= 0) & !(t & sm) & !(u & sm) & (ho < p.Ho) &
                    (wo < p.Wo);
    return src16(A + ((size_t(rp.img) * p.Ho + ho) * p.Wo + wo) * C + ch, ok);
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
  tap_hw(t, p, c.kh, c.kw);
  return c;
}

__device__ __forceinline__ u32x4 gatherB_wgrad(const Args &p, const ColTap &ct, int k, int kend) {
  const int t = divq(k, p.Wo, p.inv_wo);
  const int wo = k - t * p.Wo;
  const int img = divq(t, p.Ho, p.inv_ho);
  const int ho = t - img * p.Ho;
  const int hi = ho * p.S + ct.kh - p.P, wi = wo * p.S + ct.kw - p.P;
  const bool ok = ct.ok & (k < kend) & (hi >= 0) & (hi < p.H) & (wi >= 0) & (wi < p.W);
  return masked16(p.B + ((size_t(img) * p.H + hi) * p.W + wi) * (size_t(1) << p.cshift) + ct.ch, ok);
}

__device__ __forceinline__ const void *gatherB_wgrad_src(const Args &p, const ColTap &ct, int k, int kend) {
  const int t = divq(k, p.Wo, p.inv_wo);
  const int wo = k - t * p.Wo;
  const int img = divq(t, p.Ho, p.inv_ho);
  const int ho = t - img * p.Ho;
  const int hi = ho * p.S + ct.kh - p.P, wi = wo * p.S + ct.kw - p.P;
  const bool ok = ct.ok & (k < kend) & (hi >= 0) & (hi < p.H) & (wi >= 0) & (wi < p.W);
  return src16(p.B + ((size_t(img) * p.H + hi) * p.W + wi) * (size_t(1) << p.cshift) + ct.ch, ok);
}

__device__ __forceinline__ const void *gatherB_wdgrad_src(const Args &p, int k, int n, int kend) {
  const int Co = 1 << p.cshift;
  const int tap = k >> p.cshift, co = k & (Co - 1);
  return src16(p.B + (size_t(co) * p.R * p.R + tap) * p.N + n, (k < kend) & (n < p.N));
}

// 16 bytes from global memory straight into LDS: lane i of the wavefront
// writes lds_wave + 16 i (lds_wave must be the same for the whole wavefront).
typedef __attribute__((address_space(3))) void lds_void_t;
__device__ __forceinline__ void load_lds16(const void *src, unsigned char *lds_wave) {
  __builtin_amdgcn_global_load_lds(src, (lds_void_t *)lds_wave, 16, 0, 0);
}

// s_waitcnt immediate that waits until at most n vector-memory operations
// of this wavefront are outstanding (the other counters left alone)
constexpr int vmcnt_le(int n) { return (n & 15) | ((n >> 4) << 14) | 0x70 | 0xF00; }
// the same, and every LDS read of the wavefront has returned
constexpr int vmcnt_le_lds0(int n) { return (n & 15) | ((n >> 4) << 14) | 0x70; }

// f(integral_constant<int, 0>) ... f(integral_constant<int, N - 1>), unrolled
template <class F, int... I>
__device__ __forceinline__ void unroll_seq(F &f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, class F>
__device__ __forceinline__ void unroll(F &&f) {
  unroll_seq(f, std::make_integer_sequence<int, N>{});
}

__device__ __forceinline__ u32x4 gatherB_wdgrad(const Args &p, int k, int n, int kend) {
  const int Co = 1 << p.cshift;
  const int tap = k >> p.cshift, co = k & (Co - 1);
  return masked16(p.B + (size_t(co) * p.R * p.R + tap) * p.N + n, (k < kend) & (n < p.N));
}

// STG (direct loop only): the number of LDS stages, 2 to 5; 0 chooses three
// where two workgroups then still fit a compute unit's LDS, else two
template <int BM, int BN, int WM, int WN, bool AK, bool BK, typename TA, int EPI, int GA, int GB, bool SAFE,
          int STG = 0>
__global__ __launch_bounds__(64 * WM * WN) void k_gemm_bf16(Args p) {
  constexpr int TM = BM / WM / 16, TN = BN / WN / 16;  // 16x16 tiles per wavefront
  constexpr int NT = 64 * WM * WN;                      // threads
  static_assert((WM * WN == 4 || WM * WN == 8) && TM >= 1 && TN >= 1, "wave grid");
  static_assert(GA == G_DENSE || (AK && std::is_same<TA, __bf16>::value), "A gathers are k-contiguous bf16");
  static_assert(GB == G_DENSE || !BK, "B gathers are n-contiguous");
  constexpr int CHA = BM * KS / 8, CHB = BN * KS / 8;  // 8-element chunks per slice
  constexpr int PA = (CHA + NT - 1) / NT, PB = (CHB + NT - 1) / NT;
  constexpr int WC = BN / WN;                           // columns per wavefront
  constexpr bool DIRECT = SAFE && std::is_same<TA, __bf16>::value;
  static_assert(NT == 256 || (DIRECT && CHA % NT == 0 && CHB % NT == 0),
                "eight wavefronts: the direct loop, whole chunk rounds");
  // staging row pitch (floats): padded for the register-staged loop; unpadded
  // for the direct loop, whose first stage then holds the staging rows
  constexpr int SP = DIRECT ? WC : WC + 4;
  // Two main loops (chosen at compile time):
  // * direct (aligned bf16 operands): every 16-byte chunk goes from global
  //   memory straight into LDS (global_load_lds_dwordx4) into a two- or
  //   three-stage ring, one LDS object per stage and operand so that the compiler knows
  //   which in-flight loads an LDS read depends on; layouts are unpadded and
  //   XOR-swizzled so that the MFMA operand reads are free of bank conflicts;
  // * register-staged (an fp32 A, or rows whose extent is not a multiple of
  //   8 elements): chunks are loaded into registers two slices ahead and
  //   written to a double-buffered padded LDS tile.
  // epilogue scratch: staging rows, and the column sums of BF16STATS / BNBWD
  constexpr int EPI_SCR = cmax(WM * WN * 16 * SP * 4,
                               cmax(EPI == GEMM_EPI_BF16STATS ? WM * 4 * 2 * BN * 8 : 0,
                                    EPI == GEMM_EPI_BNBWD ? WM * (64 / (WC / 4)) * 2 * BN * 8 : 0));
  // ROWSOFTMAX: each wavefront column's (max, sum of exp) per row of the tile
  __shared__ float rsm[EPI == GEMM_EPI_ROWSOFTMAX ? WN * BM * 2 : 1];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int i16 = lane & 15, q = lane >> 4;
  // Workgroups go to the eight XCDs (one L2 each) in turn; the linear
  // workgroup id is remapped so that each XCD takes a contiguous run of
  // tiles (n fastest, then m, then the k split): the n tiles of one m tile,
  // and neighbouring m tiles whose gathers share input rows, read their
  // operands through one L2.
  int tn, tm, tz;
  {
    const int G = gridDim.x * gridDim.y * gridDim.z;
    const int id = blockIdx.x + gridDim.x * (blockIdx.y + gridDim.y * blockIdx.z);
    const int q8 = G / 8, r8 = G % 8, x8 = id % 8;
    const int L = x8 * q8 + (x8 < r8 ? x8 : r8) + id / 8;
    tn = L % gridDim.x;
    tm = (L / gridDim.x) % gridDim.y;
    tz = L / (gridDim.x * gridDim.y);
  }
  int bz = 0;  // product of a batch
  if (p.nbatch > 0) {
    bz = tz;
    tz = 0;
  }
  const int m0 = tm * BM, n0 = tn * BN;
  const int kbeg = tz * p.kper;
  const int kend = min(p.K, kbeg + p.kper);
  const int wm = (wave / WN) * (BM / WM), wn = (wave % WN) * (BN / WN);
  const TA *A = static_cast<const TA *>(p.A) + size_t(bz) * p.bstrA;

  // fixed per-chunk gather state
  RowPix rpix[(GA == GA_FWD || GA == GA_DGRAD) ? PA : 1];
  ColTap ctap[GB == GB_WGRAD ? PB : 1];
  if constexpr (GA == GA_FWD || GA == GA_DGRAD) {
#pragma unroll
    for (int c = 0; c < PA; ++c) {
      const int e = min(tid + c * NT, CHA - 1);
      const int m = m0 + e / (KS / 8);
      rpix[c] = GA == GA_FWD ? row_pixel(p, m, p.Ho, p.Wo) : row_pixel(p, m, p.H, p.W);
    }
  }
  if constexpr (GB == GB_WGRAD) {
#pragma unroll
    for (int c = 0; c < PB; ++c) {
      const int e = min(tid + c * NT, CHB - 1);
      ctap[c] = col_tap(p, n0 + (e % (BN / 8)) * 8);
    }
  }
  // GA_FWDT / GA_DGRADT: per chunk (of the direct loop's layout), the byte
  // address of its source at tap (0, 0) (an integer: the pixel may lie
  // outside the image) and the mask of taps inside the image (zero for a
  // row past M)
  constexpr bool GAT = GA == GA_FWDT || GA == GA_DGRADT;
  static_assert(!GAT || DIRECT, "the tap-uniform gathers run in the direct loop");
  uint64_t tsrc[GAT ? PA : 1];
  uint32_t tmask[GAT ? PA : 1];
  if constexpr (GAT) {
    const int C = 1 << p.cshift;
#pragma unroll
    for (int c = 0; c < PA; ++c) {
      const int e = c * NT + tid, mr = e >> 3, kc = ((e & 7) ^ (mr & 7)) * 8;
      const RowPix rp = GA == GA_FWDT ? row_pixel(p, m0 + mr, p.Ho, p.Wo) : row_pixel(p, m0 + mr, p.H, p.W);
      // tap (0, 0)'s source pixel; tap (kh, kw) adds (kh, kw) (forward) or
      // subtracts it (data gradient)
      const int oy = GA == GA_FWDT ? rp.y * p.S - p.P : rp.y + p.P;
      const int ox = GA == GA_FWDT ? rp.x * p.S - p.P : rp.x + p.P;
      const int sh = GA == GA_FWDT ? p.H : p.Ho, sw = GA == GA_FWDT ? p.W : p.Wo;
      uint32_t mk = 0;
      for (int t = 0; t < p.R * p.R; ++t) {
        int kh, kw;
        tap_hw(t, p, kh, kw);
        const int y = GA == GA_FWDT ? oy + kh : oy - kh, x = GA == GA_FWDT ? ox + kw : ox - kw;
        mk |= uint32_t((y >= 0) & (y < sh) & (x >= 0) & (x < sw)) << t;
      }
      tmask[c] = rp.ok ? mk : 0u;
      const int64_t el = ((int64_t(rp.img) * sh + oy) * sw + ox) * C + kc;
      tsrc[c] = uint64_t(reinterpret_cast<uintptr_t>(A)) + uint64_t(el * 2);
    }
  }

  floatx4 acc[TM][TN];
#pragma unroll
  for (int a = 0; a < TM; ++a)
#pragma unroll
    for (int b = 0; b < TN; ++b) acc[a][b] = floatx4{0.f, 0.f, 0.f, 0.f};

  const int nk = kend > kbeg ? (kend - kbeg + KS - 1) / KS : 0;
  // k origin of slice s; a slice past the range re-reads the last one (real,
  // spread-out addresses; it is never multiplied)
  auto kslice = [&](int s) { return kbeg + max(0, min(s, nk - 1)) * KS; };
  unsigned char *scr;  // epilogue scratch (LDS)

  if constexpr (DIRECT) {
    // Stage layouts (16-byte chunks, chunk e of a slice at byte 16 e):
    //   k-contiguous operand: [row][8 chunks of 8 k], the chunk of logical
    //     k-group g stored in slot g ^ (row & 7);
    //   k-major operand: [k][rows / 8 chunks of 8 rows], the chunk of
    //     logical row-group g stored in slot g ^ (2 (k & 3) mod chunks per
    //     row).
    constexpr int SZA1 = BM * KS * 2, SZB1 = BN * KS * 2;
    // stages: more slices in flight hide more of the load latency, fewer
    // leave LDS for a second workgroup per compute unit
    constexpr int NS = STG ? STG : (direct_three_stages(BM, BN, EPI_SCR) ? 3 : 2);
    static_assert(NS >= 2 && NS <= 5, "two to five stages");
    static_assert((NS - 2) * (PA + PB) <= 63, "loads in flight fit the vector-memory counter");
    __shared__ __align__(1024) unsigned char sa0[SZA1], sa1[SZA1], sa2[NS > 2 ? SZA1 : 1],
        sa3[NS > 3 ? SZA1 : 1], sa4[NS > 4 ? SZA1 : 1];
    __shared__ __align__(1024) unsigned char sb0[SZB1], sb1[SZB1], sb2[NS > 2 ? SZB1 : 1],
        sb3[NS > 3 ? SZB1 : 1], sb4[NS > 4 ? SZB1 : 1];
    __shared__ __align__(16) unsigned char sepi[EPI_SCR <= SZA1 ? 1 : EPI_SCR];
    if constexpr (EPI_SCR <= SZA1) scr = sa0;
    else scr = sepi;
    // stage i's arrays (i a compile-time constant: each stage is its own
    // object, so the compiler knows which loads an LDS read waits for)
    auto stage_a = [&](auto I) -> unsigned char * {
      constexpr int i = decltype(I)::value;
      if constexpr (i == 0) return sa0;
      else if constexpr (i == 1) return sa1;
      else if constexpr (i == 2) return sa2;
      else if constexpr (i == 3) return sa3;
      else return sa4;
    };
    auto stage_b = [&](auto I) -> unsigned char * {
      constexpr int i = decltype(I)::value;
      if constexpr (i == 0) return sb0;
      else if constexpr (i == 1) return sb1;
      else if constexpr (i == 2) return sb2;
      else if constexpr (i == 3) return sb3;
      else return sb4;
    };
    // GB_WGRAD: the tap and channel of each chunk's (swizzled) column, fixed
    // for the whole k loop (the swizzle depends on the chunk's row in the
    // slice, not on the slice)
    ColTap ctapd[GB == GB_WGRAD ? PB : 1];
    if constexpr (GB == GB_WGRAD && !BK) {
#pragma unroll
      for (int c = 0; c < PB; ++c) {
        constexpr int RC = BN / 8;
        const int e = c * NT + tid, kr = e / RC;
        ctapd[c] = col_tap(p, n0 + ((e % RC) ^ ((2 * (kr & 3)) & (RC - 1))) * 8);
      }
    }

    // chunk c*NT + tid of slice s into the stage arrays la, lb
    auto issue = [&](int s, unsigned char *la, unsigned char *lb) {
      const int k0 = kslice(s);
      // tap-uniform gathers: the slice's tap, its bit in the masks and the
      // byte offset of its source from tap (0, 0)'s (workgroup-uniform)
      uint32_t tbit = 0;
      int64_t toff = 0;
      if constexpr (GAT) {
        const int tap = k0 >> p.cshift, ch0 = k0 & ((1 << p.cshift) - 1);
        int kh, kw;
        tap_hw(tap, p, kh, kw);
        tbit = 1u << tap;
        const int64_t px = GA == GA_FWDT ? int64_t(kh) * p.W + kw : -(int64_t(kh) * p.Wo + kw);
        toff = (px * (int64_t(1) << p.cshift) + ch0) * 2;
      }
#pragma unroll
      for (int c = 0; c < PA; ++c) {
        const int e = c * NT + tid;
        const void *src;
        if (AK) {
          const int mr = e >> 3, kc = ((e & 7) ^ (mr & 7)) * 8;
          if constexpr (GAT) {
            (void)mr, (void)kc;  // folded into tsrc
            src = src16(reinterpret_cast<const void *>(uintptr_t(tsrc[c] + uint64_t(toff))), (tmask[c] & tbit) != 0);
          } else if constexpr (GA == GA_CAT) {
            const int kk = k0 + kc, m = m0 + mr;
            const bool second = kk >= p.K1;
            const __bf16 *base = second ? p.A2 : reinterpret_cast<const __bf16 *>(A);
            const size_t off = size_t(m) * (second ? p.lda2 : p.lda) + (second ? kk - p.K1 : kk);
            src = src16(base + off, (m < p.M) & (kk < kend));
          } else if constexpr (GA != G_DENSE) {
            src = gatherA_src<GA>(p, reinterpret_cast<const __bf16 *>(A), rpix[c], k0 + kc, kend);
          } else {
            const int m = m0 + mr, kk = k0 + kc;
            src = src16(A + size_t(m) * p.lda + kk, (m < p.M) & (kk < kend));
          }
        } else {
          constexpr int RC = BM / 8;  // chunks per k row
          const int kr = e / RC, mc = ((e % RC) ^ ((2 * (kr & 3)) & (RC - 1))) * 8;
          const int kk = k0 + kr, m = m0 + mc;
          src = src16(A + size_t(kk) * p.lda + m, (kk < kend) & (m < p.M));
        }
        load_lds16(src, la + (c * NT + wave * 64) * 16);
      }
#pragma unroll
      for (int c = 0; c < PB; ++c) {
        const int e = c * NT + tid;
        const void *src;
        if (BK) {
          const int nr = e >> 3, kc = ((e & 7) ^ (nr & 7)) * 8;
          const int n = n0 + nr, kk = k0 + kc;
          src = src16(p.B + size_t(n) * p.ldb + kk, (n < p.N) & (kk < kend));
        } else {
          constexpr int RC = BN / 8;
          const int kr = e / RC, nc = ((e % RC) ^ ((2 * (kr & 3)) & (RC - 1))) * 8;
          const int kk = k0 + kr, n = n0 + nc;
          if constexpr (GB == GB_WGRAD) {
            src = gatherB_wgrad_src(p, ctapd[c], kk, kend);
          } else if constexpr (GB == GB_WDGRAD) {
            src = gatherB_wdgrad_src(p, kk, n, kend);
          } else {
            src = src16(p.B + size_t(kk) * p.ldb + n, (kk < kend) & (n < p.N));
          }
        }
        load_lds16(src, lb + (c * NT + wave * 64) * 16);
      }
    };
    // one k step of 32 from stage (sa, sb): the MFMA operands, swizzled back
    auto compute = [&](const unsigned char *sa, const unsigned char *sb) {
#pragma unroll
      for (int ks = 0; ks < KS; ks += 32) {
        bf16x8 av[TM], bv[TN];
#pragma unroll
        for (int a = 0; a < TM; ++a) {
          if constexpr (AK) {
            const int r = wm + a * 16 + i16, g = ((ks >> 3) + q) ^ (r & 7);
            av[a] = *reinterpret_cast<const bf16x8 *>(sa + (r * 8 + g) * 16);
          } else {
            constexpr int RC = BM / 8;
            const int kr = ks + 8 * q + (i16 >> 2), col = wm + a * 16 + 4 * (i16 & 3);
            const int g = (col >> 3) ^ ((2 * (kr & 3)) & (RC - 1));
            av[a] = tr_operand(sa + (kr * RC + g) * 16 + (col & 7) * 2, 4 * RC * 16);
          }
        }
#pragma unroll
        for (int b = 0; b < TN; ++b) {
          if constexpr (BK) {
            const int r = wn + b * 16 + i16, g = ((ks >> 3) + q) ^ (r & 7);
            bv[b] = *reinterpret_cast<const bf16x8 *>(sb + (r * 8 + g) * 16);
          } else {
            constexpr int RC = BN / 8;
            const int kr = ks + 8 * q + (i16 >> 2), col = wn + b * 16 + 4 * (i16 & 3);
            const int g = (col >> 3) ^ ((2 * (kr & 3)) & (RC - 1));
            bv[b] = tr_operand(sb + (kr * RC + g) * 16 + (col & 7) * 2, 4 * RC * 16);
          }
        }
#pragma unroll
        for (int a = 0; a < TM; ++a)
#pragma unroll
          for (int b = 0; b < TN; ++b)
            acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[a], bv[b], acc[a][b], 0, 0, 0);
      }
    };
    // Slice kt sits in stage kt % NS; NS - 1 slices are in flight ahead of
    // the one being multiplied.  At step kt each wavefront waits until only
    // the loads of the next NS - 2 slices are outstanding (its own share of
    // slice kt has landed) and its LDS reads of slice kt - 1 have returned
    // (the compiler may place the MFMAs that consume them, and so its own
    // wait for them, after the barrier), then the barrier makes every share
    // visible and tells that every wavefront is done with slice kt - 1, whose
    // stage then takes slice kt + NS - 1.  (A bare s_barrier: __syncthreads'
    // fence would wait for every load in flight.)
    unroll<NS - 1>([&](auto J) { issue(decltype(J)::value, stage_a(J), stage_b(J)); });
    auto step = [&](int kt, auto J) {
      constexpr int w = (decltype(J)::value + NS - 1) % NS;
      __builtin_amdgcn_s_waitcnt(vmcnt_le_lds0((NS - 2) * (PA + PB)));
      __builtin_amdgcn_s_barrier();
      issue(kt + NS - 1, stage_a(std::integral_constant<int, w>{}), stage_b(std::integral_constant<int, w>{}));
      compute(stage_a(J), stage_b(J));
    };
    int kt = 0;
    for (; kt + NS <= nk; kt += NS) unroll<NS>([&](auto J) { step(kt + decltype(J)::value, J); });
    unroll<NS - 1>([&](auto J) {
      if (kt + decltype(J)::value < nk) step(kt + decltype(J)::value, J);
    });
    // every load (the re-reads past the range included) has landed and every
    // wavefront is done with the stages before the epilogue reuses them
    __builtin_amdgcn_s_waitcnt(vmcnt_le(0));
    __syncthreads();
  } else {
    // register-staged loop: LDS operand tiles, double-buffered.  A
    // k-contiguous operand is stored [buf][row][k] (pitch KP); a k-major one
    // is stored as it arrives, [buf][k][row] (pitch rows + 16), and read back
    // through the transposing LDS read (two 8-byte reads give a lane its 8
    // consecutive k).
    constexpr int PA_K = BM + 16, PB_K = BN + 16;
    constexpr int SZA = AK ? 2 * BM * KP * 2 : 2 * KS * PA_K * 2;
    constexpr int SZB = BK ? 2 * BN * KP * 2 : 2 * KS * PB_K * 2;
    __shared__ __align__(16) unsigned char smA[SZA];
    __shared__ __align__(16) unsigned char smB[SZB];
    static_assert(EPI_SCR <= SZA, "epilogue scratch fits the A tile");
    scr = smA;
    // Every thread loads its chunks unconditionally (threads past a tile's
    // chunk count load a duplicate and skip the LDS store), so the load
    // counters are static and the loads stay in flight across the MFMAs.
    auto gload = [&](u32x4 (&ra)[PA], u32x4 (&rb)[PB], int k0) {
#pragma unroll
      for (int c = 0; c < PA; ++c) {
        const int e = min(tid + c * 256, CHA - 1);
        if (AK) {  // chunk = 8 k of one m
          const int mr = e / (KS / 8), kc = (e % (KS / 8)) * 8;
          if constexpr (GA == GA_CAT) {  // k < K1 from A, the rest from A2 (no branch)
            const int kk = k0 + kc, m = m0 + mr;
            const bool second = kk >= p.K1;
            const __bf16 *base = second ? p.A2 : reinterpret_cast<const __bf16 *>(A);
            const size_t off = size_t(m) * (second ? p.lda2 : p.lda) + (second ? kk - p.K1 : kk);
            ra[c] = masked16(base + off, (m < p.M) & (kk < kend));
          } else if constexpr (GA != G_DENSE)
            ra[c] = gatherA<GA>(p, reinterpret_cast<const __bf16 *>(A), rpix[c], k0 + kc, kend);
          else
            ra[c] = ld8<SAFE, TA>(A, m0 + mr, k0 + kc, p.M, kend, p.lda);
        } else {   // chunk = 8 m of one k
          const int kr = e / (BM / 8), mc = (e % (BM / 8)) * 8;
          ra[c] = ld8<SAFE, TA>(A, k0 + kr, m0 + mc, kend, p.M, p.lda);
        }
      }
#pragma unroll
      for (int c = 0; c < PB; ++c) {
        const int e = min(tid + c * 256, CHB - 1);
        if (BK) {
          const int nr = e / (KS / 8), kc = (e % (KS / 8)) * 8;
          rb[c] = ld8<SAFE, __bf16>(p.B, n0 + nr, k0 + kc, p.N, kend, p.ldb);
        } else {
          const int kr = e / (BN / 8), nc = (e % (BN / 8)) * 8;
          if constexpr (GB == GB_WGRAD)
            rb[c] = gatherB_wgrad(p, ctap[c], k0 + kr, kend);
          else if constexpr (GB == GB_WDGRAD)
            rb[c] = gatherB_wdgrad(p, k0 + kr, n0 + nc, kend);
          else
            rb[c] = ld8<SAFE, __bf16>(p.B, k0 + kr, n0 + nc, kend, p.N, p.ldb);
        }
      }
    };
    // k-contiguous chunks go to LDS as one 16-byte store; the others are
    // transposed into eight 2-byte stores.
    auto sstore = [&](const u32x4 (&ra)[PA], const u32x4 (&rb)[PB], int buf) {
#pragma unroll
      for (int c = 0; c < PA; ++c) {
        const int e = tid + c * 256;
        if (CHA % 256 == 0 || e < CHA) {
          if (AK) {
            const int mr = e / (KS / 8), kc = (e % (KS / 8)) * 8;
            *reinterpret_cast<u32x4 *>(smA + ((buf * BM + mr) * KP + kc) * 2) = ra[c];
          } else {
            const int kr = e / (BM / 8), mc = (e % (BM / 8)) * 8;
            *reinterpret_cast<u32x4 *>(smA + ((buf * KS + kr) * PA_K + mc) * 2) = ra[c];
          }
        }
      }
#pragma unroll
      for (int c = 0; c < PB; ++c) {
        const int e = tid + c * 256;
        if (CHB % 256 == 0 || e < CHB) {
          if (BK) {
            const int nr = e / (KS / 8), kc = (e % (KS / 8)) * 8;
            *reinterpret_cast<u32x4 *>(smB + ((buf * BN + nr) * KP + kc) * 2) = rb[c];
          } else {
            const int kr = e / (BN / 8), nc = (e % (BN / 8)) * 8;
            *reinterpret_cast<u32x4 *>(smB + ((buf * KS + kr) * PB_K + nc) * 2) = rb[c];
          }
        }
      }
    };

    // one slice: KS / 32 MFMA k-steps; step s reads k 32 s + 8 q .. + 7
    auto compute = [&](int buf) {
#pragma unroll
      for (int ks = 0; ks < KS; ks += 32) {
        bf16x8 av[TM], bv[TN];
#pragma unroll
        for (int a = 0; a < TM; ++a) {
          if constexpr (AK)
            av[a] = *reinterpret_cast<const bf16x8 *>(smA + ((buf * BM + wm + a * 16 + i16) * KP + ks + 8 * q) * 2);
          else
            av[a] = tr_operand(
                smA + ((buf * KS + ks + 8 * q + (i16 >> 2)) * PA_K + wm + a * 16 + 4 * (i16 & 3)) * 2,
                4 * PA_K * 2);
        }
#pragma unroll
        for (int b = 0; b < TN; ++b) {
          if constexpr (BK)
            bv[b] = *reinterpret_cast<const bf16x8 *>(smB + ((buf * BN + wn + b * 16 + i16) * KP + ks + 8 * q) * 2);
          else
            bv[b] = tr_operand(
                smB + ((buf * KS + ks + 8 * q + (i16 >> 2)) * PB_K + wn + b * 16 + 4 * (i16 & 3)) * 2,
                4 * PB_K * 2);
        }
#pragma unroll
        for (int a = 0; a < TM; ++a)
#pragma unroll
          for (int b = 0; b < TN; ++b)
            acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[a], bv[b], acc[a][b], 0, 0, 0);
      }
    };

    // Two register stages: the loads of slice kt + 2 are issued right after
    // slice kt is stored to LDS, so each load has two slices of MFMA work to
    // arrive.  Slice kt is stored to LDS buffer kt & 1.  The loop body has no
    // branches (a branch there makes the compiler wait for every outstanding
    // load at each iteration): it runs while two more slices follow, and the
    // last one or two slices are multiplied after it.
    u32x4 ra0[PA], rb0[PB], ra1[PA], rb1[PB];
    gload(ra0, rb0, kslice(0));
    gload(ra1, rb1, kslice(1));
    int kt = 0;
    for (; kt + 2 < nk; kt += 2) {  // no branches in the body (see above)
      sstore(ra0, rb0, 0);
      __syncthreads();
      gload(ra0, rb0, kslice(kt + 2));
      compute(0);
      sstore(ra1, rb1, 1);
      __syncthreads();
      gload(ra1, rb1, kslice(kt + 3));
      compute(1);
    }
    if (kt < nk) {  // the last one or two slices, without further loads
      sstore(ra0, rb0, 0);
      __syncthreads();
      compute(0);
      if (kt + 1 < nk) {
        sstore(ra1, rb1, 1);
        __syncthreads();
        compute(1);
      }
    }
  }

  // BF16STATS without a statistics buffer (a re-run that reuses its
  // statistics): the bf16 result alone (the same bits: the stored value is
  // rounded once either way)
  if (EPI == GEMM_EPI_BF16STATS && p.stats) {
    // per column: sums of the bf16-rounded values over this wavefront's rows,
    // then over the lane groups and the WM wavefronts sharing the column, in
    // a fixed order
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
          const float h = float((__bf16)acc[a][b][r]);
          acc[a][b][r] = h;
          if (m < p.M && n < p.N) {
            s1[b] += double(h);
            s2[b] += double(h) * double(h);
          }
        }
    __syncthreads();
    double *red = reinterpret_cast<double *>(scr);  // [WM*4][2][BN]
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
      if (n0 + col < p.N) p.stats[(size_t(tm) * 2 + which) * p.N + n0 + col] = t;
    }
  }

  // Epilogue through LDS: each wavefront stages 16 rows x WC columns of its
  // tile at a time, then writes whole rows with 16-byte stores (and reads D
  // and the mask the same way).
  float *stage = reinterpret_cast<float *>(scr) + wave * 16 * SP;
  float *Cz = p.C + size_t(tz) * p.M * p.ldc + size_t(bz) * p.bstrC;
  constexpr int VEC = EPI == GEMM_EPI_BF16STATS ? 8 : 4;  // output elements per lane
  constexpr int LPR = WC / VEC;                           // lanes per row
  constexpr int RPP = 64 / LPR;                           // rows per pass
  static_assert(WC % VEC == 0 && 64 % LPR == 0 && 16 % RPP == 0, "epilogue layout");
  const bool vec_ok = (p.ldc % VEC == 0) &&
                      (EPI == GEMM_EPI_STORE || EPI == GEMM_EPI_BF16STATS || EPI == GEMM_EPI_BNBWD ||
                       EPI == GEMM_EPI_ROWSOFTMAX || p.ldd % 4 == 0);
  // BNBWD: each lane owns the same VEC columns in every pass; per column the
  // batch norm's mean and 1/std, and float64 sums of ds and ds * xhat
  float bmean[EPI == GEMM_EPI_BNBWD ? VEC : 1], brstd[EPI == GEMM_EPI_BNBWD ? VEC : 1];
  double bs1[EPI == GEMM_EPI_BNBWD ? VEC : 1], bs2[EPI == GEMM_EPI_BNBWD ? VEC : 1];
  if constexpr (EPI == GEMM_EPI_BNBWD) {
#pragma unroll
    for (int u = 0; u < VEC; ++u) {
      const int n = n0 + wn + (lane % LPR) * VEC + u;
      bmean[u] = n < p.N ? p.bst[n] : 0.f;
      brstd[u] = n < p.N ? p.bst[p.N + n] : 0.f;
      bs1[u] = bs2[u] = 0.0;
    }
  }
  // BF16STATS with Rb: the batch-norm apply's parameters of the lane's VEC
  // columns, loaded once
  float amean[EPI == GEMM_EPI_BF16STATS ? VEC : 1], arstd[EPI == GEMM_EPI_BF16STATS ? VEC : 1];
  float agam[EPI == GEMM_EPI_BF16STATS ? VEC : 1], abet[EPI == GEMM_EPI_BF16STATS ? VEC : 1];
  if constexpr (EPI == GEMM_EPI_BF16STATS) {
#pragma unroll
    for (int u = 0; u < VEC; ++u) {
      const int n = n0 + wn + (lane % LPR) * VEC + u;
      const bool in = p.Rb && n < p.N;
      amean[u] = in ? p.ast[n] : 0.f;
      arstd[u] = in ? p.ast[p.N + n] : 0.f;
      agam[u] = in ? p.ag[n] : 0.f;
      abet[u] = in ? p.ab[n] : 0.f;
    }
  }
  // ROWSOFTMAX: the bias of the lane's VEC columns (-inf past N), loaded once
  float rbias[EPI == GEMM_EPI_ROWSOFTMAX ? VEC : 1];
  if constexpr (EPI == GEMM_EPI_ROWSOFTMAX) {
#pragma unroll
    for (int u = 0; u < VEC; ++u) {
      const int n = n0 + wn + (lane % LPR) * VEC + u;
      rbias[u] = n < p.N ? p.bias[n] : -INFINITY;
    }
  }
#pragma unroll
  for (int a = 0; a < TM; ++a) {
    __syncthreads();
#pragma unroll
    for (int b = 0; b < TN; ++b)
#pragma unroll
      for (int r = 0; r < 4; ++r) stage[(4 * q + r) * SP + b * 16 + i16] = acc[a][b][r];
    __syncthreads();
#pragma unroll
    for (int pass = 0; pass < 16 / RPP; ++pass) {
      const int rr = pass * RPP + lane / LPR, cc = (lane % LPR) * VEC;
      const int m = m0 + wm + a * 16 + rr, n = n0 + wn + cc;
      if constexpr (EPI == GEMM_EPI_ROWSOFTMAX) {
        // C = product + bias; the LPR lanes that share a row reduce by
        // butterflies (every lane takes part)
        const bool row_ok = m < p.M;
        float v[VEC], lm = -INFINITY;
#pragma unroll
        for (int u = 0; u < VEC; ++u) {
          v[u] = row_ok ? stage[rr * SP + cc + u] + rbias[u] : -INFINITY;
          lm = fmaxf(lm, v[u]);
        }
        // the row's maximum over the wavefront's columns first, then the sum
        // of exp(x - maximum), one hardware exp per element (relative error
        // about 1e-6 in the softmax denominator)
#pragma unroll
        for (int o = 1; o < LPR; o <<= 1) lm = fmaxf(lm, __shfl_xor(lm, o, 64));
        float ls = 0.f;
#pragma unroll
        for (int u = 0; u < VEC; ++u) ls += lm == -INFINITY ? 0.f : __expf(v[u] - lm);
#pragma unroll
        for (int o = 1; o < LPR; o <<= 1) ls += __shfl_xor(ls, o, 64);
        if (lane % LPR == 0) {
          rsm[((wave % WN) * BM + wm + a * 16 + rr) * 2 + 0] = lm;
          rsm[((wave % WN) * BM + wm + a * 16 + rr) * 2 + 1] = ls;
        }
        if (row_ok && n < p.N) {
          float *dst = Cz + size_t(m) * p.ldc + n;
          if (vec_ok && n + VEC <= p.N)
            *reinterpret_cast<float4 *>(dst) = make_float4(v[0], v[1], v[2], v[3]);
          else
            for (int u = 0; u < VEC && n + u < p.N; ++u) dst[u] = v[u];
        }
        continue;
      }
      if (m >= p.M || n >= p.N) continue;
      float v[VEC];
#pragma unroll
      for (int u = 0; u < VEC; ++u) v[u] = stage[rr * SP + cc + u];
      const bool full = vec_ok && n + VEC <= p.N;
      if constexpr (EPI == GEMM_EPI_BF16STATS) {
        const size_t o = size_t(m) * p.ldc + n;
        bf16x8 h;
#pragma unroll
        for (int u = 0; u < 8; ++u) h[u] = (__bf16)v[u];
        if (full) {
          *reinterpret_cast<bf16x8 *>(p.Cb + o) = h;
        } else {
          for (int u = 0; u < VEC && n + u < p.N; ++u) p.Cb[o + u] = h[u];
        }
        if (p.Rb) {  // the batch-norm apply (+ residual) and ReLU of the rounded values
          float x[VEC];
          if (p.Xr && full) {
            const bf16x8 xh = *reinterpret_cast<const bf16x8 *>(p.Xr + o);
#pragma unroll
            for (int u = 0; u < VEC; ++u) x[u] = float(xh[u]);
          } else {
#pragma unroll
            for (int u = 0; u < VEC; ++u) x[u] = p.Xr && n + u < p.N ? float(p.Xr[o + u]) : 0.f;
          }
          bf16x8 r;
#pragma unroll
          for (int u = 0; u < VEC; ++u) {
            float y = bnb_affine(float(h[u]), amean[u], arstd[u], agam[u], abet[u]);
            if (p.Xr) y += x[u];
            r[u] = (__bf16)fmaxf(y, 0.f);
          }
          if (full)
            *reinterpret_cast<bf16x8 *>(p.Rb + o) = r;
          else
            for (int u = 0; u < VEC && n + u < p.N; ++u) p.Rb[o + u] = r[u];
        }
      } else if constexpr (EPI == GEMM_EPI_BNBWD) {
        // ds = [Ym > 0] v, stored; xhat = (Cv - mean) / std
        const size_t o = size_t(m) * p.ldc + n;
        float y[VEC], cv[VEC];
        if (full) {
          const bf16x4 yh = *reinterpret_cast<const bf16x4 *>(p.Ym + o);
          const bf16x4 ch = *reinterpret_cast<const bf16x4 *>(p.Cv + o);
#pragma unroll
          for (int u = 0; u < VEC; ++u) {
            y[u] = float(yh[u]);
            cv[u] = float(ch[u]);
          }
        } else {
#pragma unroll
          for (int u = 0; u < VEC; ++u) {
            const bool in = n + u < p.N;
            y[u] = in ? float(p.Ym[o + u]) : 0.f;
            cv[u] = in ? float(p.Cv[o + u]) : 0.f;
          }
        }
#pragma unroll
        for (int u = 0; u < VEC; ++u) {
          v[u] = y[u] > 0.f ? v[u] : 0.f;
          const float xh = (cv[u] - bmean[u]) * brstd[u];
          bs1[u] += double(v[u]);
          bs2[u] += double(v[u]) * double(xh);
        }
        float *dst = Cz + o;
        if (full)
          *reinterpret_cast<float4 *>(dst) = make_float4(v[0], v[1], v[2], v[3]);
        else
          for (int u = 0; u < VEC && n + u < p.N; ++u) dst[u] = v[u];
      } else {
        if (EPI == GEMM_EPI_ADD || EPI == GEMM_EPI_ADDMASK) {
          const size_t o = size_t(m) * p.ldd + n;
          if (full) {
            const float4 d = *reinterpret_cast<const float4 *>(p.D + o);
            float dv[4] = {d.x, d.y, d.z, d.w};
            if (EPI == GEMM_EPI_ADDMASK) {
#pragma unroll
              for (int u = 0; u < 4; ++u) dv[u] = float(p.Ym[o + u]) > 0.f ? dv[u] : 0.f;
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) v[u] += dv[u];
          } else {
            for (int u = 0; u < VEC && n + u < p.N; ++u) {
              float d = p.D[o + u];
              if (EPI == GEMM_EPI_ADDMASK && !(float(p.Ym[o + u]) > 0.f)) d = 0.f;
              v[u] += d;
            }
          }
        } else if (p.bias) {
          for (int u = 0; u < VEC && n + u < p.N; ++u) v[u] += p.bias[n + u];
        }
        float *dst = Cz + size_t(m) * p.ldc + n;
        if (full)
          *reinterpret_cast<float4 *>(dst) = make_float4(v[0], v[1], v[2], v[3]);
        else
          for (int u = 0; u < VEC && n + u < p.N; ++u) dst[u] = v[u];
      }
    }
  }
  if constexpr (EPI == GEMM_EPI_ROWSOFTMAX) {
    // per row: the WN wavefront columns' pairs combined in order, stored as
    // rstat[row][column tile][2]
    __syncthreads();
    if (tid < BM && m0 + tid < p.M) {
      float lm = rsm[tid * 2], ls = rsm[tid * 2 + 1];
      for (int w = 1; w < WN; ++w) {
        const float om = rsm[(w * BM + tid) * 2], os = rsm[(w * BM + tid) * 2 + 1];
        const float mx = fmaxf(lm, om);
        ls = mx == -INFINITY ? 0.f : ls * expf(lm - mx) + os * expf(om - mx);
        lm = mx;
      }
      float *r = p.rstat + size_t(bz) * p.bstrR + (size_t(m0 + tid) * gridDim.x + tn) * 2;
      r[0] = lm;
      r[1] = ls;
    }
  }
  if constexpr (EPI == GEMM_EPI_BNBWD) {
    // per column: over the RPP lanes of a wavefront that share it, then over
    // the WM wavefronts, in a fixed order; block-major partials
    // [row tile][sum][column] as BF16STATS stores them
    __syncthreads();
    double *red = reinterpret_cast<double *>(scr);  // [WM * RPP][2][BN]
    const int slot = (wave / WN) * RPP + lane / LPR, col0 = wn + (lane % LPR) * VEC;
#pragma unroll
    for (int u = 0; u < VEC; ++u) {
      red[(slot * 2 + 0) * BN + col0 + u] = bs1[u];
      red[(slot * 2 + 1) * BN + col0 + u] = bs2[u];
    }
    __syncthreads();
    if (tid < 2 * BN) {
      const int which = tid / BN, col = tid % BN;
      double t = 0.0;
      for (int k = 0; k < WM * RPP; ++k) t += red[(k * 2 + which) * BN + col];
      if (n0 + col < p.N) p.stats[(size_t(tm) * 2 + which) * p.N + n0 + col] = t;
    }
  }
}

// Tiles by shape: large tiles while they still give at least half the compute
// units a workgroup (workgroups here are latency-bound, so fewer larger tiles
// win), and a tile width that follows N.
struct Tile {
  int BM, BN;
};

inline long tiles_for(int M, int N, int BM, int BN) {
  return long((M + BM - 1) / BM) * ((N + BN - 1) / BN);
}

inline Tile tile_of(int M, int N) {
  if (N <= 32) return {64, 32};
  if (N <= 64) {
    if (tiles_for(M, N, 256, 64) >= 256) return {256, 64};
    if (tiles_for(M, N, 128, 64) >= 128) return {128, 64};
    return {64, 64};
  }
  if (M >= 256 && tiles_for(M, N, 128, 128) >= 128) return {128, 128};
  if (tiles_for(M, N, 64, 64) >= 64) return {64, 64};
  return {64, 32};
}

template <int BM, int BN, int WM, int WN, bool AK, bool BK, typename TA, int GA, int GB, bool SAFE, int STG>
void launch_epi_s(const Args &a, int epi, int splits, hipStream_t s) {
  dim3 grid((a.N + BN - 1) / BN, (a.M + BM - 1) / BM, splits);
  if (epi == GEMM_EPI_ADD) {
    launch_timed((k_gemm_bf16<BM, BN, WM, WN, AK, BK, TA, GEMM_EPI_ADD, GA, GB, SAFE, STG>), grid, dim3(64 * WM * WN), 0, s, a);
    return;
  }
  if constexpr (std::is_same<TA, __bf16>::value) {
    if (epi == GEMM_EPI_ADDMASK) {
      launch_timed((k_gemm_bf16<BM, BN, WM, WN, AK, BK, TA, GEMM_EPI_ADDMASK, GA, GB, SAFE, STG>), grid, dim3(64 * WM * WN), 0, s, a);
      return;
    }
    if (epi == GEMM_EPI_BF16STATS) {
      launch_timed((k_gemm_bf16<BM, BN, WM, WN, AK, BK, TA, GEMM_EPI_BF16STATS, GA, GB, SAFE, STG>), grid, dim3(64 * WM * WN), 0, s, a);
      return;
    }
    // instantiated for the operand forms the host wrappers accept only
    if constexpr (AK && !BK && SAFE) {
      if (epi == GEMM_EPI_BNBWD) {
        launch_timed((k_gemm_bf16<BM, BN, WM, WN, AK, BK, TA, GEMM_EPI_BNBWD, GA, GB, SAFE, STG>), grid, dim3(64 * WM * WN), 0, s, a);
        return;
      }
    }
    if constexpr (AK && BK && SAFE && GA == G_DENSE && GB == G_DENSE) {
      if (epi == GEMM_EPI_ROWSOFTMAX) {
        launch_timed((k_gemm_bf16<BM, BN, WM, WN, AK, BK, TA, GEMM_EPI_ROWSOFTMAX, GA, GB, SAFE, STG>), grid, dim3(64 * WM * WN), 0, s, a);
        return;
      }
    }
  }
  launch_timed((k_gemm_bf16<BM, BN, WM, WN, AK, BK, TA, GEMM_EPI_STORE, GA, GB, SAFE, STG>), grid, dim3(64 * WM * WN), 0, s, a);
}

// The direct loop of the two largest tiles runs with three stages when the
// grid has no more tiles than the device has compute units (a second
// workgroup per unit would not exist anyway), else with two, so that two
// workgroups share a unit.
template <int BM, int BN, int WM, int WN, bool AK, bool BK, typename TA, int GA, int GB, bool SAFE>
void launch_epi(const Args &a, int epi, int splits, hipStream_t s) {
  constexpr bool direct = SAFE && std::is_same<TA, __bf16>::value;
  constexpr int scr = cmax(WM * WN * 16 * (BN / WN) * 4, 4 * 2 * BN * 8 * 4);  // a bound on any epilogue's scratch
  if constexpr (direct && !direct_three_stages(BM, BN, scr)) {
    const long tiles = long((a.N + BN - 1) / BN) * ((a.M + BM - 1) / BM) * splits;
    if (tiles <= 256) {
      launch_epi_s<BM, BN, WM, WN, AK, BK, TA, GA, GB, SAFE, 3>(a, epi, splits, s);
      return;
    }
  }
  launch_epi_s<BM, BN, WM, WN, AK, BK, TA, GA, GB, SAFE, 0>(a, epi, splits, s);
}

// Wavefronts per workgroup (the direct loop only; the tile, and so every
// result bit, is the same either way): with fewer workgroups than compute
// units, a latency-bound workgroup of four wavefronts issues from one
// wavefront per SIMD and one of eight from two, which pays once the k loop is
// long enough to outweigh the eight-wave epilogue's extra passes.  Measured
// per layer shape of the bottleneck ResNet and the LSTM on gfx950: eight
// wavefronts for every 256 x 64 tile, and, when the grid has fewer than 256
// workgroups, for 128 x 128 from 512 k per workgroup and for 64 x 64 from
// 2048.  The
// convolution weight gradients (few rows, a long k range per split) take 256-
// or 128-row tiles of eight wavefronts; their split partials have no
// row-block layout, so the tile may differ from tile_of's.
template <bool AK, bool BK, typename TA, int GA, int GB, bool SAFE>
void pick_tile(const Args &a, int epi, int splits, hipStream_t s) {
  const Tile t = tile_of(a.M, a.N);
  if constexpr (SAFE && std::is_same<TA, __bf16>::value) {
    if constexpr (GB == GB_WGRAD) {
      if (a.M >= 256) {
        launch_epi<256, 64, 4, 2, AK, BK, TA, GA, GB, SAFE>(a, epi, splits, s);
        return;
      }
      if (a.M >= 128) {
        launch_epi<128, 64, 4, 2, AK, BK, TA, GA, GB, SAFE>(a, epi, splits, s);
        return;
      }
    }
    if (t.BM == 256) {
      launch_epi<256, 64, 4, 2, AK, BK, TA, GA, GB, SAFE>(a, epi, splits, s);
      return;
    }
    const bool few = tiles_for(a.M, a.N, t.BM, t.BN) * splits < 256;
    if (t.BM == 128 && t.BN == 128 && few && a.kper >= 512) {
      launch_epi<128, 128, 4, 2, AK, BK, TA, GA, GB, SAFE>(a, epi, splits, s);
      return;
    }
    if (t.BM == 64 && t.BN == 64 && few && a.kper >= 2048) {
      launch_epi<64, 64, 4, 2, AK, BK, TA, GA, GB, SAFE>(a, epi, splits, s);
      return;
    }
  }
  if (t.BM == 256) launch_epi<256, 64, 4, 1, AK, BK, TA, GA, GB, SAFE>(a, epi, splits, s);
  else if (t.BM == 128 && t.BN == 128) launch_epi<128, 128, 2, 2, AK, BK, TA, GA, GB, SAFE>(a, epi, splits, s);
  else if (t.BM == 128) launch_epi<128, 64, 2, 2, AK, BK, TA, GA, GB, SAFE>(a, epi, splits, s);
  else if (t.BN == 64) launch_epi<64, 64, 2, 2, AK, BK, TA, GA, GB, SAFE>(a, epi, splits, s);
  else launch_epi<64, 32, 4, 1, AK, BK, TA, GA, GB, SAFE>(a, epi, splits, s);
}

// Every dense chunk is wholly inside or outside its operand when the
// contiguous extent and the leading dimension are multiples of 8.
inline bool safe8(const Args &a, bool ak, bool bk) {
  const int acols = ak ? a.K : a.M, bcols = bk ? a.K : a.N;
  return acols % 8 == 0 && a.lda % 8 == 0 && bcols % 8 == 0 && a.ldb % 8 == 0;
}

}  // namespace gb
}  // namespace ckpt
