// Elementwise and reduction kernels of the bf16 bottleneck network: batch
// norm apply (+ReLU, +identity or projected shortcut) and backward on bf16
// NHWC tensors, the 7x7/2 stem's im2col, and the 3x3/2 max pool.  Every
// thread moves 8 channels (16 bytes of bf16); channel counts are powers of
// two, at least 8.  Statistics and their gradient sums are float64 and
// reduced in a fixed order (bit-reproducible); all other arithmetic is fp32.
#include <hip/hip_runtime.h>

#include "bnb_act.h"
#include "common.h"
#include "kernels.h"

namespace ckpt {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ void load8(const __bf16 *p, float v[8]) {
  const bf16x8 h = *reinterpret_cast<const bf16x8 *>(p);
#pragma unroll
  for (int k = 0; k < 8; ++k) v[k] = float(h[k]);
}

__device__ __forceinline__ void store8(__bf16 *p, const float v[8]) {
  bf16x8 h;
#pragma unroll
  for (int k = 0; k < 8; ++k) h[k] = (__bf16)v[k];
  *reinterpret_cast<bf16x8 *>(p) = h;
}

__device__ __forceinline__ void load8f(const float *p, float v[8]) {
  const float4 a = *reinterpret_cast<const float4 *>(p);
  const float4 b = *reinterpret_cast<const float4 *>(p + 4);
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
  v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}

__device__ __forceinline__ void store8f(float *p, const float v[8]) {
  *reinterpret_cast<float4 *>(p) = make_float4(v[0], v[1], v[2], v[3]);
  *reinterpret_cast<float4 *>(p + 4) = make_float4(v[4], v[5], v[6], v[7]);
}

inline int ew_grid(int64_t work) {
  int64_t g = (work + 255) / 256;
  return int(g < 16384 ? (g < 1 ? 1 : g) : 16384);
}

// y = bf16(relu( gamma (c - mean) rstd + beta [+ x | + gp (cp - meanp) rstdp + bp] ))
template <int RES>
__global__ __launch_bounds__(256) void k_bnb_apply(int64_t P, int J, const __bf16 *__restrict__ Cv,
                                                   const float *__restrict__ st,
                                                   const float *__restrict__ gamma,
                                                   const float *__restrict__ beta,
                                                   const __bf16 *__restrict__ X,
                                                   const float *__restrict__ stp,
                                                   const float *__restrict__ gp,
                                                   const float *__restrict__ bp,
                                                   __bf16 *__restrict__ Y) {
  const int CQ = J / 8;
  const int64_t total = P * CQ;
  for (int64_t e = blockIdx.x * int64_t(256) + threadIdx.x; e < total; e += int64_t(gridDim.x) * 256) {
    const int c0 = int(e % CQ) * 8;
    const int64_t o = (e / CQ) * J + c0;
    float c[8], v[8];
    load8(Cv + o, c);
#pragma unroll
    for (int k = 0; k < 8; ++k) v[k] = bnb_affine(c[k], st[c0 + k], st[J + c0 + k], gamma[c0 + k], beta[c0 + k]);
    if (RES == BNB_RES_ID) {
      float x[8];
      load8(X + o, x);
#pragma unroll
      for (int k = 0; k < 8; ++k) v[k] += x[k];
    } else if (RES == BNB_RES_BN) {
      float x[8];
      load8(X + o, x);
#pragma unroll
      for (int k = 0; k < 8; ++k) v[k] += bnb_affine(x[k], stp[c0 + k], stp[J + c0 + k], gp[c0 + k], bp[c0 + k]);
    }
#pragma unroll
    for (int k = 0; k < 8; ++k) v[k] = fmaxf(v[k], 0.f);
    store8(Y + o, v);
  }
}

// partial sums for the backward: sum(ds), sum(ds * xhat), ds = [Ym > 0] G.
// Workgroup (x, y) = pixels [x PB, (x + 1) PB) of the channel slab
// [y SL, (y + 1) SL), SL = min(J, 256): SL / 8 threads per pixel (eight
// channels each), 256 / (SL / 8) pixel lanes; block-major partials
// part[x][2][J].
template <bool MASKED>
__global__ __launch_bounds__(256) void k_bnb_bwd_partials(int P, int J, int PB, const float *__restrict__ G,
                                                          const __bf16 *__restrict__ Ym,
                                                          const __bf16 *__restrict__ Cv,
                                                          const float *__restrict__ st,
                                                          double *__restrict__ part) {
  __shared__ double red[2][256][8];
  const int SL = J < 256 ? J : 256;
  const int CQ = SL / 8, PL = 256 / CQ;
  const int cq = threadIdx.x % CQ, pl = threadIdx.x / CQ;
  const int c0 = blockIdx.y * SL + cq * 8;
  const int p0 = blockIdx.x * PB, p1 = min(P, p0 + PB);
  float mean[8], rstd[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    mean[k] = st[c0 + k];
    rstd[k] = st[J + c0 + k];
  }
  double s1[8], s2[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) s1[k] = s2[k] = 0.0;
  if (pl < PL) {
    // pixels p0 + pl, + PL, + 2 PL, ... in turn; the loads of four of them are
    // issued before any is used (a pixel past the range reads p and is skipped)
    for (int p = p0 + pl; p < p1; p += 4 * PL) {
      float g[4][8], c[4][8], y[4][8];
      bool ok[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int pp = p + u * PL;
        ok[u] = pp < p1;
        const size_t o = size_t(ok[u] ? pp : p) * J + c0;
        load8f(G + o, g[u]);
        load8(Cv + o, c[u]);
        if (MASKED) load8(Ym + o, y[u]);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        if (!ok[u]) continue;
        if (MASKED) {
#pragma unroll
          for (int k = 0; k < 8; ++k) g[u][k] = y[u][k] > 0.f ? g[u][k] : 0.f;
        }
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          const float xh = (c[u][k] - mean[k]) * rstd[k];
          s1[k] += double(g[u][k]);
          s2[k] += double(g[u][k]) * double(xh);
        }
      }
    }
  }
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    red[0][threadIdx.x][k] = s1[k];
    red[1][threadIdx.x][k] = s2[k];
  }
  __syncthreads();
  for (int w = PL / 2; w > 0; w >>= 1) {
    if (pl < w) {
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        red[0][threadIdx.x][k] += red[0][threadIdx.x + w * CQ][k];
        red[1][threadIdx.x][k] += red[1][threadIdx.x + w * CQ][k];
      }
    }
    __syncthreads();
  }
  if (pl == 0) {
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      part[(size_t(blockIdx.x) * 2 + 0) * J + c0 + k] = red[0][threadIdx.x][k];
      part[(size_t(blockIdx.x) * 2 + 1) * J + c0 + k] = red[1][threadIdx.x][k];
    }
  }
}

// D = bf16( gamma rstd (ds - mean(ds) - xhat mean(ds xhat)) ),  ds = [Ym > 0] G
template <bool MASKED>
__global__ __launch_bounds__(256) void k_bnb_bwd_apply(int64_t P, int J, const float *__restrict__ G,
                                                       const __bf16 *__restrict__ Ym,
                                                       const __bf16 *__restrict__ Cv,
                                                       const float *__restrict__ st,
                                                       const float *__restrict__ gamma,
                                                       const float *__restrict__ sums,
                                                       __bf16 *__restrict__ D) {
  const int CQ = J / 8;
  const int64_t total = P * CQ;
  for (int64_t e = blockIdx.x * int64_t(256) + threadIdx.x; e < total; e += int64_t(gridDim.x) * 256) {
    const int c0 = int(e % CQ) * 8;
    const int64_t o = (e / CQ) * J + c0;
    float g[8], c[8], r[8];
    load8f(G + o, g);
    load8(Cv + o, c);
    if (MASKED) {
      float y[8];
      load8(Ym + o, y);
#pragma unroll
      for (int k = 0; k < 8; ++k) g[k] = y[k] > 0.f ? g[k] : 0.f;
    }
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int ch = c0 + k;
      const float rs = st[J + ch];
      const float xh = (c[k] - st[ch]) * rs;
      r[k] = gamma[ch] * rs * (g[k] - sums[ch] - xh * sums[J + ch]);
    }
    store8(D + o, r);
  }
}

// col[m][(kh*7 + kw)*3 + ci] = x[n, 2ho + kh - 3, 2wo + kw - 3, ci] (zero outside)
__global__ __launch_bounds__(256) void k_im2col7(int N, int H, int W, int Ho, int Wo,
                                                 const __bf16 *__restrict__ X,
                                                 __bf16 *__restrict__ col) {
  const int64_t total = int64_t(N) * Ho * Wo * 147;
  for (int64_t e = blockIdx.x * int64_t(256) + threadIdx.x; e < total; e += int64_t(gridDim.x) * 256) {
    const int k = int(e % 147);
    const int64_t m = e / 147;
    const int wo = int(m % Wo), ho = int((m / Wo) % Ho), n = int(m / (int64_t(Wo) * Ho));
    const int ci = k % 3, t = k / 3, kh = t / 7, kw = t % 7;
    const int hi = 2 * ho + kh - 3, wi = 2 * wo + kw - 3;
    __bf16 v = (__bf16)0.f;
    if (hi >= 0 && hi < H && wi >= 0 && wi < W) v = X[((int64_t(n) * H + hi) * W + wi) * 3 + ci];
    col[e] = v;
  }
}

// The same patches in rows of KP >= 147 elements (KP a multiple of 8), the
// columns past 147 zero: one 16-byte chunk of a row per thread.
__global__ __launch_bounds__(256) void k_im2col7p(int N, int H, int W, int Ho, int Wo, int KP,
                                                  const __bf16 *__restrict__ X, __bf16 *__restrict__ col) {
  const int CH = KP / 8;
  const int64_t total = int64_t(N) * Ho * Wo * CH;
  for (int64_t e = blockIdx.x * int64_t(256) + threadIdx.x; e < total; e += int64_t(gridDim.x) * 256) {
    const int j = int(e % CH);
    const int64_t m = e / CH;
    const int wo = int(m % Wo), ho = int((m / Wo) % Ho), n = int(m / (int64_t(Wo) * Ho));
    bf16x8 v;
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int k = j * 8 + u;
      const int ci = k % 3, t = k / 3, kh = t / 7, kw = t % 7;
      const int hi = 2 * ho + kh - 3, wi = 2 * wo + kw - 3;
      v[u] = (k < 147 && hi >= 0 && hi < H && wi >= 0 && wi < W) ? X[((int64_t(n) * H + hi) * W + wi) * 3 + ci]
                                                                : (__bf16)0.f;
    }
    *reinterpret_cast<bf16x8 *>(col + m * KP + j * 8) = v;
  }
}

// dst [R, KP] bf16 = src [R, C] fp32 rounded, the columns past C zero
__global__ __launch_bounds__(256) void k_cvt_pad_rows(int R, int C, int KP, const float *__restrict__ src,
                                                      __bf16 *__restrict__ dst) {
  const int e = blockIdx.x * 256 + threadIdx.x;
  if (e >= R * KP) return;
  const int r = e / KP, k = e % KP;
  dst[e] = k < C ? (__bf16)src[r * C + k] : (__bf16)0.f;
}

// 3x3 / stride 2 / pad 1 max pool; padding never wins
__global__ __launch_bounds__(256) void k_maxpool_fwd(int N, int H, int W, int C, int Ho, int Wo,
                                                     const __bf16 *__restrict__ R,
                                                     __bf16 *__restrict__ Y) {
  const int CQ = C / 8;
  const int64_t total = int64_t(N) * Ho * Wo * CQ;
  for (int64_t e = blockIdx.x * int64_t(256) + threadIdx.x; e < total; e += int64_t(gridDim.x) * 256) {
    const int c0 = int(e % CQ) * 8;
    const int64_t m = e / CQ;
    const int wo = int(m % Wo), ho = int((m / Wo) % Ho), n = int(m / (int64_t(Wo) * Ho));
    float best[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) best[k] = -INFINITY;
    for (int kh = 0; kh < 3; ++kh) {
      const int hi = 2 * ho + kh - 1;
      if (hi < 0 || hi >= H) continue;
      for (int kw = 0; kw < 3; ++kw) {
        const int wi = 2 * wo + kw - 1;
        if (wi < 0 || wi >= W) continue;
        float v[8];
        load8(R + ((int64_t(n) * H + hi) * W + wi) * C + c0, v);
#pragma unroll
        for (int k = 0; k < 8; ++k) best[k] = v[k] > best[k] ? v[k] : best[k];
      }
    }
    store8(Y + m * C + c0, best);
  }
}

// Two passes for the gradient: per window and channel, the tap of its first
// maximum (row-major order inside the window, taps outside the image
// skipped; the forward's output Y is the maximum), as a byte ...
__global__ __launch_bounds__(256) void k_maxpool_arg(int N, int H, int W, int C, int Ho, int Wo,
                                                     const __bf16 *__restrict__ R, const __bf16 *__restrict__ Y,
                                                     unsigned char *__restrict__ arg) {
  const int CQ = C / 8;
  const int64_t total = int64_t(N) * Ho * Wo * CQ;
  for (int64_t e = blockIdx.x * int64_t(256) + threadIdx.x; e < total; e += int64_t(gridDim.x) * 256) {
    const int c0 = int(e % CQ) * 8;
    const int64_t m = e / CQ;
    const int wo = int(m % Wo), ho = int((m / Wo) % Ho), n = int(m / (int64_t(Wo) * Ho));
    float ymax[8];
    load8(Y + m * C + c0, ymax);
    unsigned char a[8];
    bool found[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      a[k] = 9;
      found[k] = false;
    }
    for (int t = 0; t < 9; ++t) {
      const int hi = 2 * ho - 1 + t / 3, wi = 2 * wo - 1 + t % 3;
      if (hi < 0 || hi >= H || wi < 0 || wi >= W) continue;
      float v[8];
      load8(R + ((int64_t(n) * H + hi) * W + wi) * C + c0, v);
#pragma unroll
      for (int k = 0; k < 8; ++k)
        if (!found[k] && v[k] == ymax[k]) {
          found[k] = true;
          a[k] = (unsigned char)t;
        }
    }
    *reinterpret_cast<uint2 *>(arg + m * C + c0) =
        make_uint2(a[0] | a[1] << 8 | a[2] << 16 | uint32_t(a[3]) << 24, a[4] | a[5] << 8 | a[6] << 16 | uint32_t(a[7]) << 24);
  }
}

// ... then per input pixel the windows that hold it, in the order the
// one-pass kernel below visits them: dR[n, h, w, c] = sum of G over the
// windows whose first maximum is (h, w).
__global__ __launch_bounds__(256) void k_maxpool_bwd2(int N, int H, int W, int C, int Ho, int Wo,
                                                      const float *__restrict__ G,
                                                      const unsigned char *__restrict__ arg,
                                                      float *__restrict__ dR) {
  const int CQ = C / 8;
  const int64_t total = int64_t(N) * H * W * CQ;
  for (int64_t e = blockIdx.x * int64_t(256) + threadIdx.x; e < total; e += int64_t(gridDim.x) * 256) {
    const int c0 = int(e % CQ) * 8;
    const int64_t m = e / CQ;
    const int w = int(m % W), h = int((m / W) % H), n = int(m / (int64_t(W) * H));
    float acc[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) acc[k] = 0.f;
    const int ho_lo = h / 2, ho_hi = min(Ho - 1, (h + 1) / 2);
    const int wo_lo = w / 2, wo_hi = min(Wo - 1, (w + 1) / 2);
    for (int ho = ho_lo; ho <= ho_hi; ++ho)
      for (int wo = wo_lo; wo <= wo_hi; ++wo) {
        if (2 * ho - 1 > h || 2 * wo - 1 > w) continue;
        const int64_t oo = ((int64_t(n) * Ho + ho) * Wo + wo) * C + c0;
        const uint2 ab = *reinterpret_cast<const uint2 *>(arg + oo);
        float g[8];
        load8f(G + oo, g);
        const unsigned my = unsigned((h - (2 * ho - 1)) * 3 + (w - (2 * wo - 1)));
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          const unsigned a = ((k < 4 ? ab.x : ab.y) >> (8 * (k & 3))) & 0xFF;
          if (a == my) acc[k] += g[k];
        }
      }
    store8f(dR + m * C + c0, acc);
  }
}

// dR[n, h, w, c] = sum over the pooling windows whose first maximum (row-major
// order inside the window) is (h, w) of G at that window (one pass).
__global__ __launch_bounds__(256) void k_maxpool_bwd(int N, int H, int W, int C, int Ho, int Wo,
                                                     const float *__restrict__ G,
                                                     const __bf16 *__restrict__ R,
                                                     const __bf16 *__restrict__ Y,
                                                     float *__restrict__ dR) {
  const int CQ = C / 8;
  const int64_t total = int64_t(N) * H * W * CQ;
  for (int64_t e = blockIdx.x * int64_t(256) + threadIdx.x; e < total; e += int64_t(gridDim.x) * 256) {
    const int c0 = int(e % CQ) * 8;
    const int64_t m = e / CQ;
    const int w = int(m % W), h = int((m / W) % H), n = int(m / (int64_t(W) * H));
    float acc[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) acc[k] = 0.f;
    // windows ho with 2 ho - 1 <= h <= 2 ho + 1
    const int ho_lo = h / 2, ho_hi = min(Ho - 1, (h + 1) / 2);
    const int wo_lo = w / 2, wo_hi = min(Wo - 1, (w + 1) / 2);
    for (int ho = ho_lo; ho <= ho_hi; ++ho)
      for (int wo = wo_lo; wo <= wo_hi; ++wo) {
        if (2 * ho - 1 > h || 2 * wo - 1 > w) continue;
        float ymax[8], g[8];
        const int64_t oo = ((int64_t(n) * Ho + ho) * Wo + wo) * C + c0;
        load8(Y + oo, ymax);
        load8f(G + oo, g);
        const int my = (h - (2 * ho - 1)) * 3 + (w - (2 * wo - 1));  // this pixel's tap
        bool found[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) found[k] = false;
        // scan taps before and at `my` in row-major order: this pixel is the
        // argmax iff no earlier tap holds the maximum and it does
        for (int t = 0; t <= my; ++t) {
          const int hi = 2 * ho - 1 + t / 3, wi = 2 * wo - 1 + t % 3;
          if (hi < 0 || hi >= H || wi < 0 || wi >= W) continue;
          float v[8];
          load8(R + ((int64_t(n) * H + hi) * W + wi) * C + c0, v);
#pragma unroll
          for (int k = 0; k < 8; ++k) {
            if (!found[k] && v[k] == ymax[k]) {
              found[k] = true;
              if (t == my) acc[k] += g[k];
            }
          }
        }
      }
    store8f(dR + m * C + c0, acc);
  }
}

}  // namespace

// pixel blocks of the backward partial sums: about 512 workgroups over the
// channel slabs, each block a whole number of pixel-lane rounds
int bnb_partial_blocks(int64_t P, int J) {
  const int SL = J < 256 ? J : 256, slabs = J / SL, PL = 256 / (SL / 8);
  const int64_t nbp = (512 + slabs - 1) / slabs;
  int64_t pb = (P + nbp - 1) / nbp;
  pb = (pb + PL - 1) / PL * PL;
  if (pb < PL) pb = PL;
  return int((P + pb - 1) / pb);
}

void bnb_apply(hipStream_t s, int res, int64_t P, int J, const void *Cv, const float *st,
               const float *gamma, const float *beta, const void *X, const float *stp,
               const float *gp, const float *bp, void *Y) {
  const int g = ew_grid(P * (J / 8));
  const __bf16 *c = static_cast<const __bf16 *>(Cv), *x = static_cast<const __bf16 *>(X);
  __bf16 *y = static_cast<__bf16 *>(Y);
  if (res == BNB_RES_NONE)
    hipLaunchKernelGGL((k_bnb_apply<BNB_RES_NONE>), dim3(g), dim3(256), 0, s, P, J, c, st, gamma, beta, x, stp, gp, bp, y);
  else if (res == BNB_RES_ID)
    hipLaunchKernelGGL((k_bnb_apply<BNB_RES_ID>), dim3(g), dim3(256), 0, s, P, J, c, st, gamma, beta, x, stp, gp, bp, y);
  else
    hipLaunchKernelGGL((k_bnb_apply<BNB_RES_BN>), dim3(g), dim3(256), 0, s, P, J, c, st, gamma, beta, x, stp, gp, bp, y);
}

void bnb_backward_sums(hipStream_t s, int64_t P, int J, const float *G, const void *Ym, const void *Cv,
                       const float *st, double *part, float *sums, float *dgamma, float *dbeta) {
  const int nb = bnb_partial_blocks(P, J);
  const int pb = int((P + nb - 1) / nb);
  const __bf16 *ym = static_cast<const __bf16 *>(Ym), *c = static_cast<const __bf16 *>(Cv);
  const dim3 grid(nb, J < 256 ? 1 : J / 256);
  if (ym)
    hipLaunchKernelGGL((k_bnb_bwd_partials<true>), grid, dim3(256), 0, s, int(P), J, pb, G, ym, c, st, part);
  else
    hipLaunchKernelGGL((k_bnb_bwd_partials<false>), grid, dim3(256), 0, s, int(P), J, pb, G, ym, c, st, part);
  bn_finalize_bwd(s, part, nb, J, P, sums, dgamma, dbeta, false);
}

void bnb_backward(hipStream_t s, int64_t P, int J, const float *G, const void *Ym, const void *Cv,
                  const float *st, const float *gamma, double *part, float *sums, float *dgamma,
                  float *dbeta, void *D) {
  bnb_backward_sums(s, P, J, G, Ym, Cv, st, part, sums, dgamma, dbeta);
  bnb_backward_apply(s, P, J, G, Ym, Cv, st, gamma, sums, D);
}

void bnb_backward_apply(hipStream_t s, int64_t P, int J, const float *G, const void *Ym,
                        const void *Cv, const float *st, const float *gamma, const float *sums,
                        void *D) {
  const int g = ew_grid(P * (J / 8));
  const __bf16 *ym = static_cast<const __bf16 *>(Ym), *c = static_cast<const __bf16 *>(Cv);
  __bf16 *d = static_cast<__bf16 *>(D);
  if (ym)
    hipLaunchKernelGGL((k_bnb_bwd_apply<true>), dim3(g), dim3(256), 0, s, P, J, G, ym, c, st, gamma, sums, d);
  else
    hipLaunchKernelGGL((k_bnb_bwd_apply<false>), dim3(g), dim3(256), 0, s, P, J, G, ym, c, st, gamma, sums, d);
}

void im2col7(hipStream_t s, int N, int H, int W, int Ho, int Wo, int KP, const void *X, void *col) {
  if (KP == 147) {
    const int g = ew_grid(int64_t(N) * Ho * Wo * 147);
    hipLaunchKernelGGL(k_im2col7, dim3(g), dim3(256), 0, s, N, H, W, Ho, Wo, static_cast<const __bf16 *>(X),
                       static_cast<__bf16 *>(col));
    return;
  }
  if (KP < 147 || KP % 8) fail(CKPT_E_INVALID, "im2col7: rows of 147, or of a multiple of 8 above it");
  const int g = ew_grid(int64_t(N) * Ho * Wo * (KP / 8));
  hipLaunchKernelGGL(k_im2col7p, dim3(g), dim3(256), 0, s, N, H, W, Ho, Wo, KP, static_cast<const __bf16 *>(X),
                     static_cast<__bf16 *>(col));
}

void cvt_pad_rows(hipStream_t s, int R, int C, int KP, const float *src, void *dst) {
  hipLaunchKernelGGL(k_cvt_pad_rows, dim3((R * KP + 255) / 256), dim3(256), 0, s, R, C, KP, src,
                     static_cast<__bf16 *>(dst));
}

void maxpool_fwd(hipStream_t s, int N, int H, int W, int C, int Ho, int Wo, const void *R, void *Y) {
  const int g = ew_grid(int64_t(N) * Ho * Wo * (C / 8));
  hipLaunchKernelGGL(k_maxpool_fwd, dim3(g), dim3(256), 0, s, N, H, W, C, Ho, Wo,
                     static_cast<const __bf16 *>(R), static_cast<__bf16 *>(Y));
}

void maxpool_bwd(hipStream_t s, int N, int H, int W, int C, int Ho, int Wo, const float *G,
                 const void *R, const void *Y, float *dR, void *arg) {
  if (!arg) {
    const int g = ew_grid(int64_t(N) * H * W * (C / 8));
    hipLaunchKernelGGL(k_maxpool_bwd, dim3(g), dim3(256), 0, s, N, H, W, C, Ho, Wo, G,
                       static_cast<const __bf16 *>(R), static_cast<const __bf16 *>(Y), dR);
    return;
  }
  const int ga = ew_grid(int64_t(N) * Ho * Wo * (C / 8)), gb = ew_grid(int64_t(N) * H * W * (C / 8));
  hipLaunchKernelGGL(k_maxpool_arg, dim3(ga), dim3(256), 0, s, N, H, W, C, Ho, Wo, static_cast<const __bf16 *>(R),
                     static_cast<const __bf16 *>(Y), static_cast<unsigned char *>(arg));
  hipLaunchKernelGGL(k_maxpool_bwd2, dim3(gb), dim3(256), 0, s, N, H, W, C, Ho, Wo, G,
                     static_cast<const unsigned char *>(arg), dR);
}

}  // namespace ckpt
