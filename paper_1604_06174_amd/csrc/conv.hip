// 3x3 convolutions (pad 1) as implicit GEMMs on fp32 MFMA (v_mfma_f32_16x16x4f32),
// NHWC activations, weights [Cout, 3, 3, Cin].
//
// Forward / data-gradient kernel (k_conv3x3):
//   out[n, h, w, j] = sum_{tap, c} in(n, h, w, tap, c) * B(tap, c, j)
// One workgroup = R consecutive output rows of one image x BN output channels.
// The input rows it needs (a halo, zero outside the image) are staged once in
// LDS; the 3x3 taps are then read from LDS, so every input element is fetched
// from memory once per workgroup.  Weights for one tap are staged per tap with
// double buffering.
//   FWD:   in = x[n, h*S + kh - 1, w*S + kw - 1, c],  B = W[j, kh, kw, c]
//   DGRAD: the output gradient is up-sampled by the stride U (zeros between
//          samples) and correlated with the flipped kernel:
//          in = dy_up[n, h + 1 - kh, w + 1 - kw, c], B = W[c, kh, kw, j]
// Epilogues: STATS (store, plus per-workgroup float64 sums of v and v^2 per
// channel for batch-norm statistics, stored channel-major: all workgroups'
// sums of one channel are contiguous), MASK (store acc * [m > 0]), SC1 / SC2
// (add the shortcut's gradient g * [y > 0]: identity, or the option-A
// subsample-and-zero-pad shortcut of a stride-2 block).
//
// Weight-gradient kernel (k_conv3x3_wgrad): per workgroup (same row tiling as
// the forward) a partial dW[j, kh, kw, c] = sum over its pixels of
// dy[p, j] * x(p, tap, c); a second kernel sums the partials over workgroups
// in a fixed order.  No atomics anywhere: results are bit-reproducible.
#include <hip/hip_runtime.h>

#include "common.h"
#include "kernel_args.h"
#include "kernels.h"
#include "launch.h"

namespace ckpt {

typedef float floatx4 __attribute__((ext_vector_type(4)));

namespace {


// bn_relu of four consecutive channels c..c+3 (C = channel count of the
// statistics: st = mean[C] | rstd[C])
__device__ __forceinline__ float4 bn_relu4(float4 v, const float *st, const float *g, const float *b,
                                           int c, int C) {
  return make_float4(bn_relu(v.x, st[c], st[C + c], g[c], b[c]),
                     bn_relu(v.y, st[c + 1], st[C + c + 1], g[c + 1], b[c + 1]),
                     bn_relu(v.z, st[c + 2], st[C + c + 2], g[c + 2], b[c + 2]),
                     bn_relu(v.w, st[c + 3], st[C + c + 3], g[c + 3], b[c + 3]));
}

__device__ __forceinline__ int cpad4(int c) { return (c + 3) & ~3; }

template <int PSW, int NSUB, int MODE, int S, int EPI>
__global__ __launch_bounds__(256) void k_conv3x3(ConvArgs a) {
  constexpr int BN = 16 * NSUB;
  extern __shared__ __align__(16) float smem[];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int i16 = lane & 15, q = lane >> 4;
  const int blk = blockIdx.x;
  const int n = blk / a.rblk, r0 = (blk % a.rblk) * a.R;
  const int j0 = blockIdx.y * BN;
  const int Cp = cpad4(a.C), Cs = Cp + 4;
  const int HR = MODE == CONV_FWD ? (a.R - 1) * S + 3 : a.R + 2;
  const int HC = MODE == CONV_FWD ? (a.W - 1) * S + 3 : a.W + 2;
  float *halo = smem;
  float *Bs = smem + HR * HC * Cs;

  // ---- halo fill: halo[(hr*HC + hc)*Cs + c] ----
  {
    const int cq = Cp / 4;
    const int total = HR * HC * cq;
    for (int e = tid; e < total; e += 256) {
      const int c4 = (e % cq) * 4;
      const int hc = (e / cq) % HC;
      const int hr = e / (cq * HC);
      int ir, ic;
      bool ok;
      if (MODE == CONV_FWD) {
        ir = r0 * S - 1 + hr;
        ic = hc - 1;
        ok = ir >= 0 && ir < a.Hx && ic >= 0 && ic < a.Wx;
      } else {  // up-sampled output gradient
        const int ur = r0 - 1 + hr, uc = hc - 1;
        ok = ur >= 0 && uc >= 0 && (ur % S) == 0 && (uc % S) == 0;
        ir = ur / S;
        ic = uc / S;
        ok = ok && ir < a.Hx && ic < a.Wx;
      }
      float v[4] = {0.f, 0.f, 0.f, 0.f};
      if (ok) {
        const float *src = a.X + ((size_t(n) * a.Hx + ir) * a.Wx + ic) * a.C + c4;
        if ((a.C & 3) == 0) {
          float4 t = *reinterpret_cast<const float4 *>(src);
          v[0] = t.x; v[1] = t.y; v[2] = t.z; v[3] = t.w;
        } else {
#pragma unroll
          for (int k = 0; k < 4; ++k) v[k] = (c4 + k < a.C) ? src[k] : 0.f;
        }
        if (MODE == CONV_FWD && a.tst) {
#pragma unroll
          for (int k = 0; k < 4; ++k)
            if (c4 + k < a.C)
              v[k] = bn_relu(v[k], a.tst[c4 + k], a.tst[a.C + c4 + k], a.tg[c4 + k], a.tb[c4 + k]);
          // stride 1: halo rows 1..R are this workgroup's own output rows
          if (MODE == CONV_FWD && S == 1 && a.rout && blockIdx.y == 0 && hr >= 1 && hr <= a.R)
            *reinterpret_cast<float4 *>(a.rout + ((size_t(n) * a.Hx + ir) * a.Wx + ic) * a.C + c4) =
                make_float4(v[0], v[1], v[2], v[3]);
        }
      }
      *reinterpret_cast<float4 *>(halo + (hr * HC + hc) * Cs + c4) = make_float4(v[0], v[1], v[2], v[3]);
    }
  }

  // ---- weights of one tap: Bs[buf][c*BN + jj] ----
  auto wval = [&](int tap, int c, int jj) -> float {
    const int j = j0 + jj;
    if (c >= a.C || j >= a.J) return 0.f;
    if (MODE == CONV_FWD) return a.Wt[(size_t(j) * 9 + tap) * a.C + c];
    return a.Wt[(size_t(c) * 9 + tap) * a.J + j];
  };
  const int bel = Cp * BN;  // elements per tap
  constexpr int BREG = 8;   // supports Cp * BN <= 2048
  float breg[BREG];
  auto bload = [&](int tap) {
#pragma unroll
    for (int k = 0; k < BREG; ++k) {
      const int e = tid + k * 256;
      breg[k] = (e < bel) ? wval(tap, e / BN, e % BN) : 0.f;
    }
  };
  auto bstore = [&](int buf) {
#pragma unroll
    for (int k = 0; k < BREG; ++k) {
      const int e = tid + k * 256;
      if (e < bel) Bs[buf * bel + e] = breg[k];
    }
  };
  bload(0);
  bstore(0);
  __syncthreads();

  // ---- pixel of each A-fragment row this lane supplies ----
  const int npix = a.R * a.W;
  int pr[PSW], pc[PSW];
#pragma unroll
  for (int s = 0; s < PSW; ++s) {
    int p = (wave * PSW + s) * 16 + i16;
    if (p >= npix) p = npix - 1;  // clamped rows are computed but never stored
    pr[s] = p / a.W;
    pc[s] = p % a.W;
  }

  floatx4 acc[PSW][NSUB];
#pragma unroll
  for (int s = 0; s < PSW; ++s)
#pragma unroll
    for (int t = 0; t < NSUB; ++t) acc[s][t] = floatx4{0.f, 0.f, 0.f, 0.f};

  for (int tap = 0; tap < 9; ++tap) {
    const int kh = tap / 3, kw = tap % 3, buf = tap & 1;
    if (tap + 1 < 9) bload(tap + 1);
    int base[PSW];
#pragma unroll
    for (int s = 0; s < PSW; ++s) {
      const int hr = MODE == CONV_FWD ? pr[s] * S + kh : pr[s] + 2 - kh;
      const int hc = MODE == CONV_FWD ? pc[s] * S + kw : pc[s] + 2 - kw;
      base[s] = (hr * HC + hc) * Cs + q;
    }
    const float *Bt = Bs + buf * bel + q * BN + i16;
    for (int c = 0; c < Cp; c += 4) {
      float av[PSW], bv[NSUB];
#pragma unroll
      for (int s = 0; s < PSW; ++s) av[s] = halo[base[s] + c];
#pragma unroll
      for (int t = 0; t < NSUB; ++t) bv[t] = Bt[c * BN + t * 16];
#pragma unroll
      for (int s = 0; s < PSW; ++s)
#pragma unroll
        for (int t = 0; t < NSUB; ++t)
          acc[s][t] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[s], bv[t], acc[s][t], 0, 0, 0);
    }
    if (tap + 1 < 9) bstore(buf ^ 1);
    __syncthreads();
  }

  // ---- epilogue ----
  double s1[NSUB], s2[NSUB];
#pragma unroll
  for (int t = 0; t < NSUB; ++t) s1[t] = s2[t] = 0.0;
#pragma unroll
  for (int s = 0; s < PSW; ++s) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int p = (wave * PSW + s) * 16 + 4 * q + r;
      const int rr = p / a.W, cc = p % a.W;
      const int h = r0 + rr;
      const bool pv = p < npix && h < a.H;
#pragma unroll
      for (int t = 0; t < NSUB; ++t) {
        const int j = j0 + t * 16 + i16;
        if (!pv || j >= a.J) continue;
        const size_t o = ((size_t(n) * a.H + h) * a.W + cc) * a.J + j;
        float v = acc[s][t][r];
        if (EPI == CONV_EPI_STATS) {
          s1[t] += double(v);
          s2[t] += double(v) * double(v);
        } else if (EPI == CONV_EPI_MASK) {
          const float e = a.tst ? bn_relu(a.E0[o], a.tst[j], a.tst[a.J + j], a.tg[j], a.tb[j]) : a.E0[o];
          v = e > 0.f ? v : 0.f;
        } else if (EPI == CONV_EPI_MASKSTATS) {
          const float c = a.E0[o], mean = a.tst[j], rs = a.tst[a.J + j];
          v = bn_relu(c, mean, rs, a.tg[j], a.tb[j]) > 0.f ? v : 0.f;
          const float xh = (c - mean) * rs;
          s1[t] += double(v);
          s2[t] += double(v) * double(xh);
        } else if (EPI == CONV_EPI_SC1) {
          v += a.E1[o] > 0.f ? a.E0[o] : 0.f;
        } else if (EPI == CONV_EPI_SC2) {
          if (((h | cc) & 1) == 0) {
            const size_t o2 = ((size_t(n) * a.Eh + (h >> 1)) * a.Ew + (cc >> 1)) * a.Ec + j;
            v += a.E1[o2] > 0.f ? a.E0[o2] : 0.f;
          }
        }
        a.Y[o] = v;
      }
    }
  }
  if (EPI == CONV_EPI_STATS || EPI == CONV_EPI_MASKSTATS) {
    // per-channel sums over the workgroup: lanes (q) then waves, fixed order
    double *red = reinterpret_cast<double *>(smem);  // halo is no longer read
    __syncthreads();
#pragma unroll
    for (int t = 0; t < NSUB; ++t) {
      red[((wave * 4 + q) * 2 + 0) * BN + t * 16 + i16] = s1[t];
      red[((wave * 4 + q) * 2 + 1) * BN + t * 16 + i16] = s2[t];
    }
    __syncthreads();
    if (tid < 2 * BN) {
      const int which = tid / BN, jj = tid % BN;
      double acc2 = 0.0;
      for (int k = 0; k < 16; ++k) acc2 += red[(k * 2 + which) * BN + jj];
      if (j0 + jj < a.J) a.stats[(size_t(which) * a.J + j0 + jj) * gridDim.x + blk] = acc2;
    }
  }
}

// ------------------------------------------------ specialised fwd / dgrad --
// Same computation as k_conv3x3 for channel counts that are multiples of 16
// and compile-time shapes.  Each lane fetches a float4 of 4 consecutive
// channels of its pixel (ds_read_b128) and of its output channel's weights,
// and feeds them to 4 successive MFMA k-steps: step u pairs channel
// c0 + 4q + u of both operands, so the 4 steps cover channels c0..c0+15.
// Workgroup = RB output rows x BN output channels; each wavefront owns
// RB*W/64 pixel tiles of 16 and all BN/16 channel tiles.
template <int C, int J, int W, int S, int MODE, int RB, int BN>
constexpr size_t spec_lds();

template <int C, int J, int W, int S, int MODE, int EPI, int RB, int BN>
__global__ __launch_bounds__(256) void k_conv3x3s(ConvArgs a) {
  constexpr int NS = BN / 16;
  constexpr int NPIX = RB * W;
  static_assert(NPIX % 64 == 0 && C % 16 == 0 && BN % 16 == 0, "tile shape");
  constexpr int PSW = NPIX / 64;
  constexpr int Cs = C + 4;
  constexpr int C4 = C / 4;
  constexpr int HR = MODE == CONV_FWD ? (RB - 1) * S + 3 : RB + 2;
  constexpr int HC = MODE == CONV_FWD ? (W - 1) * S + 3 : W + 2;
  constexpr int WX = MODE == CONV_FWD ? W * S : W / S;  // input width
  __shared__ __align__(16) float smem[spec_lds<C, J, W, S, MODE, RB, BN>() / 4];
  float *halo = smem;
  float *Ws = smem + HR * HC * Cs;  // all nine taps: [9][BN][Cs]
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int i16 = lane & 15, q = lane >> 4;
  const int rblk = (a.H + RB - 1) / RB;
  const int n = blockIdx.x / rblk, r0 = (blockIdx.x % rblk) * RB;
  const int j0 = blockIdx.y * BN;
  const int Hx = a.Hx;

  // One load phase: the input halo and the weights of all nine taps are
  // fetched together (every load issued before any is used; an outside
  // address is replaced by the base and its value by zero), so the tap loop
  // below runs out of LDS with no further waits.  256 is a multiple of C4,
  // so a thread's halo chunks all hold channels 4 c4 .. 4 c4 + 3.
  {
    constexpr int HE = HR * HC * C4, NH = (HE + 255) / 256;
    static_assert(256 % C4 == 0, "channel chunk per thread");
    // weights: fwd Wt[j][tap][c] (float4 chunks of c), dgrad Wt[c][tap][j]
    constexpr int WE = MODE == CONV_FWD ? 9 * BN * C4 : 9 * BN * C, NW = (WE + 255) / 256;
    float4 hv[NH];
    bool hok[NH];
    float4 wq[MODE == CONV_FWD ? NW : 1];
    float wsr[MODE == CONV_FWD ? 1 : NW];
#pragma unroll
    for (int k = 0; k < NH; ++k) {
      const int e = tid + 256 * k;
      const int c4 = e % C4, hc = (e / C4) % HC, hr = e / (C4 * HC);
      int ir, ic;
      bool ok;
      if (MODE == CONV_FWD) {
        ir = r0 * S - 1 + hr;
        ic = hc - 1;
        ok = ir >= 0 && ir < Hx && ic >= 0 && ic < WX;
      } else {
        const int ur = r0 - 1 + hr, uc = hc - 1;
        ir = ur / S;
        ic = uc / S;
        ok = ur >= 0 && uc >= 0 && (ur % S) == 0 && (uc % S) == 0 && ir < Hx && ic < WX;
      }
      ok = ok && e < HE;
      const float4 v = *reinterpret_cast<const float4 *>(
          ok ? a.X + ((size_t(n) * Hx + ir) * WX + ic) * C + 4 * c4 : a.X);
      hv[k] = ok ? v : make_float4(0.f, 0.f, 0.f, 0.f);
      hok[k] = ok;
    }
#pragma unroll
    for (int k = 0; k < NW; ++k) {
      const int e = tid + 256 * k;
      if constexpr (MODE == CONV_FWD) {
        const int jj = e / (9 * C4), tap = (e / C4) % 9, c4 = e % C4, j = j0 + jj;
        const bool ok = e < WE && j < J;
        const float4 v = *reinterpret_cast<const float4 *>(
            ok ? a.Wt + (size_t(j) * 9 + tap) * C + 4 * c4 : a.Wt);
        wq[k] = ok ? v : make_float4(0.f, 0.f, 0.f, 0.f);
      } else {
        const int c = e / (9 * BN), tap = (e / BN) % 9, jj = e % BN, j = j0 + jj;
        const bool ok = e < WE && j < J;
        const float v = a.Wt[ok ? (size_t(c) * 9 + tap) * J + j : 0];
        wsr[k] = ok ? v : 0.f;
      }
    }
    if (MODE == CONV_FWD && a.tst) {  // relu(bn(.)) of the stored convolution output
      const int c = 4 * (tid % C4);
      float tm[4], tr[4], tg[4], tb[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        tm[u] = a.tst[c + u];
        tr[u] = a.tst[C + c + u];
        tg[u] = a.tg[c + u];
        tb[u] = a.tb[c + u];
      }
#pragma unroll
      for (int k = 0; k < NH; ++k)
        if (hok[k])
          hv[k] = make_float4(bn_relu(hv[k].x, tm[0], tr[0], tg[0], tb[0]),
                              bn_relu(hv[k].y, tm[1], tr[1], tg[1], tb[1]),
                              bn_relu(hv[k].z, tm[2], tr[2], tg[2], tb[2]),
                              bn_relu(hv[k].w, tm[3], tr[3], tg[3], tb[3]));
      // stride 1: halo rows 1..RB are this workgroup's own output rows; the
      // first channel block stores them (every element once over the grid)
      if (S == 1 && a.rout && blockIdx.y == 0) {
#pragma unroll
        for (int k = 0; k < NH; ++k) {
          const int e = tid + 256 * k;
          const int c4 = e % C4, hc = (e / C4) % HC, hr = e / (C4 * HC);
          const int ir = r0 - 1 + hr, ic = hc - 1;
          if (hok[k] && hr >= 1 && hr <= RB)
            *reinterpret_cast<float4 *>(a.rout + ((size_t(n) * Hx + ir) * WX + ic) * C + 4 * c4) = hv[k];
        }
      }
    }
#pragma unroll
    for (int k = 0; k < NH; ++k) {
      const int e = tid + 256 * k;
      if (e < HE) {
        const int c4 = e % C4, hc = (e / C4) % HC, hr = e / (C4 * HC);
        *reinterpret_cast<float4 *>(halo + (hr * HC + hc) * Cs + 4 * c4) = hv[k];
      }
    }
#pragma unroll
    for (int k = 0; k < NW; ++k) {
      const int e = tid + 256 * k;
      if (e < WE) {
        if constexpr (MODE == CONV_FWD) {
          const int jj = e / (9 * C4), tap = (e / C4) % 9, c4 = e % C4;
          *reinterpret_cast<float4 *>(Ws + (tap * BN + jj) * Cs + 4 * c4) = wq[k];
        } else {
          const int c = e / (9 * BN), tap = (e / BN) % 9, jj = e % BN;
          Ws[(tap * BN + jj) * Cs + c] = wsr[k];
        }
      }
    }
  }
  __syncthreads();

  int pr[PSW], pc[PSW];
#pragma unroll
  for (int s = 0; s < PSW; ++s) {
    const int p = (wave * PSW + s) * 16 + i16;
    pr[s] = p / W;
    pc[s] = p % W;
  }
  floatx4 acc[PSW][NS];
#pragma unroll
  for (int s = 0; s < PSW; ++s)
#pragma unroll
    for (int t = 0; t < NS; ++t) acc[s][t] = floatx4{0.f, 0.f, 0.f, 0.f};

  for (int tap = 0; tap < 9; ++tap) {
    const int kh = tap / 3, kw = tap % 3;
    int hoff[PSW];
#pragma unroll
    for (int s = 0; s < PSW; ++s)
      hoff[s] = MODE == CONV_FWD ? ((pr[s] * S + kh) * HC + pc[s] * S + kw) * Cs + 4 * q
                                 : ((pr[s] + 2 - kh) * HC + pc[s] + 2 - kw) * Cs + 4 * q;
    const float *Bt = Ws + (tap * BN + i16) * Cs + 4 * q;
#pragma unroll
    for (int c0 = 0; c0 < C; c0 += 16) {
      float4 av[PSW], bv[NS];
#pragma unroll
      for (int s = 0; s < PSW; ++s) av[s] = *reinterpret_cast<const float4 *>(halo + hoff[s] + c0);
#pragma unroll
      for (int t = 0; t < NS; ++t) bv[t] = *reinterpret_cast<const float4 *>(Bt + t * 16 * Cs + c0);
#pragma unroll
      for (int s = 0; s < PSW; ++s)
#pragma unroll
        for (int t = 0; t < NS; ++t) {
          acc[s][t] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[s].x, bv[t].x, acc[s][t], 0, 0, 0);
          acc[s][t] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[s].y, bv[t].y, acc[s][t], 0, 0, 0);
          acc[s][t] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[s].z, bv[t].z, acc[s][t], 0, 0, 0);
          acc[s][t] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[s].w, bv[t].w, acc[s][t], 0, 0, 0);
        }
    }
  }

  // epilogue operands (forward activations for the ReLU mask, the
  // shortcut's input and mask) fetched for all of the lane's outputs before
  // any is used; outside elements read the base and are never stored
  float e0[PSW][4][NS], e1[PSW][4][NS];
  if constexpr (EPI != CONV_EPI_STATS && EPI != CONV_EPI_STORE) {
#pragma unroll
    for (int s = 0; s < PSW; ++s)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int p = (wave * PSW + s) * 16 + 4 * q + r;
        const int rr = p / W, cc = p % W, h = r0 + rr;
#pragma unroll
        for (int t = 0; t < NS; ++t) {
          const int j = j0 + t * 16 + i16;
          bool ok = h < a.H && j < J;
          size_t o = ((size_t(n) * a.H + h) * W + cc) * J + j;
          if (EPI == CONV_EPI_SC2) {
            ok = ok && ((h | cc) & 1) == 0;
            o = ((size_t(n) * a.Eh + (h >> 1)) * a.Ew + (cc >> 1)) * a.Ec + j;
          }
          e0[s][r][t] = a.E0[ok ? o : 0];
          if (EPI != CONV_EPI_MASK && EPI != CONV_EPI_MASKSTATS) e1[s][r][t] = a.E1[ok ? o : 0];
        }
      }
  }
  float tm[NS], tr[NS], tg[NS], tb[NS];
  if ((EPI == CONV_EPI_MASK && a.tst) || EPI == CONV_EPI_MASKSTATS) {
#pragma unroll
    for (int t = 0; t < NS; ++t) {
      const int j = j0 + t * 16 + i16, jc = j < J ? j : 0;
      tm[t] = a.tst[jc];
      tr[t] = a.tst[a.J + jc];
      tg[t] = a.tg[jc];
      tb[t] = a.tb[jc];
    }
  }
  double s1[NS], s2[NS];
#pragma unroll
  for (int t = 0; t < NS; ++t) s1[t] = s2[t] = 0.0;
#pragma unroll
  for (int s = 0; s < PSW; ++s) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int p = (wave * PSW + s) * 16 + 4 * q + r;
      const int rr = p / W, cc = p % W;
      const int h = r0 + rr;
      if (h >= a.H) continue;
#pragma unroll
      for (int t = 0; t < NS; ++t) {
        const int j = j0 + t * 16 + i16;
        if (j >= J) continue;
        const size_t o = ((size_t(n) * a.H + h) * W + cc) * J + j;
        float v = acc[s][t][r];
        if (EPI == CONV_EPI_STATS) {
          s1[t] += double(v);
          s2[t] += double(v) * double(v);
        } else if (EPI == CONV_EPI_MASK) {
          const float e = a.tst ? bn_relu(e0[s][r][t], tm[t], tr[t], tg[t], tb[t]) : e0[s][r][t];
          v = e > 0.f ? v : 0.f;
        } else if (EPI == CONV_EPI_MASKSTATS) {
          v = bn_relu(e0[s][r][t], tm[t], tr[t], tg[t], tb[t]) > 0.f ? v : 0.f;
          const float xh = (e0[s][r][t] - tm[t]) * tr[t];
          s1[t] += double(v);
          s2[t] += double(v) * double(xh);
        } else if (EPI == CONV_EPI_SC1) {
          v += e1[s][r][t] > 0.f ? e0[s][r][t] : 0.f;
        } else if (EPI == CONV_EPI_SC2) {
          if (((h | cc) & 1) == 0) v += e1[s][r][t] > 0.f ? e0[s][r][t] : 0.f;
        }
        a.Y[o] = v;
      }
    }
  }
  if (EPI == CONV_EPI_STATS || EPI == CONV_EPI_MASKSTATS) {
    double *red = reinterpret_cast<double *>(smem);
    __syncthreads();
#pragma unroll
    for (int t = 0; t < NS; ++t) {
      red[((wave * 4 + q) * 2 + 0) * BN + t * 16 + i16] = s1[t];
      red[((wave * 4 + q) * 2 + 1) * BN + t * 16 + i16] = s2[t];
    }
    __syncthreads();
    if (tid < 2 * BN) {
      const int which = tid / BN, jj = tid % BN;
      double acc2 = 0.0;
      for (int k = 0; k < 16; ++k) acc2 += red[(k * 2 + which) * BN + jj];
      if (j0 + jj < J) a.stats[(size_t(which) * J + j0 + jj) * gridDim.x + blockIdx.x] = acc2;
    }
  }
}

template <int C, int J, int W, int S, int MODE, int RB, int BN>
constexpr size_t spec_lds() {
  constexpr int Cs = C + 4;
  constexpr int HR = MODE == CONV_FWD ? (RB - 1) * S + 3 : RB + 2;
  constexpr int HC = MODE == CONV_FWD ? (W - 1) * S + 3 : W + 2;
  constexpr size_t st = size_t(HR * HC * Cs + 9 * BN * Cs) * 4;
  constexpr size_t red = size_t(16) * 2 * BN * 8;
  return st > red ? st : red;
}

struct SpecUse {
  int RB = 0, BN = 0;
};

// One row of the specialisation table; returns whether it matches the launch.
template <int C, int J, int W, int S, int MODE, int EPI, int RB, int BN>
bool spec_try(const ConvArgs &a, int mode, int s, int epi, hipStream_t st, bool launch, SpecUse *u) {
  if (mode != MODE || s != S || epi != EPI || a.C != C || a.J != J || a.W != W) return false;
  if (a.Wx != (MODE == CONV_FWD ? W * S : W / S)) return false;
  static_assert(spec_lds<C, J, W, S, MODE, RB, BN>() <= 96 * 1024, "LDS");
  if (u) *u = {RB, BN};
  if (launch) {
    dim3 grid(a.N * ((a.H + RB - 1) / RB), (J + BN - 1) / BN);
    launch_timed((k_conv3x3s<C, J, W, S, MODE, EPI, RB, BN>), grid, dim3(256), 0, st, a);
  }
  return true;
}

// The CIFAR-shaped network's convolutions: 16/32/64 channels at 32/16/8 pixels.
bool spec_dispatch(const ConvArgs &a, int mode, int s, int epi, hipStream_t st, bool launch, SpecUse *u) {
  constexpr int F = CONV_FWD, D = CONV_DGRAD;
  constexpr int STATS = CONV_EPI_STATS, MASK = CONV_EPI_MASK, SC1 = CONV_EPI_SC1, SC2 = CONV_EPI_SC2,
                MST = CONV_EPI_MASKSTATS, STORE = CONV_EPI_STORE;
  // rows per workgroup and output channels per workgroup as measured best on
  // MI355X for these shapes (the forward without statistics: a re-run that
  // reuses them)
  return spec_try<16, 16, 32, 1, F, STATS, 4, 16>(a, mode, s, epi, st, launch, u) ||
         spec_try<16, 16, 32, 1, F, STORE, 4, 16>(a, mode, s, epi, st, launch, u) ||
         spec_try<16, 32, 16, 2, F, STORE, 4, 32>(a, mode, s, epi, st, launch, u) ||
         spec_try<32, 32, 16, 1, F, STORE, 8, 16>(a, mode, s, epi, st, launch, u) ||
         spec_try<32, 64, 8, 2, F, STORE, 8, 16>(a, mode, s, epi, st, launch, u) ||
         spec_try<64, 64, 8, 1, F, STORE, 8, 16>(a, mode, s, epi, st, launch, u) ||
         spec_try<16, 32, 16, 2, F, STATS, 4, 32>(a, mode, s, epi, st, launch, u) ||
         spec_try<32, 32, 16, 1, F, STATS, 8, 16>(a, mode, s, epi, st, launch, u) ||
         spec_try<32, 64, 8, 2, F, STATS, 8, 16>(a, mode, s, epi, st, launch, u) ||
         spec_try<64, 64, 8, 1, F, STATS, 8, 16>(a, mode, s, epi, st, launch, u) ||
         spec_try<16, 16, 32, 1, D, MASK, 4, 16>(a, mode, s, epi, st, launch, u) ||
         spec_try<32, 32, 16, 1, D, MASK, 4, 16>(a, mode, s, epi, st, launch, u) ||
         spec_try<64, 64, 8, 1, D, MASK, 8, 16>(a, mode, s, epi, st, launch, u) ||
         spec_try<16, 16, 32, 1, D, MST, 4, 16>(a, mode, s, epi, st, launch, u) ||
         spec_try<32, 32, 16, 1, D, MST, 4, 16>(a, mode, s, epi, st, launch, u) ||
         spec_try<64, 64, 8, 1, D, MST, 8, 16>(a, mode, s, epi, st, launch, u) ||
         spec_try<16, 16, 32, 1, D, SC1, 4, 16>(a, mode, s, epi, st, launch, u) ||
         spec_try<32, 32, 16, 1, D, SC1, 4, 16>(a, mode, s, epi, st, launch, u) ||
         spec_try<64, 64, 8, 1, D, SC1, 8, 16>(a, mode, s, epi, st, launch, u) ||
         spec_try<32, 16, 32, 2, D, SC2, 4, 16>(a, mode, s, epi, st, launch, u) ||
         spec_try<64, 32, 16, 2, D, SC2, 4, 16>(a, mode, s, epi, st, launch, u);
}

// ---------------------------------------------------------------- wgrad --
// dW[j][n] = sum_p dy[p][j] * col[p][n],  n = tap*C + c, col = im2col(x)
// (M = J, N = 9C, K = N*Ho*Wo pixels).  Workgroup = one 144-column slice of
// n (9 MFMA column tiles) x all J rows x a contiguous pixel range; its four
// wavefronts split the J row tiles (up to 4) and, when J < 64, the pixel
// range (reduced through LDS in a fixed order at the end).  Pixel chunks of 32
// are staged in double-buffered LDS: dy rows (float4 along j) and the gathered
// im2col rows (float4 along c).  Each workgroup writes one partial dW slice;
// k_sum_partials adds the partials of all pixel ranges in a fixed order.
constexpr int WG_KC = 32;    // pixels per LDS chunk
constexpr int WG_NB = 144;   // n columns per workgroup (9 tiles of 16)


__device__ __forceinline__ int wg_as(int J) { return J + ((16 - J % 32) + 32) % 32; }  // == 16 mod 32

// CT, JT, WT, HT, ST: compile-time channel counts, output width/height and
// stride (0 = take the runtime value): the network's few shapes get
// instantiations whose index arithmetic folds to shifts and multiplies.
template <int CT, int JT, int WT, int HT, int ST>
__global__ __launch_bounds__(256) void k_conv3x3_wgrad(WgArgs a) {
  extern __shared__ __align__(16) float smem[];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int i16 = lane & 15, q = lane >> 4;
  const int J = JT ? JT : a.J, C = CT ? CT : a.C, NC = 9 * C;
  const int OW = WT ? WT : a.W, OH = HT ? HT : a.H, SS = ST ? ST : a.S;
  const int jt_n = (J + 15) / 16;                  // j tiles (1..4)
  const int wgj = jt_n < 4 ? jt_n : 4;            // wavefronts across j tiles
  const int wgk = 4 / wgj;                         // wavefronts across pixels
  const int my_jt = wave % wgj, my_kg = wave / wgj;
  const int AS = wg_as(jt_n * 16);                // dy row stride in LDS
  constexpr int BS = WG_NB;                       // == 16 mod 32
  float *Abuf = smem;                              // [2][KC][AS]
  float *Bbuf = smem + 2 * WG_KC * AS;             // [2][KC][BS]
  const int n0 = blockIdx.y * WG_NB;
  const int P = a.N * OH * OW;
  const int p0 = blockIdx.x * a.pix_per_blk;
  const int nchunk = a.pix_per_blk / WG_KC;

  // staging: A = dy[p][0..16*jt_n) as float4, B = im2col[p][n0..n0+144) as float4
  const int a4 = jt_n * 4;          // float4 per dy row
  const int b4 = WG_NB / 4;         // 36 float4 per im2col row
  const int na = WG_KC * a4, nbq = WG_KC * b4;
  constexpr int MAXA = 2, MAXB = 5;  // per thread: na <= 512, nbq = 1152
  float4 ra[MAXA], rb[MAXB];
  auto gload = [&](int ck) {
    const int pc = p0 + ck * WG_KC;
#pragma unroll
    for (int k = 0; k < MAXA; ++k) {
      const int e = tid + k * 256;
      float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
      if (e < na) {
        const int pl = e / a4, j4 = (e % a4) * 4;
        const int p = pc + pl;
        if (p < P && j4 < J) v = *reinterpret_cast<const float4 *>(a.DY + size_t(p) * J + j4);
      }
      ra[k] = v;
    }
#pragma unroll
    for (int k = 0; k < MAXB; ++k) {
      const int e = tid + k * 256;
      float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
      if (e < nbq) {
        const int pl = e / b4, nn = n0 + (e % b4) * 4;
        const int p = pc + pl;
        if (p < P && nn < NC) {
          const int ow = p % OW;
          const int t = p / OW;
          const int oh = t % OH, img = t / OH;
          if ((C & 3) == 0) {  // the 4 columns are 4 channels of one tap
            const int tap = nn / C, c = nn % C;
            const int ih = oh * SS + tap / 3 - 1, iw = ow * SS + tap % 3 - 1;
            if (ih >= 0 && ih < a.Hx && iw >= 0 && iw < a.Wx) {
              v = *reinterpret_cast<const float4 *>(a.X + ((size_t(img) * a.Hx + ih) * a.Wx + iw) * C + c);
              if (a.tst) v = bn_relu4(v, a.tst, a.tg, a.tb, c, C);
            }
          } else {
            float vv[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
              const int n = nn + u;
              const int tap = n / C, c = n % C;
              const int ih = oh * SS + tap / 3 - 1, iw = ow * SS + tap % 3 - 1;
              const bool in = n < NC && ih >= 0 && ih < a.Hx && iw >= 0 && iw < a.Wx;
              vv[u] = in ? a.X[((size_t(img) * a.Hx + ih) * a.Wx + iw) * C + c] : 0.f;
              if (in && a.tst) vv[u] = bn_relu(vv[u], a.tst[c], a.tst[C + c], a.tg[c], a.tb[c]);
            }
            v = make_float4(vv[0], vv[1], vv[2], vv[3]);
          }
        }
      }
      rb[k] = v;
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int k = 0; k < MAXA; ++k) {
      const int e = tid + k * 256;
      if (e < na) {
        const int pl = e / a4, j4 = (e % a4) * 4;
        *reinterpret_cast<float4 *>(Abuf + (buf * WG_KC + pl) * AS + j4) = ra[k];
      }
    }
#pragma unroll
    for (int k = 0; k < MAXB; ++k) {
      const int e = tid + k * 256;
      if (e < nbq) {
        const int pl = e / b4, nc4 = (e % b4) * 4;
        *reinterpret_cast<float4 *>(Bbuf + (buf * WG_KC + pl) * BS + nc4) = rb[k];
      }
    }
  };

  floatx4 acc[9];
#pragma unroll
  for (int t = 0; t < 9; ++t) acc[t] = floatx4{0.f, 0.f, 0.f, 0.f};

  gload(0);
  const bool active = my_kg < wgk;  // with 3 j tiles one wavefront has no work
  for (int ck = 0; ck < nchunk; ++ck) {
    const int buf = ck & 1;
    sstore(buf);
    __syncthreads();
    if (ck + 1 < nchunk) gload(ck + 1);
    if (!active) continue;
    // this wavefront's pixels of the chunk: [my_kg * KC/wgk, (my_kg+1) * KC/wgk)
    const int kb = my_kg * (WG_KC / wgk), ke = kb + WG_KC / wgk;
    const float *Ab = Abuf + buf * WG_KC * AS + my_jt * 16 + i16;
    const float *Bb = Bbuf + buf * WG_KC * BS + i16;
    for (int k0 = kb; k0 < ke; k0 += 4) {
      const float av = Ab[(k0 + q) * AS];
#pragma unroll
      for (int t = 0; t < 9; ++t) {
        const float bv = Bb[(k0 + q) * BS + t * 16];
        acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(av, bv, acc[t], 0, 0, 0);
      }
    }
  }

  // reduce the pixel groups of the same j tile in a fixed order (group 0 + 1 + ...)
  if (wgk > 1) {
    __syncthreads();
    float *red = smem;  // [wave][9][4][64]
    if (my_kg > 0) {
#pragma unroll
      for (int t = 0; t < 9; ++t)
#pragma unroll
        for (int r = 0; r < 4; ++r) red[((wave * 9 + t) * 4 + r) * 64 + lane] = acc[t][r];
    }
    __syncthreads();
    if (my_kg == 0) {
      for (int g = 1; g < wgk; ++g) {
        const int w2 = g * wgj + my_jt;
#pragma unroll
        for (int t = 0; t < 9; ++t)
#pragma unroll
          for (int r = 0; r < 4; ++r) acc[t][r] += red[((w2 * 9 + t) * 4 + r) * 64 + lane];
      }
    }
  }
  if (my_kg == 0 && active) {
    float *dst = a.part + size_t(blockIdx.x) * J * NC;
#pragma unroll
    for (int t = 0; t < 9; ++t) {
      const int n = n0 + t * 16 + i16;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int j = my_jt * 16 + 4 * q + r;
        if (j < J && n < NC) dst[size_t(j) * NC + n] = acc[t][r];
      }
    }
  }
}

// ------------------------------------------- specialised weight gradient --
// Compile-time shapes.  Workgroup = TPB tiles of RB output rows of one image
// x one 144-column slice of n = tap*C + c (NT <= 9 tiles of 16).  The input
// halo of a tile (zero outside the image) and its dy rows are staged in LDS
// once; the im2col operand is read straight from the halo with per-lane tap
// offsets, so every input element is fetched from memory once per tile.
// Wavefronts split the J row tiles and, when J < 64, the tile's pixels
// (summed through LDS in a fixed order at the end).
template <int C, int J, int W, int S, int RB, int TPB>
__global__ __launch_bounds__(256) void k_wgrad_s(WgArgs a) {
  constexpr int NC = 9 * C;
  constexpr int Cp = (C + 3) & ~3;
  constexpr int Cs = Cp + 4;
  constexpr int HR = (RB - 1) * S + 3, HC = (W - 1) * S + 3;
  constexpr int NPIX = RB * W;
  constexpr int JT = (J + 15) / 16;
  constexpr int WGJ = JT < 4 ? JT : 4;
  constexpr int WGK = 4 / WGJ;
  static_assert(WGJ * WGK == 4 && NPIX % (4 * WGK) == 0, "wave split");
  constexpr int JS = JT * 16 + (((16 - (JT * 16) % 32) + 32) % 32);  // == 16 (mod 32)
  constexpr int NTT = (NC + 15) / 16;
  constexpr int WX = W * S;
  extern __shared__ __align__(16) float smem[];
  float *halo = smem;
  float *dys = smem + HR * HC * Cs;  // [NPIX][JS]
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int i16 = lane & 15, q = lane >> 4;
  const int my_jt = wave % WGJ, my_kg = wave / WGJ;
  const int n0 = blockIdx.y * 144;
  const int NT = min(9, NTT - blockIdx.y * 9);  // n tiles in this slice
  const int rblk = (a.H + RB - 1) / RB;
  const int ntiles = a.N * rblk;

  // per-lane im2col column offsets within the halo (tap shift + channel)
  int boff[9];
  bool bok[9];
#pragma unroll
  for (int t = 0; t < 9; ++t) {
    const int nn = n0 + t * 16 + i16;
    const int tap = nn / C, c = nn % C;
    bok[t] = t < NT && nn < NC;
    // a column outside the slice reads the halo's first element: its
    // accumulator is never stored
    boff[t] = bok[t] ? ((tap / 3) * HC + tap % 3) * Cs + c : 0;
  }
  floatx4 acc[9];
#pragma unroll
  for (int t = 0; t < 9; ++t) acc[t] = floatx4{0.f, 0.f, 0.f, 0.f};

  for (int tt = 0; tt < TPB; ++tt) {
    const int g = blockIdx.x * TPB + tt;
    if (g >= ntiles) break;
    const int img = g / rblk, r0 = (g % rblk) * RB;
    if (tt > 0) __syncthreads();
    for (int e = tid; e < HR * HC * (Cp / 4); e += 256) {
      const int c4 = (e % (Cp / 4)) * 4, hc = (e / (Cp / 4)) % HC, hr = e / ((Cp / 4) * HC);
      const int ir = r0 * S - 1 + hr, ic = hc - 1;
      float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
      if (ir >= 0 && ir < a.Hx && ic >= 0 && ic < WX) {
        const float *src = a.X + ((size_t(img) * a.Hx + ir) * WX + ic) * C + c4;
        if constexpr (C % 4 == 0) {
          v = *reinterpret_cast<const float4 *>(src);
          if (a.tst) v = bn_relu4(v, a.tst, a.tg, a.tb, c4, C);
        } else {
          float vv[4];
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            vv[u] = (c4 + u < C) ? src[u] : 0.f;
            if (c4 + u < C && a.tst) vv[u] = bn_relu(vv[u], a.tst[c4 + u], a.tst[C + c4 + u], a.tg[c4 + u], a.tb[c4 + u]);
          }
          v = make_float4(vv[0], vv[1], vv[2], vv[3]);
        }
      }
      *reinterpret_cast<float4 *>(halo + (hr * HC + hc) * Cs + c4) = v;
    }
    for (int e = tid; e < NPIX * (JT * 4); e += 256) {
      const int j4 = (e % (JT * 4)) * 4, p = e / (JT * 4);
      const int h = r0 + p / W, w = p % W;
      float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
      if (h < a.H && j4 < J) v = *reinterpret_cast<const float4 *>(a.DY + ((size_t(img) * a.H + h) * W + w) * J + j4);
      *reinterpret_cast<float4 *>(dys + p * JS + j4) = v;
    }
    __syncthreads();
    // k steps of 4 pixels: the ten LDS operands of step s + 1 are read before
    // the nine MFMAs of step s are issued (the scheduling barriers keep that
    // order), so LDS latency overlaps matrix-core work
    constexpr int PK = NPIX / WGK, NSTEP = PK / 4;
    const int kb = my_kg * PK;
    const float *Ab = dys + my_jt * 16 + i16;
    float av[2], bv[2][9];
    auto rd = [&](int st, float &a1, float (&b1)[9]) {
      const int p = kb + 4 * st + q;
      const int pb = ((p / W) * S * HC + (p % W) * S) * Cs;
      a1 = Ab[p * JS];
#pragma unroll
      for (int t = 0; t < 9; ++t) b1[t] = halo[pb + boff[t]];
    };
    rd(0, av[0], bv[0]);
#pragma unroll 2
    for (int st = 0; st < NSTEP; ++st) {
      const int cur = st & 1;
      if (st + 1 < NSTEP) rd(st + 1, av[cur ^ 1], bv[cur ^ 1]);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int t = 0; t < 9; ++t)
        acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[cur], bv[cur][t], acc[t], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
  }

  if constexpr (WGK > 1) {
    __syncthreads();
    float *red = smem;  // [wave][9][4][64]
    if (my_kg > 0) {
#pragma unroll
      for (int t = 0; t < 9; ++t)
#pragma unroll
        for (int r = 0; r < 4; ++r) red[((wave * 9 + t) * 4 + r) * 64 + lane] = acc[t][r];
    }
    __syncthreads();
    if (my_kg == 0) {
      for (int k = 1; k < WGK; ++k) {
        const int w2 = k * WGJ + my_jt;
#pragma unroll
        for (int t = 0; t < 9; ++t)
#pragma unroll
          for (int r = 0; r < 4; ++r) acc[t][r] += red[((w2 * 9 + t) * 4 + r) * 64 + lane];
      }
    }
  }
  if (my_kg == 0) {
    float *dst = a.part + size_t(blockIdx.x) * J * NC;
#pragma unroll
    for (int t = 0; t < 9; ++t) {
      const int nn = n0 + t * 16 + i16;
      if (!bok[t]) continue;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int j = my_jt * 16 + 4 * q + r;
        if (j < J) dst[size_t(j) * NC + nn] = acc[t][r];
      }
    }
  }
}

template <int C, int J, int W, int S, int RB>
constexpr size_t wgs_lds() {
  constexpr int Cs = ((C + 3) & ~3) + 4;
  constexpr int HR = (RB - 1) * S + 3, HC = (W - 1) * S + 3;
  constexpr int JT = (J + 15) / 16;
  constexpr int JS = JT * 16 + (((16 - (JT * 16) % 32) + 32) % 32);
  constexpr size_t st = size_t(HR * HC * Cs + RB * W * JS) * 4;
  constexpr size_t red = size_t(4) * 9 * 4 * 64 * 4;
  return st > red ? st : red;
}

struct WgUse {
  int nbx = 0;
};

template <int C, int J, int W, int S, int RB, int TPB>
bool wgs_try(const WgArgs &a, hipStream_t st, bool launch, WgUse *u) {
  if (a.C != C || a.J != J || a.W != W || a.S != S || a.Wx != W * S) return false;
  static_assert(wgs_lds<C, J, W, S, RB>() <= 64 * 1024, "LDS");
  const int ntiles = a.N * ((a.H + RB - 1) / RB);
  const int nbx = (ntiles + TPB - 1) / TPB;
  if (u) u->nbx = nbx;
  if (launch) {
    dim3 grid(nbx, (9 * C + 143) / 144);
    constexpr size_t lds = wgs_lds<C, J, W, S, RB>();
    hipLaunchKernelGGL((k_wgrad_s<C, J, W, S, RB, TPB>), grid, dim3(256), lds, st, a);
  }
  return true;
}

// rows per tile and tiles per workgroup as measured best on MI355X for the
// CIFAR-shaped network's shapes (batch 128, weight gradient + partial sums)
bool wgs_dispatch(const WgArgs &a, hipStream_t st, bool launch, WgUse *u) {
  return wgs_try<3, 16, 32, 1, 8, 1>(a, st, launch, u) ||
         wgs_try<16, 16, 32, 1, 4, 2>(a, st, launch, u) ||
         wgs_try<16, 32, 16, 2, 4, 2>(a, st, launch, u) ||
         wgs_try<32, 32, 16, 1, 4, 2>(a, st, launch, u) ||
         wgs_try<32, 64, 8, 2, 4, 2>(a, st, launch, u);
}

// out[e] = sum over b of part[b][e], b in a fixed order: SL slices of b
// (slice k takes b = k, k + SL, ...), then the slices in order.  A workgroup
// covers 256 / SL consecutive e; SL = 64 for small E, 16 otherwise.
// Workgroups are dispatched to the eight XCDs (each with its own L2) in
// turn; consecutive column groups are mapped to one XCD so that the cache
// lines they share are fetched from HBM once, not once per XCD.
__device__ __forceinline__ int xcd_grouped(int id, int G) {
  const int q = G / 8, r = G % 8, x = id % 8, k = id / 8;
  return x * q + (x < r ? x : r) + k;
}

template <int SL>
__global__ __launch_bounds__(256) void k_sum_partials(const float *__restrict__ part, int nb,
                                                      int E, float *__restrict__ out) {
  constexpr int ES = 256 / SL;
  __shared__ float red[SL][ES];
  const int ex = threadIdx.x % ES, sl = threadIdx.x / ES;
  const int e = xcd_grouped(blockIdx.x, gridDim.x) * ES + ex;
  float s = 0.f;
  if (e < E) {
    // b = sl, sl + SL, ... in order; sixteen loads in flight per round
    int b = sl;
    for (; b + 15 * SL < nb; b += 16 * SL) {
      float t[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) t[u] = part[size_t(b + u * SL) * E + e];
#pragma unroll
      for (int u = 0; u < 16; ++u) s += t[u];
    }
    for (; b < nb; b += SL) s += part[size_t(b) * E + e];
  }
  red[sl][ex] = s;
  __syncthreads();
  if (sl == 0 && e < E) {
    float t = 0.f;
    for (int k = 0; k < SL; ++k) t += red[k][ex];
    out[e] = t;
  }
}

// The same sum when nb is at most 16: k_sum_partials then gives each of the
// first nb thread slices one partial and adds the slices in order, i.e.
// ((0 + part[0][e]) + part[1][e]) + ..., which this kernel forms directly,
// four consecutive e per thread (one 16-byte load per partial).
__global__ __launch_bounds__(256) void k_sum_partials_seq(const float4 *__restrict__ part, int nb,
                                                          int E4, float4 *__restrict__ out) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= E4) return;
  float4 t = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll 4
  for (int b = 0; b < nb; ++b) {
    const float4 v = part[size_t(b) * E4 + i];
    t.x += v.x;
    t.y += v.y;
    t.z += v.z;
    t.w += v.w;
  }
  out[i] = t;
}

}  // namespace

void sum_partials(hipStream_t st, const float *part, int nb, int E, float *out) {
  if (nb <= 16 && E % 4 == 0 && (reinterpret_cast<uintptr_t>(part) & 15) == 0 &&
      (reinterpret_cast<uintptr_t>(out) & 15) == 0) {
    const int E4 = E / 4;
    hipLaunchKernelGGL(k_sum_partials_seq, dim3((E4 + 255) / 256), dim3(256), 0, st,
                       reinterpret_cast<const float4 *>(part), nb, E4, reinterpret_cast<float4 *>(out));
    return;
  }
  if (E < 16 * 2048)
    hipLaunchKernelGGL((k_sum_partials<64>), dim3((E + 3) / 4), dim3(256), 0, st, part, nb, E, out);
  else
    hipLaunchKernelGGL((k_sum_partials<16>), dim3((E + 15) / 16), dim3(256), 0, st, part, nb, E, out);
}

namespace {

struct Tile {
  int R, rblk, psw;
};

constexpr size_t kMaxLds = 64 * 1024;

size_t conv_lds(int mode, int S, int R, int W, int C, int J) {
  const int Cp = (C + 3) & ~3, Cs = Cp + 4;
  const int HR = mode == CONV_FWD ? (R - 1) * S + 3 : R + 2;
  const int HC = mode == CONV_FWD ? (W - 1) * S + 3 : W + 2;
  const int BN = J > 16 ? 32 : 16;
  size_t halo = size_t(HR) * HC * Cs * 4;
  size_t red = size_t(16) * 2 * BN * 8;
  return (halo > red ? halo : red) + size_t(2) * Cp * BN * 4;
}

// Whole output rows, at most 128 output pixels (8 MFMA row tiles) per
// workgroup, shrunk until the LDS footprint fits.
template <class Lds>
Tile tile_for(int H, int W, Lds lds) {
  int R = 128 / W;
  if (R < 1) R = 1;
  if (R > H) R = H;
  while (R > 1 && lds(R) > kMaxLds) --R;
  const int npix = R * W;
  const int psw = (npix + 63) / 64;  // 16-pixel tiles per wavefront
  return {R, (H + R - 1) / R, psw};
}

Tile conv_tile(int mode, int S, int H, int W, int C, int J) {
  return tile_for(H, W, [&](int R) { return conv_lds(mode, S, R, W, C, J); });
}

// Pixels per weight-gradient workgroup: enough workgroups (columns x pixel
// ranges) to give every compute unit about one, in whole LDS chunks.
int wgrad_pix(int64_t P, int NC) {
  const int ny = (NC + WG_NB - 1) / WG_NB;
  int64_t want = 256 / ny;
  if (want < 1) want = 1;
  int64_t ppb = (P + want - 1) / want;
  ppb = (ppb + WG_KC - 1) / WG_KC * WG_KC;
  return int(ppb);
}

size_t wgrad_lds(int J) {
  const int AS = (((J + 15) / 16) * 16) + ((16 - (((J + 15) / 16) * 16) % 32) + 32) % 32;
  const size_t stage = size_t(2) * WG_KC * (AS + WG_NB) * 4;
  const size_t red = size_t(4) * 9 * 4 * 64 * 4;
  return stage > red ? stage : red;
}

template <int PSW, int NSUB, int MODE, int S>
void launch_conv(const ConvArgs &a, int epi, size_t lds, dim3 grid, hipStream_t st) {
  switch (epi) {
    case CONV_EPI_STATS: launch_timed((k_conv3x3<PSW, NSUB, MODE, S, CONV_EPI_STATS>), grid, dim3(256), lds, st, a); break;
    case CONV_EPI_MASK: launch_timed((k_conv3x3<PSW, NSUB, MODE, S, CONV_EPI_MASK>), grid, dim3(256), lds, st, a); break;
    case CONV_EPI_MASKSTATS: launch_timed((k_conv3x3<PSW, NSUB, MODE, S, CONV_EPI_MASKSTATS>), grid, dim3(256), lds, st, a); break;
    case CONV_EPI_SC1: launch_timed((k_conv3x3<PSW, NSUB, MODE, S, CONV_EPI_SC1>), grid, dim3(256), lds, st, a); break;
    case CONV_EPI_SC2: launch_timed((k_conv3x3<PSW, NSUB, MODE, S, CONV_EPI_SC2>), grid, dim3(256), lds, st, a); break;
    default: launch_timed((k_conv3x3<PSW, NSUB, MODE, S, CONV_EPI_STORE>), grid, dim3(256), lds, st, a); break;
  }
}

template <int PSW, int NSUB>
void launch_mode(const ConvArgs &a, int mode, int S, int epi, size_t lds, dim3 grid, hipStream_t st) {
  if (mode == CONV_FWD) {
    if (S == 1) launch_conv<PSW, NSUB, CONV_FWD, 1>(a, epi, lds, grid, st);
    else launch_conv<PSW, NSUB, CONV_FWD, 2>(a, epi, lds, grid, st);
  } else {
    if (S == 1) launch_conv<PSW, NSUB, CONV_DGRAD, 1>(a, epi, lds, grid, st);
    else launch_conv<PSW, NSUB, CONV_DGRAD, 2>(a, epi, lds, grid, st);
  }
}

}  // namespace

static ConvArgs shape_args(int mode, int S, int N, int H, int W, int C, int J) {
  ConvArgs a{};
  a.N = N;
  a.H = H;
  a.W = W;
  a.C = C;
  a.J = J;
  a.Wx = mode == CONV_FWD ? W * S : W / S;
  return a;
}

int conv3x3_blocks(int mode, int S, int N, int H, int W, int C, int J) {
  SpecUse u;
  // the statistics partials are indexed by blockIdx.x only (STATS in the
  // forward, MASKSTATS in the data gradient)
  if (spec_dispatch(shape_args(mode, S, N, H, W, C, J), mode, S,
                    mode == CONV_FWD ? CONV_EPI_STATS : CONV_EPI_MASKSTATS, nullptr, false, &u))
    return N * ((H + u.RB - 1) / u.RB);
  return N * conv_tile(mode, S, H, W, C, J).rblk;
}

int conv3x3_wgrad_blocks(int S, int N, int H, int W, int C, int J) {
  WgArgs wa{};
  wa.N = N; wa.H = H; wa.W = W; wa.Wx = W * S; wa.C = C; wa.J = J; wa.S = S;
  WgUse u;
  if (wgs_dispatch(wa, nullptr, false, &u)) return u.nbx;
  const int64_t P = int64_t(N) * H * W;
  const int ppb = wgrad_pix(P, 9 * C);
  return int((P + ppb - 1) / ppb);
}

bool conv3x3_supported(int mode, int S, int H, int W, int C, int J) {
  const int BN = J > 16 ? 32 : 16;
  if (((C + 3) & ~3) * BN > 2048) return false;  // per-tap weight staging
  if (W > 128) return false;                      // <= 2 row tiles per wavefront
  if (conv_lds(mode, S, conv_tile(mode, S, H, W, C, J).R, W, C, J) > kMaxLds) return false;
  if (mode == CONV_FWD && (J > 64 || wgrad_lds(J) > kMaxLds)) return false;
  return true;
}

void conv3x3(hipStream_t st, int mode, int S, int epi, const float *X, const float *Wt, float *Y,
             int N, int H, int W, int Hx, int Wx, int C, int J, const float *E0, const float *E1,
             int Eh, int Ew, int Ec, double *stats, const float *tst, const float *tg,
             const float *tb, float *rout) {
  if (epi == CONV_EPI_MASKSTATS && (mode != CONV_DGRAD || !tst || !tg || !tb || !stats || !E0))
    fail(CKPT_E_INVALID, "conv3x3: MASKSTATS needs a data gradient, the mask operand, its statistics and stats");
  if (rout && (mode != CONV_FWD || S != 1 || !tst || (C & 3) != 0))
    fail(CKPT_E_INVALID, "conv3x3: the transformed input is stored only by a stride-1 forward with a transform");
  Tile t = conv_tile(mode, S, H, W, C, J);
  const int NSUB = J > 16 ? 2 : 1;
  ConvArgs a{X, Wt, Y, N, H, W, Hx, Wx, C, J, t.R, t.rblk, E0, E1, Eh, Ew, Ec, stats, tst, tg, tb, rout};
  if (spec_dispatch(a, mode, S, epi, st, true, nullptr)) return;
  dim3 grid(N * t.rblk, (J + 16 * NSUB - 1) / (16 * NSUB));
  const size_t lds = conv_lds(mode, S, t.R, W, C, J);
  if (t.psw == 1) {
    if (NSUB == 1) launch_mode<1, 1>(a, mode, S, epi, lds, grid, st);
    else launch_mode<1, 2>(a, mode, S, epi, lds, grid, st);
  } else {
    if (NSUB == 1) launch_mode<2, 1>(a, mode, S, epi, lds, grid, st);
    else launch_mode<2, 2>(a, mode, S, epi, lds, grid, st);
  }
}

void conv3x3_wgrad(hipStream_t st, int S, const float *X, const float *DY, float *part, float *dW,
                   int N, int H, int W, int Hx, int Wx, int C, int J, const float *tst,
                   const float *tg, const float *tb) {
  const int64_t P = int64_t(N) * H * W;
  const int NC = 9 * C;
  const int ppb = wgrad_pix(P, NC);
  const int nbx = int((P + ppb - 1) / ppb);
  WgArgs a{X, DY, part, N, H, W, Hx, Wx, C, J, S, ppb, tst, tg, tb};
  {
    WgUse u;
    if (wgs_dispatch(a, st, true, &u)) {
      sum_partials(st, part, u.nbx, J * NC, dW);
      return;
    }
  }
  dim3 grid(nbx, (NC + WG_NB - 1) / WG_NB);
  const size_t lds = wgrad_lds(J);
#define CKPT_WG(C_, J_, W_, S_)                                                              \
  if (C == C_ && J == J_ && W == W_ && H == W_ && S == S_) {                                 \
    hipLaunchKernelGGL((k_conv3x3_wgrad<C_, J_, W_, W_, S_>), grid, dim3(256), lds, st, a); \
  } else
  CKPT_WG(3, 16, 32, 1)
  CKPT_WG(16, 16, 32, 1)
  CKPT_WG(16, 32, 16, 2)
  CKPT_WG(32, 32, 16, 1)
  CKPT_WG(32, 64, 8, 2)
  CKPT_WG(64, 64, 8, 1)
  hipLaunchKernelGGL((k_conv3x3_wgrad<0, 0, 0, 0, 0>), grid, dim3(256), lds, st, a);
#undef CKPT_WG
  sum_partials(st, part, nbx, J * NC, dW);
}

}  // namespace ckpt
