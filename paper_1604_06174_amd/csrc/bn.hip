// Batch normalisation (training mode, per-channel statistics over N*H*W),
// its backward, and the global-average-pool + FC + softmax cross-entropy head.
// NHWC fp32 tensors; channel counts are multiples of 4 so every thread moves
// one float4 of channels.  Channel sums are accumulated in float64 and
// reduced in a fixed order (per-workgroup partials, then a fixed combine), so the
// results are bit-reproducible and insensitive to cancellation in
// E[x^2] - E[x]^2.
#include <hip/hip_runtime.h>

#include "kernels.h"

namespace ckpt {
namespace {

constexpr float BN_EPS = 1e-5f;

// ---- partial sums for the backward: sum(ds), sum(ds * xhat) per channel ----
template <bool MASKED>
__global__ __launch_bounds__(256) void k_bn_bwd_partials(int P, int J, int PB, const float *__restrict__ G,
                                                         const float *__restrict__ Ym,
                                                         const float *__restrict__ Cv,
                                                         const float *__restrict__ st,
                                                         double *__restrict__ part) {
  __shared__ double red[2][256][4];
  const int CQ = J / 4, PL = 256 / CQ;
  const int cq = threadIdx.x % CQ, pl = threadIdx.x / CQ;
  const int c0 = cq * 4;
  const int p0 = blockIdx.x * PB, p1 = min(P, p0 + PB);
  float mean[4], rstd[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    mean[k] = st[c0 + k];
    rstd[k] = st[J + c0 + k];
  }
  double s1[4] = {0, 0, 0, 0}, s2[4] = {0, 0, 0, 0};
  if (pl < PL) {
    // pixels p0 + pl, + PL, + 2 PL, ... in turn; the loads of four of them are
    // issued before any is used (a pixel past the range reads p and is skipped)
    for (int p = p0 + pl; p < p1; p += 4 * PL) {
      float4 g[4], c[4], y[4];
      bool ok[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int pp = p + u * PL;
        ok[u] = pp < p1;
        const size_t o = size_t(ok[u] ? pp : p) * J + c0;
        g[u] = *reinterpret_cast<const float4 *>(G + o);
        c[u] = *reinterpret_cast<const float4 *>(Cv + o);
        if (MASKED) y[u] = *reinterpret_cast<const float4 *>(Ym + o);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        if (!ok[u]) continue;
        float gv[4] = {g[u].x, g[u].y, g[u].z, g[u].w}, cv[4] = {c[u].x, c[u].y, c[u].z, c[u].w};
        if (MASKED) {
          const float yv[4] = {y[u].x, y[u].y, y[u].z, y[u].w};
#pragma unroll
          for (int k = 0; k < 4; ++k) gv[k] = yv[k] > 0.f ? gv[k] : 0.f;
        }
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const float xh = (cv[k] - mean[k]) * rstd[k];
          s1[k] += double(gv[k]);
          s2[k] += double(gv[k]) * double(xh);
        }
      }
    }
  }
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    red[0][threadIdx.x][k] = s1[k];
    red[1][threadIdx.x][k] = s2[k];
  }
  __syncthreads();
  // tree over pixel lanes (threads with the same cq are tid = cq + CQ*pl)
  for (int w = PL / 2; w > 0; w >>= 1) {
    if (pl < w) {
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        red[0][threadIdx.x][k] += red[0][threadIdx.x + w * CQ][k];
        red[1][threadIdx.x][k] += red[1][threadIdx.x + w * CQ][k];
      }
    }
    __syncthreads();
  }
  if (pl == 0) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      part[size_t(c0 + k) * gridDim.x + blockIdx.x] = red[0][threadIdx.x][k];
      part[(size_t(J) + c0 + k) * gridDim.x + blockIdx.x] = red[1][threadIdx.x][k];
    }
  }
}

// One workgroup per channel j; the per-workgroup partials k = 0..nb-1 of the
// two sums w = 0, 1 are stored either channel-major, part[(w * J + j) * nb + k]
// (a channel's partials contiguous: coalesced loads; for producers that write
// few channels per workgroup), or block-major, part[(k * 2 + w) * J + j] (each
// workgroup's sums contiguous: coalesced stores for producers that write many
// channels).  Fixed order either way: thread t adds k = t, t + 256, ... in
// turn, each wavefront combines its 64 lanes by a butterfly (the value lane 0
// ends with), and the four wavefront sums are added in wavefront order.
//   FWD: partials are (sum v, sum v^2) -> out0 = mean, out1 = rstd
//   BWD: partials are (sum ds, sum ds*xhat) -> out0 = mean(ds),
//        out1 = mean(ds*xhat); dgamma = sum ds*xhat, dbeta = sum ds
// channel j's statistics from its two sums over m values
template <bool FWD>
__device__ __forceinline__ void finalize_channel(int j, int J, double sa, double sb, double m,
                                                 float *__restrict__ out, float *__restrict__ dgamma,
                                                 float *__restrict__ dbeta) {
  if (FWD) {
    const double mean = sa / m;
    double var = sb / m - mean * mean;
    if (var < 0) var = 0;
    out[j] = float(mean);
    out[J + j] = float(1.0 / sqrt(var + double(BN_EPS)));
  } else {
    out[j] = float(sa / m);
    out[J + j] = float(sb / m);
    dbeta[j] = float(sa);
    dgamma[j] = float(sb);
  }
}

template <bool FWD, bool CM>
__global__ __launch_bounds__(256) void k_bn_finalize(const double *__restrict__ part, int nb, int J,
                                                     double m, float *__restrict__ out,
                                                     float *__restrict__ dgamma,
                                                     float *__restrict__ dbeta) {
  __shared__ double r0[4], r1[4];
  const int j = blockIdx.x;
  // element k of sum w at p_w[k * step]
  const double *p0 = CM ? part + size_t(j) * nb : part + j;
  const double *p1 = CM ? part + (size_t(J) + j) * nb : part + J + j;
  const size_t step = CM ? 1 : size_t(2) * J;
  double a = 0, b = 0;
  int k = threadIdx.x;
  for (; k + 3 * 256 < nb; k += 4 * 256) {  // four partials of each sum in flight
    double ta[4], tb[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      ta[u] = p0[(k + 256 * u) * step];
      tb[u] = p1[(k + 256 * u) * step];
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      a += ta[u];
      b += tb[u];
    }
  }
  for (; k < nb; k += 256) {
    a += p0[k * step];
    b += p1[k * step];
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    a += __shfl_xor(a, off);
    b += __shfl_xor(b, off);
  }
  const int wave = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    r0[wave] = a;
    r1[wave] = b;
  }
  __syncthreads();
  if (threadIdx.x == 0)
    finalize_channel<FWD>(j, J, ((r0[0] + r0[1]) + r0[2]) + r0[3], ((r1[0] + r1[1]) + r1[2]) + r1[3], m,
                          out, dgamma, dbeta);
}

// Block-major partials of many channels: a workgroup takes 16 consecutive
// channels (16 lanes read 128 contiguous bytes per partial) and splits the nb
// partials into 16 slices; slice s adds k = s, s + 16, ... in turn (eight
// loads in flight), and the 16 slice sums of a channel are added in slice
// order.
template <bool FWD>
__global__ __launch_bounds__(256) void k_bn_finalize_wide(const double *__restrict__ part, int nb, int J,
                                                          double m, float *__restrict__ out,
                                                          float *__restrict__ dgamma,
                                                          float *__restrict__ dbeta) {
  __shared__ double r0[16][17], r1[16][17];
  const int cl = threadIdx.x % 16, sl = threadIdx.x / 16;
  const int j = blockIdx.x * 16 + cl;
  double a = 0, b = 0;
  if (j < J) {
    int k = sl;
    for (; k + 7 * 16 < nb; k += 8 * 16) {
      double ta[8], tb[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        ta[u] = part[(size_t(k + 16 * u) * 2 + 0) * J + j];
        tb[u] = part[(size_t(k + 16 * u) * 2 + 1) * J + j];
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        a += ta[u];
        b += tb[u];
      }
    }
    for (; k < nb; k += 16) {
      a += part[(size_t(k) * 2 + 0) * J + j];
      b += part[(size_t(k) * 2 + 1) * J + j];
    }
  }
  r0[sl][cl] = a;
  r1[sl][cl] = b;
  __syncthreads();
  if (sl == 0 && j < J) {
    double sa = 0, sb = 0;
    for (int t = 0; t < 16; ++t) {
      sa += r0[t][cl];
      sb += r1[t][cl];
    }
    finalize_channel<FWD>(j, J, sa, sb, m, out, dgamma, dbeta);
  }
}

// y = [relu]( gamma (c - mean) rstd + beta [+ shortcut] )
template <int RES>
__global__ __launch_bounds__(256) void k_bn_apply(int64_t P, int J, const float *__restrict__ Cv,
                                                  const float *__restrict__ st,
                                                  const float *__restrict__ gamma,
                                                  const float *__restrict__ beta,
                                                  const float *__restrict__ X, int H, int W, int Cx,
                                                  float *__restrict__ Y) {
  const int CQ = J / 4;
  const int64_t total = P * CQ;
  for (int64_t e = blockIdx.x * int64_t(256) + threadIdx.x; e < total; e += int64_t(gridDim.x) * 256) {
    const int c0 = int(e % CQ) * 4;
    const int64_t p = e / CQ;
    const float4 c = *reinterpret_cast<const float4 *>(Cv + p * J + c0);
    float cv[4] = {c.x, c.y, c.z, c.w}, o[4];
#pragma unroll
    for (int k = 0; k < 4; ++k)
      o[k] = __builtin_fmaf(gamma[c0 + k], (cv[k] - st[c0 + k]) * st[J + c0 + k], beta[c0 + k]);
    if (RES == BN_RES_ID) {
      const float4 x = *reinterpret_cast<const float4 *>(X + p * J + c0);
      o[0] += x.x; o[1] += x.y; o[2] += x.z; o[3] += x.w;
    } else if (RES == BN_RES_A) {
      // option A: x[n, 2h, 2w, c] for c < Cx, zero for the appended channels
      const int64_t w = p % W, h = (p / W) % H, n = p / (int64_t(W) * H);
      const int64_t xo = ((n * 2 * H + 2 * h) * 2 * W + 2 * w) * Cx;
#pragma unroll
      for (int k = 0; k < 4; ++k)
        if (c0 + k < Cx) o[k] += X[xo + c0 + k];
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) o[k] = fmaxf(o[k], 0.f);
    *reinterpret_cast<float4 *>(Y + p * J + c0) = make_float4(o[0], o[1], o[2], o[3]);
  }
}

// dc = gamma rstd (ds - mean(ds) - xhat mean(ds xhat)),  ds = [mask] g
template <bool MASKED>
__global__ __launch_bounds__(256) void k_bn_bwd_apply(int64_t P, int J, const float *__restrict__ G,
                                                      const float *__restrict__ Ym,
                                                      const float *__restrict__ Cv,
                                                      const float *__restrict__ st,
                                                      const float *__restrict__ gamma,
                                                      const float *__restrict__ sums,
                                                      float *__restrict__ D) {
  const int CQ = J / 4;
  const int64_t total = P * CQ;
  for (int64_t e = blockIdx.x * int64_t(256) + threadIdx.x; e < total; e += int64_t(gridDim.x) * 256) {
    const int c0 = int(e % CQ) * 4;
    const int64_t o = (e / CQ) * J + c0;
    const float4 g = *reinterpret_cast<const float4 *>(G + o);
    const float4 c = *reinterpret_cast<const float4 *>(Cv + o);
    float gv[4] = {g.x, g.y, g.z, g.w}, cv[4] = {c.x, c.y, c.z, c.w}, r[4];
    if (MASKED) {
      const float4 y = *reinterpret_cast<const float4 *>(Ym + o);
      float yv[4] = {y.x, y.y, y.z, y.w};
#pragma unroll
      for (int k = 0; k < 4; ++k) gv[k] = yv[k] > 0.f ? gv[k] : 0.f;
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int ch = c0 + k;
      const float rs = st[J + ch];
      const float xh = (cv[k] - st[ch]) * rs;
      r[k] = gamma[ch] * rs * (gv[k] - sums[ch] - xh * sums[J + ch]);
    }
    *reinterpret_cast<float4 *>(D + o) = make_float4(r[0], r[1], r[2], r[3]);
  }
}

// ---- head: global average pool -> FC -> softmax cross-entropy ----
// One workgroup per sample; X is fp32 or bf16 NHWC.
template <typename TX>
__global__ __launch_bounds__(256) void k_head_sample(int N, int HW, int C, int K,
                                                     const TX *__restrict__ X,
                                                     const float *__restrict__ Wf,
                                                     const float *__restrict__ bf,
                                                     const int *__restrict__ labels,
                                                     float *__restrict__ pooled,
                                                     float *__restrict__ dlog,
                                                     float *__restrict__ lossn,
                                                     float *__restrict__ G) {
  extern __shared__ float sh[];
  float *pl = sh;           // [C]
  float *lg = sh + C;       // [K]
  float *red = sh + C + K;  // [256]
  const int n = blockIdx.x, t = threadIdx.x;
  const float inv = 1.0f / float(HW);
  for (int c = t; c < C; c += 256) {
    float s = 0.f;
    for (int p = 0; p < HW; ++p) s += float(X[(size_t(n) * HW + p) * C + c]);
    pl[c] = s * inv;
    pooled[size_t(n) * C + c] = s * inv;
  }
  __syncthreads();
  for (int k = t; k < K; k += 256) {
    float s = bf[k];
    for (int c = 0; c < C; ++c) s += pl[c] * Wf[size_t(c) * K + k];
    lg[k] = s;
  }
  __syncthreads();
  float mx = -INFINITY;
  for (int k = t; k < K; k += 256) mx = fmaxf(mx, lg[k]);
  red[t] = mx;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (t < w) red[t] = fmaxf(red[t], red[t + w]);
    __syncthreads();
  }
  mx = red[0];
  __syncthreads();
  float se = 0.f;
  for (int k = t; k < K; k += 256) se += expf(lg[k] - mx);
  red[t] = se;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (t < w) red[t] += red[t + w];
    __syncthreads();
  }
  se = red[0];
  // a label outside [0, K) yields a NaN loss for the sample and no one-hot term
  const int lab = labels[n];
  const bool lab_ok = lab >= 0 && lab < K;
  if (t == 0) lossn[n] = lab_ok ? (logf(se) + mx) - lg[lab] : NAN;
  __syncthreads();
  const float invN = 1.0f / float(N);
  for (int k = t; k < K; k += 256) {
    const float p = expf(lg[k] - mx) / se;
    const float d = (p - (k == lab ? 1.f : 0.f)) * invN;
    dlog[size_t(n) * K + k] = d;
    lg[k] = d;
  }
  __syncthreads();
  for (int c = t; c < C; c += 256) {
    float s = 0.f;
    for (int k = 0; k < K; ++k) s += lg[k] * Wf[size_t(c) * K + k];
    s *= inv;
    for (int p = 0; p < HW; ++p) G[(size_t(n) * HW + p) * C + c] = s;
  }
}

// The same head for a wide classifier (the bf16 net: C = 2048 features,
// K = 1000 classes) in six launches: pool, logits as an fp32 GEMM (bias
// epilogue), softmax, the pooled gradient as an fp32 GEMM, its broadcast over
// the pixels, the parameter gradients.
// pooled[n][c] = (sum over p of X[n][p][c]) / HW
__global__ __launch_bounds__(256) void k_head_pool_bf16(int N, int HW, int C, const __bf16 *__restrict__ X,
                                                        float *__restrict__ pooled) {
  const int e = blockIdx.x * 256 + threadIdx.x;
  if (e >= N * C) return;
  const int n = e / C, c = e % C;
  const float inv = 1.0f / float(HW);
  float s = 0.f;
#pragma unroll 8
  for (int p = 0; p < HW; ++p) s += float(X[(size_t(n) * HW + p) * C + c]);
  pooled[e] = s * inv;
}

// per sample: max, sum of exp, loss and dlog = (softmax - onehot) / N, in
// place over the logits (the row is read into LDS first)
__global__ __launch_bounds__(256) void k_head_softmax(int N, int K, const int *__restrict__ labels,
                                                      float *__restrict__ dlog, float *__restrict__ lossn) {
  extern __shared__ float sh[];
  float *lg = sh;       // [K]
  float *red = sh + K;  // [256]
  const int n = blockIdx.x, t = threadIdx.x;
  for (int k = t; k < K; k += 256) lg[k] = dlog[size_t(n) * K + k];
  __syncthreads();
  float mx = -INFINITY;
  for (int k = t; k < K; k += 256) mx = fmaxf(mx, lg[k]);
  red[t] = mx;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (t < w) red[t] = fmaxf(red[t], red[t + w]);
    __syncthreads();
  }
  mx = red[0];
  __syncthreads();
  float se = 0.f;
  for (int k = t; k < K; k += 256) se += expf(lg[k] - mx);
  red[t] = se;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (t < w) red[t] += red[t + w];
    __syncthreads();
  }
  se = red[0];
  const int lab = labels[n];
  const bool lab_ok = lab >= 0 && lab < K;
  if (t == 0) lossn[n] = lab_ok ? (logf(se) + mx) - lg[lab] : NAN;
  const float invN = 1.0f / float(N);
  for (int k = t; k < K; k += 256) {
    const float p = expf(lg[k] - mx) / se;
    dlog[size_t(n) * K + k] = (p - (k == lab ? 1.f : 0.f)) * invN;
  }
}

// G[n][p][c] = dpool[n][c] / HW at every pixel p
__global__ __launch_bounds__(256) void k_head_bcast(int N, int HW, int C, const float *__restrict__ dpool,
                                                    float *__restrict__ G) {
  const int64_t tot = int64_t(N) * HW * C;
  const float inv = 1.0f / float(HW);
  for (int64_t e = blockIdx.x * int64_t(256) + threadIdx.x; e < tot; e += int64_t(gridDim.x) * 256) {
    const int64_t n = e / (int64_t(HW) * C);
    G[e] = dpool[n * C + e % C] * inv;
  }
}

// dW[c][k] = sum_n pooled[n][c] dlog[n][k]; db[k] = sum_n dlog[n][k];
// loss = sum_n lossn[n] / N  (n in order)
__global__ __launch_bounds__(256) void k_head_params(int N, int C, int K,
                                                     const float *__restrict__ pooled,
                                                     const float *__restrict__ dlog,
                                                     const float *__restrict__ lossn,
                                                     float *__restrict__ dW, float *__restrict__ db,
                                                     float *__restrict__ loss) {
  const int e = blockIdx.x * 256 + threadIdx.x;
  if (e < C * K) {
    const int c = e / K, k = e % K;
    float s = 0.f;
    for (int n = 0; n < N; ++n) s += pooled[size_t(n) * C + c] * dlog[size_t(n) * K + k];
    dW[e] = s;
  } else if (e < C * K + K) {
    const int k = e - C * K;
    float s = 0.f;
    for (int n = 0; n < N; ++n) s += dlog[size_t(n) * K + k];
    db[k] = s;
  } else if (e == C * K + K) {
    float s = 0.f;
    for (int n = 0; n < N; ++n) s += lossn[n];
    loss[0] = s / float(N);
  }
}

inline int ew_grid(int64_t work) {
  int64_t g = (work + 255) / 256;
  return int(g < 8192 ? (g < 1 ? 1 : g) : 8192);
}

// ---- operators of the node-level graph (standalone forms of the fused ones) ----

// partial sums (sum x, sum x^2) per channel over this workgroup's pixels,
// float64, stored channel-major [2][J][nb] as the convolutions' STATS
// epilogue stores them; the same pixel split and lane tree as the backward
// partials
__global__ __launch_bounds__(256) void k_bn_stats_partials(int P, int J, int PB, const float *__restrict__ X,
                                                           double *__restrict__ part) {
  __shared__ double red[2][256][4];
  const int CQ = J / 4, PL = 256 / CQ;
  const int cq = threadIdx.x % CQ, pl = threadIdx.x / CQ;
  const int c0 = cq * 4;
  const int p0 = blockIdx.x * PB, p1 = min(P, p0 + PB);
  double s1[4] = {0, 0, 0, 0}, s2[4] = {0, 0, 0, 0};
  if (pl < PL) {
    for (int p = p0 + pl; p < p1; p += 4 * PL) {
      float4 x[4];
      bool ok[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int pp = p + u * PL;
        ok[u] = pp < p1;
        x[u] = *reinterpret_cast<const float4 *>(X + size_t(ok[u] ? pp : p) * J + c0);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        if (!ok[u]) continue;
        const float xv[4] = {x[u].x, x[u].y, x[u].z, x[u].w};
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          s1[k] += double(xv[k]);
          s2[k] += double(xv[k]) * double(xv[k]);
        }
      }
    }
  }
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    red[0][threadIdx.x][k] = s1[k];
    red[1][threadIdx.x][k] = s2[k];
  }
  __syncthreads();
  for (int w = PL / 2; w > 0; w >>= 1) {
    if (pl < w) {
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        red[0][threadIdx.x][k] += red[0][threadIdx.x + w * CQ][k];
        red[1][threadIdx.x][k] += red[1][threadIdx.x + w * CQ][k];
      }
    }
    __syncthreads();
  }
  if (pl == 0) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      part[size_t(c0 + k) * gridDim.x + blockIdx.x] = red[0][threadIdx.x][k];
      part[(size_t(J) + c0 + k) * gridDim.x + blockIdx.x] = red[1][threadIdx.x][k];
    }
  }
}

// y = gamma (x - mean) rstd + beta (no activation)
__global__ __launch_bounds__(256) void k_bn_norm(int64_t P, int J, const float *__restrict__ X,
                                                 const float *__restrict__ st,
                                                 const float *__restrict__ gamma,
                                                 const float *__restrict__ beta, float *__restrict__ Y) {
  const int CQ = J / 4;
  const int64_t total = P * CQ;
  for (int64_t e = blockIdx.x * int64_t(256) + threadIdx.x; e < total; e += int64_t(gridDim.x) * 256) {
    const int c0 = int(e % CQ) * 4;
    const int64_t o = (e / CQ) * J + c0;
    const float4 x = *reinterpret_cast<const float4 *>(X + o);
    const float xv[4] = {x.x, x.y, x.z, x.w};
    float r[4];
#pragma unroll
    for (int k = 0; k < 4; ++k)
      r[k] = __builtin_fmaf(gamma[c0 + k], (xv[k] - st[c0 + k]) * st[J + c0 + k], beta[c0 + k]);
    *reinterpret_cast<float4 *>(Y + o) = make_float4(r[0], r[1], r[2], r[3]);
  }
}

// option-A shortcut: Y[n, h, w, c] = X[n, 2h, 2w, c] for c < Cx, 0 for the
// appended channels (Y [N, H, W, J], X [N, 2H, 2W, Cx]); backward: DX[n, h,
// w, c] = DY[n, h/2, w/2, c] at even h and w, 0 elsewhere
__global__ __launch_bounds__(256) void k_shortcut_a(int64_t P, int H, int W, int J, int Cx,
                                                    const float *__restrict__ X, float *__restrict__ Y) {
  const int64_t total = P * J;
  for (int64_t e = blockIdx.x * int64_t(256) + threadIdx.x; e < total; e += int64_t(gridDim.x) * 256) {
    const int c = int(e % J);
    const int64_t p = e / J;
    const int64_t w = p % W, h = (p / W) % H, n = p / (int64_t(W) * H);
    Y[e] = c < Cx ? X[((n * 2 * H + 2 * h) * 2 * W + 2 * w) * Cx + c] : 0.f;
  }
}
__global__ __launch_bounds__(256) void k_shortcut_a_bwd(int64_t P, int H, int W, int J, int Cx,
                                                        const float *__restrict__ DY,
                                                        float *__restrict__ DX) {
  // P = N * 2H * 2W input pixels
  const int64_t total = P * Cx;
  for (int64_t e = blockIdx.x * int64_t(256) + threadIdx.x; e < total; e += int64_t(gridDim.x) * 256) {
    const int c = int(e % Cx);
    const int64_t p = e / Cx;
    const int64_t wi = p % (2 * W), hi = (p / (2 * W)) % (2 * H), n = p / (int64_t(4) * W * H);
    DX[e] = ((wi | hi) & 1) ? 0.f : DY[((n * H + hi / 2) * W + wi / 2) * J + c];
  }
}

// global average pool: Y[n, c] = (sum over p in order of X[n, p, c]) / HW;
// backward: DX[n, p, c] = DY[n, c] / HW
__global__ __launch_bounds__(256) void k_avgpool(int N, int HW, int C, const float *__restrict__ X,
                                                 float *__restrict__ Y) {
  const int e = blockIdx.x * 256 + threadIdx.x;
  if (e >= N * C) return;
  const int n = e / C, c = e % C;
  const float inv = 1.0f / float(HW);
  float s = 0.f;
  for (int p = 0; p < HW; ++p) s += X[(size_t(n) * HW + p) * C + c];
  Y[e] = s * inv;
}
__global__ __launch_bounds__(256) void k_avgpool_bwd(int64_t total, int HW, int C,
                                                     const float *__restrict__ DY, float *__restrict__ DX) {
  const float inv = 1.0f / float(HW);
  for (int64_t e = blockIdx.x * int64_t(256) + threadIdx.x; e < total; e += int64_t(gridDim.x) * 256) {
    const int c = int(e % C);
    const int64_t n = e / (int64_t(HW) * C);
    DX[e] = DY[n * C + c] * inv;
  }
}

// softmax cross-entropy of each row of logits [N, K] with its label: lossn[n]
// = log(sum exp(l - max)) + max - l[label], G = (softmax - onehot) / N; one
// workgroup per row (the same arithmetic as the fused head's)
__global__ __launch_bounds__(256) void k_softmax_ce_rows(int N, int K, const float *__restrict__ L,
                                                         const int *__restrict__ labels,
                                                         float *__restrict__ G, float *__restrict__ lossn) {
  __shared__ float red[256];
  const int n = blockIdx.x, t = threadIdx.x;
  const float *lg = L + size_t(n) * K;
  float mx = -INFINITY;
  for (int k = t; k < K; k += 256) mx = fmaxf(mx, lg[k]);
  red[t] = mx;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (t < w) red[t] = fmaxf(red[t], red[t + w]);
    __syncthreads();
  }
  mx = red[0];
  __syncthreads();
  float se = 0.f;
  for (int k = t; k < K; k += 256) se += expf(lg[k] - mx);
  red[t] = se;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (t < w) red[t] += red[t + w];
    __syncthreads();
  }
  se = red[0];
  const int lab = labels[n];
  const bool lab_ok = lab >= 0 && lab < K;
  if (t == 0) lossn[n] = lab_ok ? (logf(se) + mx) - lg[lab] : NAN;
  const float invN = 1.0f / float(N);
  for (int k = t; k < K; k += 256) {
    const float p = expf(lg[k] - mx) / se;
    G[size_t(n) * K + k] = (p - (k == lab ? 1.f : 0.f)) * invN;
  }
}

// loss = (sum over n in order of lossn[n]) / N
__global__ void k_loss_mean(int N, const float *__restrict__ lossn, float *__restrict__ loss) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  float s = 0.f;
  for (int n = 0; n < N; ++n) s += lossn[n];
  loss[0] = s / float(N);
}

}  // namespace

int bn_partial_blocks(int64_t P, int J) {
  const int PL = 256 / (J / 4);
  int64_t pb = (P + 511) / 512;
  pb = (pb + PL - 1) / PL * PL;
  if (pb < PL) pb = PL;
  return int((P + pb - 1) / pb);
}

static int64_t bn_pb(int64_t P, int J) {
  const int nb = bn_partial_blocks(P, J);
  return (P + nb - 1) / nb;
}

// block-major partials of this many channels or more take the tiled finalize
constexpr int BN_WIDE_J = 512;

void bn_finalize_fwd(hipStream_t s, const double *part, int nb, int J, int64_t m, float *st,
                     bool channel_major) {
  if (!channel_major && J >= BN_WIDE_J)
    hipLaunchKernelGGL((k_bn_finalize_wide<true>), dim3((J + 15) / 16), dim3(256), 0, s, part, nb, J,
                       double(m), st, nullptr, nullptr);
  else if (channel_major)
    hipLaunchKernelGGL((k_bn_finalize<true, true>), dim3(J), dim3(256), 0, s, part, nb, J, double(m),
                       st, nullptr, nullptr);
  else
    hipLaunchKernelGGL((k_bn_finalize<true, false>), dim3(J), dim3(256), 0, s, part, nb, J, double(m),
                       st, nullptr, nullptr);
}

void bn_finalize_bwd(hipStream_t s, const double *part, int nb, int J, int64_t m, float *sums,
                     float *dgamma, float *dbeta, bool channel_major) {
  if (!channel_major && J >= BN_WIDE_J)
    hipLaunchKernelGGL((k_bn_finalize_wide<false>), dim3((J + 15) / 16), dim3(256), 0, s, part, nb, J,
                       double(m), sums, dgamma, dbeta);
  else if (channel_major)
    hipLaunchKernelGGL((k_bn_finalize<false, true>), dim3(J), dim3(256), 0, s, part, nb, J, double(m),
                       sums, dgamma, dbeta);
  else
    hipLaunchKernelGGL((k_bn_finalize<false, false>), dim3(J), dim3(256), 0, s, part, nb, J, double(m),
                       sums, dgamma, dbeta);
}

void bn_apply(hipStream_t s, int res, int64_t P, int J, const float *Cv, const float *st,
              const float *gamma, const float *beta, const float *X, int H, int W, int Cx, float *Y) {
  const int g = ew_grid(P * (J / 4));
  if (res == BN_RES_NONE)
    hipLaunchKernelGGL((k_bn_apply<BN_RES_NONE>), dim3(g), dim3(256), 0, s, P, J, Cv, st, gamma, beta, X, H, W, Cx, Y);
  else if (res == BN_RES_ID)
    hipLaunchKernelGGL((k_bn_apply<BN_RES_ID>), dim3(g), dim3(256), 0, s, P, J, Cv, st, gamma, beta, X, H, W, Cx, Y);
  else
    hipLaunchKernelGGL((k_bn_apply<BN_RES_A>), dim3(g), dim3(256), 0, s, P, J, Cv, st, gamma, beta, X, H, W, Cx, Y);
}

void bn_stats(hipStream_t s, int64_t P, int J, const float *X, double *part, float *st) {
  const int nb = bn_partial_blocks(P, J);
  hipLaunchKernelGGL(k_bn_stats_partials, dim3(nb), dim3(256), 0, s, int(P), J, int(bn_pb(P, J)), X, part);
  bn_finalize_fwd(s, part, nb, J, P, st, true);
}

void bn_norm(hipStream_t s, int64_t P, int J, const float *X, const float *st, const float *gamma,
             const float *beta, float *Y) {
  hipLaunchKernelGGL(k_bn_norm, dim3(ew_grid(P * (J / 4))), dim3(256), 0, s, P, J, X, st, gamma, beta, Y);
}

void shortcut_a(hipStream_t s, int N, int H, int W, int J, int Cx, const float *X, float *Y) {
  const int64_t P = int64_t(N) * H * W;
  hipLaunchKernelGGL(k_shortcut_a, dim3(ew_grid(P * J)), dim3(256), 0, s, P, H, W, J, Cx, X, Y);
}

void shortcut_a_bwd(hipStream_t s, int N, int H, int W, int J, int Cx, const float *DY, float *DX) {
  const int64_t P = int64_t(N) * 4 * H * W;
  hipLaunchKernelGGL(k_shortcut_a_bwd, dim3(ew_grid(P * Cx)), dim3(256), 0, s, P, H, W, J, Cx, DY, DX);
}

void avgpool(hipStream_t s, int N, int HW, int C, const float *X, float *Y) {
  hipLaunchKernelGGL(k_avgpool, dim3((N * C + 255) / 256), dim3(256), 0, s, N, HW, C, X, Y);
}

void avgpool_bwd(hipStream_t s, int N, int HW, int C, const float *DY, float *DX) {
  const int64_t total = int64_t(N) * HW * C;
  hipLaunchKernelGGL(k_avgpool_bwd, dim3(ew_grid(total)), dim3(256), 0, s, total, HW, C, DY, DX);
}

void softmax_ce_rows(hipStream_t s, int N, int K, const float *L, const int *labels, float *G,
                     float *lossn, float *loss) {
  hipLaunchKernelGGL(k_softmax_ce_rows, dim3(N), dim3(256), 0, s, N, K, L, labels, G, lossn);
  hipLaunchKernelGGL(k_loss_mean, dim3(1), dim3(64), 0, s, N, lossn, loss);
}

void bn_backward_apply(hipStream_t s, int64_t P, int J, const float *G, const float *Ym,
                       const float *Cv, const float *st, const float *gamma, const float *sums,
                       float *D) {
  const int g = ew_grid(P * (J / 4));
  if (Ym)
    hipLaunchKernelGGL((k_bn_bwd_apply<true>), dim3(g), dim3(256), 0, s, P, J, G, Ym, Cv, st, gamma, sums, D);
  else
    hipLaunchKernelGGL((k_bn_bwd_apply<false>), dim3(g), dim3(256), 0, s, P, J, G, Ym, Cv, st, gamma, sums, D);
}

void bn_backward(hipStream_t s, int64_t P, int J, const float *G, const float *Ym, const float *Cv,
                 const float *st, const float *gamma, double *part, float *sums, float *dgamma,
                 float *dbeta, float *D) {
  const int nb = bn_partial_blocks(P, J);
  const int pb = int(bn_pb(P, J));
  if (Ym)
    hipLaunchKernelGGL((k_bn_bwd_partials<true>), dim3(nb), dim3(256), 0, s, int(P), J, pb, G, Ym, Cv, st, part);
  else
    hipLaunchKernelGGL((k_bn_bwd_partials<false>), dim3(nb), dim3(256), 0, s, int(P), J, pb, G, Ym, Cv, st, part);
  bn_finalize_bwd(s, part, nb, J, P, sums, dgamma, dbeta, true);
  const int g = ew_grid(P * (J / 4));
  if (Ym)
    hipLaunchKernelGGL((k_bn_bwd_apply<true>), dim3(g), dim3(256), 0, s, P, J, G, Ym, Cv, st, gamma, sums, D);
  else
    hipLaunchKernelGGL((k_bn_bwd_apply<false>), dim3(g), dim3(256), 0, s, P, J, G, Ym, Cv, st, gamma, sums, D);
}

void pool_fc_ce_head(hipStream_t s, int N, int HW, int C, int K, const float *X, const float *Wf,
                     const float *bf, const int *labels, float *pooled, float *dlog, float *lossn,
                     float *G, float *dW, float *db, float *loss) {
  const size_t lds = size_t(C + K + 256) * 4;
  hipLaunchKernelGGL(k_head_sample<float>, dim3(N), dim3(256), lds, s, N, HW, C, K, X, Wf, bf, labels,
                     pooled, dlog, lossn, G);
  const int tot = C * K + K + 1;
  hipLaunchKernelGGL(k_head_params, dim3((tot + 255) / 256), dim3(256), 0, s, N, C, K, pooled,
                     dlog, lossn, dW, db, loss);
}

void pool_fc_ce_head_bf16(hipStream_t s, int N, int HW, int C, int K, const void *X, const float *Wf,
                          const float *bf, const int *labels, float *pooled, float *dlog,
                          float *lossn, float *dpool, float *G, float *dW, float *db, float *loss) {
  hipLaunchKernelGGL(k_head_pool_bf16, dim3((N * C + 255) / 256), dim3(256), 0, s, N, HW, C,
                     static_cast<const __bf16 *>(X), pooled);
  gemm_f32(s, N, K, C, pooled, C, false, Wf, K, false, dlog, K, GEMM_EPI_BIAS, nullptr, 0, bf);
  hipLaunchKernelGGL(k_head_softmax, dim3(N), dim3(256), size_t(K + 256) * 4, s, N, K, labels, dlog, lossn);
  gemm_f32(s, N, C, K, dlog, K, false, Wf, K, true, dpool, C, GEMM_EPI_STORE);
  hipLaunchKernelGGL(k_head_bcast, dim3(ew_grid(int64_t(N) * HW * C)), dim3(256), 0, s, N, HW, C, dpool, G);
  const int tot = C * K + K + 1;
  hipLaunchKernelGGL(k_head_params, dim3((tot + 255) / 256), dim3(256), 0, s, N, C, K, pooled,
                     dlog, lossn, dW, db, loss);
}

}  // namespace ckpt
