// Pointwise and row kernels of the LSTM step with its softmax head.
//   gates  i, f, g, o = sigma(z_i), sigma(z_f), tanh(z_g), sigma(z_o)
//          (z columns [0,H), [H,2H), [2H,3H), [3H,4H))
//   cell   c_t = f c_{t-1} + i g,   h_t = o tanh(c_t)   (c fp32, h rounded to bf16)
//   head   softmax cross-entropy of a [B, V] row block; the gradient
//          (p - onehot) * scale is kept in fp32
// Every sum (split-K slices, bias-gradient columns) runs in an order fixed by
// the shapes alone, so a step is bit-reproducible whatever the schedule.
#include <hip/hip_runtime.h>

#include "common.h"
#include "kernels.h"

namespace ckpt {
namespace {

__device__ __forceinline__ float sigm(float x) { return 1.0f / (1.0f + expf(-x)); }

// NV elements o[0..NV) of a split-K product: each element's ns partial
// slices (slice stride `slice`) added in slice order -- the order sum_slices
// uses.  Slices are fetched U at a time for all NV elements before any of
// them is added, so the loads of a round are in flight together.
template <int NV, int U>
__device__ __forceinline__ void slices_sum(const float *__restrict__ part, int ns, size_t slice,
                                           const size_t (&o)[NV], float (&v)[NV]) {
#pragma unroll
  for (int k = 0; k < NV; ++k) v[k] = part[o[k]];
  int z = 1;
  for (; z + U <= ns; z += U) {
    float t[U][NV];
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int k = 0; k < NV; ++k) t[u][k] = part[(z + u) * slice + o[k]];
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int k = 0; k < NV; ++k) v[k] += t[u][k];
  }
  for (; z < ns; ++z)
#pragma unroll
    for (int k = 0; k < NV; ++k) v[k] += part[z * slice + o[k]];
}

// dst[c][r] = bf16(src[r][c]) for src [R][C] fp32, through 32x32 LDS tiles.
__global__ __launch_bounds__(256) void k_transpose_bf16(int R, int C, const float *__restrict__ src,
                                                        __bf16 *__restrict__ dst, int ld) {
  __shared__ float t[32][33];
  const int c0 = blockIdx.x * 32, r0 = blockIdx.y * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  for (int k = ty; k < 32; k += 8) {
    const int r = r0 + k, c = c0 + tx;
    t[k][tx] = (r < R && c < C) ? src[size_t(r) * C + c] : 0.f;
  }
  __syncthreads();
  for (int k = ty; k < 32; k += 8) {
    const int c = c0 + k, r = r0 + tx;
    if (c < C && r < R) dst[size_t(c) * ld + r] = (__bf16)t[tx][k];
  }
}

__global__ __launch_bounds__(256) void k_cvt_bf16(int64_t n, const float *__restrict__ src,
                                                  __bf16 *__restrict__ dst) {
  for (int64_t e = blockIdx.x * int64_t(256) + threadIdx.x; e < n; e += int64_t(gridDim.x) * 256)
    dst[e] = (__bf16)src[e];
}

// the same conversion, eight elements per thread and iteration (two 16-byte
// loads, one 16-byte store) for n a multiple of 8 with src 16-byte and dst
// 16-byte aligned
__global__ __launch_bounds__(256) void k_cvt_bf16x8(int64_t n8, const float4 *__restrict__ src,
                                                    uint4 *__restrict__ dst) {
  for (int64_t e = blockIdx.x * int64_t(256) + threadIdx.x; e < n8; e += int64_t(gridDim.x) * 256) {
    const float4 a = src[2 * e], b = src[2 * e + 1];
    const float f[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
    unsigned w[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const __bf16 lo = (__bf16)f[2 * k], hi = (__bf16)f[2 * k + 1];
      w[k] = unsigned(__builtin_bit_cast(unsigned short, lo)) |
             (unsigned(__builtin_bit_cast(unsigned short, hi)) << 16);
    }
    dst[e] = make_uint4(w[0], w[1], w[2], w[3]);
  }
}

// dst[r * ld + c] = bf16(src[r * C + c]) for src [R][C] fp32
__global__ __launch_bounds__(256) void k_cvt_bf16_rows(int R, int C, const float *__restrict__ src,
                                                       __bf16 *__restrict__ dst, int ld) {
  const int64_t n = int64_t(R) * C;
  for (int64_t e = blockIdx.x * int64_t(256) + threadIdx.x; e < n; e += int64_t(gridDim.x) * 256)
    dst[(e / C) * ld + e % C] = (__bf16)src[e];
}

// one thread per (b, j); z = sum of the ns partial slices [B, 4H] + bias
__global__ __launch_bounds__(256) void k_lstm_fwd_point(int B, int H, const float *__restrict__ zpart,
                                                        int ns, const float *__restrict__ bias,
                                                        const float *__restrict__ c_prev,
                                                        float *__restrict__ gates,
                                                        __bf16 *__restrict__ h_out,
                                                        float *__restrict__ c_out) {
  const int e = blockIdx.x * 256 + threadIdx.x;
  if (e >= B * H) return;
  const int b = e / H, j = e % H;
  const size_t r = size_t(b) * 4 * H + j;
  const size_t o[4] = {r, r + H, r + 2 * H, r + 3 * H};
  float z[4];
  slices_sum<4, 4>(zpart, ns, size_t(B) * 4 * H, o, z);
  const float ig = sigm(z[0] + bias[j]);
  const float fg = sigm(z[1] + bias[H + j]);
  const float gg = tanhf(z[2] + bias[2 * H + j]);
  const float og = sigm(z[3] + bias[3 * H + j]);
  const float cp = c_prev ? c_prev[e] : 0.f;
  const float c = fg * cp + ig * gg;
  float *gr = gates + size_t(b) * 4 * H;
  gr[j] = ig;
  gr[H + j] = fg;
  gr[2 * H + j] = gg;
  gr[3 * H + j] = og;
  c_out[e] = c;
  h_out[e] = (__bf16)(og * tanhf(c));
}

// (m, s) <- the pair for the union of two column sets: m the larger maximum,
// s both sums rescaled to it (0 while both sets are empty)
__device__ __forceinline__ void lse_combine(float &m, float &s, float om, float os) {
  const float mx = fmaxf(m, om);
  s = mx == -INFINITY ? 0.f : s * expf(m - mx) + os * expf(om - mx);
  m = mx;
}

// Softmax cross-entropy: loss_row = log sum exp(l - max) + max - l[label],
// dlog = (softmax - onehot) * scale (a label outside [0, V) gives a NaN loss
// for the row and no one-hot term), from the logits l (bias included) and
// each row's (max, sum of exp) pairs per column tile of the product that
// wrote them.  Every
// wavefront combines its row's pairs itself (lane j takes tiles j, j + 64,
// ... in order, then a butterfly, whose pairwise combinations are symmetric),
// so all workgroups of a row use the same maximum and sum with no exchange
// between them.  Workgroup = 1024 columns of one row, four per thread;
// blockIdx.z = the unit of a batch (its logits, dlog and statistics ul, ul
// and ur floats after the previous unit's, its labels and loss rows `rows`
// after).  The row's loss is formed by the thread that holds the label's
// logit, from its register, so dlog may overwrite the logits in place.
__global__ __launch_bounds__(256) void k_softmax_ce_tiles(int V, const float *logits, int nt,
                                                          const float *__restrict__ rstat,
                                                          const int *__restrict__ labels, float scale,
                                                          float *dlog, float *__restrict__ loss_rows,
                                                          int rows, int64_t ul, int64_t ur) {
  const int row = blockIdx.y, lane = threadIdx.x & 63;
  const int64_t u = blockIdx.z;
  logits += u * ul;
  dlog += u * ul;
  labels += u * rows;
  loss_rows += u * rows;
  const float *rs = rstat + u * ur + size_t(row) * nt * 2;
  float m = -INFINITY, se = 0.f;
  for (int j = lane; j < nt; j += 64) lse_combine(m, se, rs[2 * j], rs[2 * j + 1]);
  for (int o = 32; o > 0; o >>= 1) {
    const float om = __shfl_xor(m, o, 64), os = __shfl_xor(se, o, 64);
    lse_combine(m, se, om, os);
  }
  const int lab = labels[row];
  const float inv = 1.0f / se;
  const int v0 = (blockIdx.x * 256 + threadIdx.x) * 4;
  const float *x = logits + size_t(row) * V;
  if (v0 < V) {
    const float4 xv = *reinterpret_cast<const float4 *>(x + v0);
    const float xs[4] = {xv.x, xv.y, xv.z, xv.w};
    float d[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      d[k] = (expf(xs[k] - m) * inv - (v0 + k == lab ? 1.f : 0.f)) * scale;
      if (v0 + k == lab) loss_rows[row] = (logf(se) + m) - xs[k];
    }
    *reinterpret_cast<float4 *>(dlog + size_t(row) * V + v0) = make_float4(d[0], d[1], d[2], d[3]);
  }
  if (blockIdx.x == 0 && threadIdx.x == 0 && !(lab >= 0 && lab < V)) loss_rows[row] = NAN;
}

// Workgroup = 32 columns x 16 row groups, so V = 10000 gives 313 workgroups,
// more than there are compute units; group rg takes rows b = rg, rg + 16, ...,
// issuing four row loads before it uses any, and adds them in row order.  The
// column sums of the groups are combined as a fixed pairwise tree.

// dl_bf[b][v] = bf16(dlog[b][v]);  db_o[v] (+)= sum_b dlog[b][v]
__global__ __launch_bounds__(512) void k_head_bwd_prep(int B, int V, const float *__restrict__ dlog,
                                                       __bf16 *__restrict__ dl_bf,
                                                       float *__restrict__ db_o, int first) {
  __shared__ float part[16][32];
  const int cx = threadIdx.x & 31, rg = threadIdx.x >> 5;
  const int v = blockIdx.x * 32 + cx;
  float s = 0.f;
  if (v < V)
    for (int b0 = rg; b0 < B; b0 += 64) {
      float d[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int b = b0 + 16 * u;
        d[u] = b < B ? dlog[size_t(b) * V + v] : 0.f;
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int b = b0 + 16 * u;
        if (b < B) {
          dl_bf[size_t(b) * V + v] = (__bf16)d[u];
          s += d[u];
        }
      }
    }
  part[rg][cx] = s;
  __syncthreads();
  if (rg == 0 && v < V) {
    float q[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) q[i] = part[2 * i][cx] + part[2 * i + 1][cx];
    const float t = (((q[0] + q[1]) + (q[2] + q[3])) + ((q[4] + q[5]) + (q[6] + q[7])));
    db_o[v] = first ? t : db_o[v] + t;
  }
}

// Gate backward, one thread per (b, j): workgroup = 64 hidden units x 4
// batch rows (blockIdx.y = row block).  dh = the ns partial slices [B, H] of
// the product that forms it (head gradient and, but for the last step, the
// next step's dz W_h^T), added in order.
// The workgroup's bias-gradient column sums over its 4 rows, ((r0 + r1) + r2)
// + r3, go to dbp[blockIdx.y][4H]; k_db_chunk adds them up.
__global__ __launch_bounds__(256) void k_lstm_bwd_point(int B, int H, const float *__restrict__ dhpart,
                                                        int ns, const float *__restrict__ dc_in,
                                                        const float *__restrict__ gates,
                                                        const float *__restrict__ c_t,
                                                        const float *__restrict__ c_prev,
                                                        const __bf16 *__restrict__ h_prev,
                                                        const __bf16 *__restrict__ h_t,
                                                        __bf16 *__restrict__ dz,
                                                        float *__restrict__ dc_prev,
                                                        __bf16 *__restrict__ hp_copy,
                                                        __bf16 *__restrict__ hc_copy,
                                                        float *__restrict__ dbp) {
  __shared__ float part[4][4][64];
  const int cx = threadIdx.x & 63, rg = threadIdx.x >> 6;
  const int j = blockIdx.x * 64 + cx, b = blockIdx.y * 4 + rg;
  float zv[4] = {0.f, 0.f, 0.f, 0.f};
  if (j < H && b < B) {
    const size_t e = size_t(b) * H + j;
    const size_t oe[1] = {e};
    float dh[1];
    slices_sum<1, 8>(dhpart, ns, size_t(B) * H, oe, dh);
    const float dhv = dh[0];
    const float *gr = gates + size_t(b) * 4 * H;
    const float ig = gr[j], fg = gr[H + j], gg = gr[2 * H + j], og = gr[3 * H + j];
    const float tc = tanhf(c_t[e]);
    const float dct = dc_in[e] + dhv * og * (1.f - tc * tc);
    const float cp = c_prev ? c_prev[e] : 0.f;
    zv[0] = dct * gg * ig * (1.f - ig);
    zv[1] = dct * cp * fg * (1.f - fg);
    zv[2] = dct * ig * (1.f - gg * gg);
    zv[3] = dhv * tc * og * (1.f - og);
    __bf16 *dr = dz + size_t(b) * 4 * H;
#pragma unroll
    for (int k = 0; k < 4; ++k) dr[k * H + j] = (__bf16)zv[k];
    if (dc_prev) dc_prev[e] = dct * fg;
    hp_copy[e] = h_prev ? h_prev[e] : (__bf16)0.f;
    hc_copy[e] = h_t[e];
  }
#pragma unroll
  for (int k = 0; k < 4; ++k) part[k][rg][cx] = zv[k];
  __syncthreads();
  if (j < H) {
    const int k = rg;  // row group rg writes gate k's column sum
    const float t = ((part[k][0][cx] + part[k][1][cx]) + part[k][2][cx]) + part[k][3][cx];
    dbp[size_t(blockIdx.y) * 4 * H + size_t(k) * H + j] = t;
  }
}

// db[n] (+)= the nrec records rec[r][n] (record stride N), r = 0 .. nrec-1:
// workgroup = 64 columns x 4 groups of consecutive records; each group adds
// its records in order, the groups combine as ((g0 + g1) + g2) + g3.
__global__ __launch_bounds__(256) void k_db_chunk(int N, int nrec, const float *__restrict__ rec,
                                                  float *__restrict__ db, int first) {
  __shared__ float part[4][64];
  const int cx = threadIdx.x & 63, g = threadIdx.x >> 6;
  const int n = blockIdx.x * 64 + cx;
  const int per = (nrec + 3) / 4, r0 = min(nrec, g * per), r1 = min(nrec, r0 + per);
  float s = 0.f;
  if (n < N) {
    int r = r0;
    for (; r + 8 <= r1; r += 8) {
      float t[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) t[u] = rec[size_t(r + u) * N + n];
#pragma unroll
      for (int u = 0; u < 8; ++u) s += t[u];
    }
    for (; r < r1; ++r) s += rec[size_t(r) * N + n];
  }
  part[g][cx] = s;
  __syncthreads();
  if (g == 0 && n < N) {
    const float t = ((part[0][cx] + part[1][cx]) + part[2][cx]) + part[3][cx];
    db[n] = first ? t : db[n] + t;
  }
}

// loss = scale * sum of rows (fixed order: thread t takes rows t, t+1024, ...)
__global__ __launch_bounds__(1024) void k_loss_reduce(int64_t rows, const float *__restrict__ v,
                                                      float scale, float *__restrict__ loss) {
  __shared__ float red[1024];
  float s = 0.f;
  for (int64_t r = threadIdx.x; r < rows; r += 1024) s += v[r];
  red[threadIdx.x] = s;
  __syncthreads();
  for (int w = 512; w > 0; w >>= 1) {
    if (threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) loss[0] = red[0] * scale;
}

__global__ __launch_bounds__(256) void k_fill_f32(int64_t n, float *__restrict__ p, float v) {
  for (int64_t e = blockIdx.x * int64_t(256) + threadIdx.x; e < n; e += int64_t(gridDim.x) * 256) p[e] = v;
}

inline int grid_for(int64_t n) {
  int64_t g = (n + 255) / 256;
  return int(g < 1 ? 1 : (g > 8192 ? 8192 : g));
}

}  // namespace

void transpose_bf16(hipStream_t s, int R, int C, const float *src, void *dst, int ld) {
  hipLaunchKernelGGL(k_transpose_bf16, dim3((C + 31) / 32, (R + 31) / 32), dim3(256), 0, s, R, C,
                     src, static_cast<__bf16 *>(dst), ld > 0 ? ld : R);
}

void cvt_bf16_rows(hipStream_t s, int R, int C, const float *src, void *dst, int ld) {
  hipLaunchKernelGGL(k_cvt_bf16_rows, dim3(grid_for(int64_t(R) * C)), dim3(256), 0, s, R, C, src,
                     static_cast<__bf16 *>(dst), ld);
}

void cvt_bf16(hipStream_t s, int64_t n, const float *src, void *dst) {
  if (n % 8 == 0 && uintptr_t(src) % 16 == 0 && uintptr_t(dst) % 16 == 0) {
    hipLaunchKernelGGL(k_cvt_bf16x8, dim3(grid_for(n / 8)), dim3(256), 0, s, n / 8,
                       reinterpret_cast<const float4 *>(src), static_cast<uint4 *>(dst));
    return;
  }
  hipLaunchKernelGGL(k_cvt_bf16, dim3(grid_for(n)), dim3(256), 0, s, n, src, static_cast<__bf16 *>(dst));
}

void lstm_fwd_point(hipStream_t s, int B, int H, const float *zpart, int ns, const float *bias,
                    const float *c_prev, float *gates, void *h_out, float *c_out) {
  hipLaunchKernelGGL(k_lstm_fwd_point, dim3((B * H + 255) / 256), dim3(256), 0, s, B, H, zpart, ns,
                     bias, c_prev, gates, static_cast<__bf16 *>(h_out), c_out);
}

void softmax_ce_tiles(hipStream_t s, int rows, int V, const float *logits, int nt, const float *rstat,
                      const int *labels, float scale, float *dlog, float *loss_rows) {
  if (V % 4 != 0 || reinterpret_cast<uintptr_t>(logits) % 16 != 0 ||
      reinterpret_cast<uintptr_t>(dlog) % 16 != 0)
    fail(CKPT_E_INVALID, "softmax_ce_tiles: V must be a multiple of 4 and the rows 16-byte aligned");
  hipLaunchKernelGGL(k_softmax_ce_tiles, dim3((V + 1023) / 1024, rows), dim3(256), 0, s, V, logits, nt,
                     rstat, labels, scale, dlog, loss_rows, rows, int64_t(0), int64_t(0));
}

void softmax_ce_tiles_batched(hipStream_t s, int nunits, int rows, int V, float *logits, int64_t ul, int nt,
                              const float *rstat, int64_t ur, const int *labels, float scale,
                              float *loss_rows) {
  if (nunits <= 0) return;
  if (V % 4 != 0 || ul % 4 != 0 || reinterpret_cast<uintptr_t>(logits) % 16 != 0)
    fail(CKPT_E_INVALID, "softmax_ce_tiles_batched: V and the unit stride multiples of 4, rows 16-byte aligned");
  hipLaunchKernelGGL(k_softmax_ce_tiles, dim3((V + 1023) / 1024, rows, nunits), dim3(256), 0, s, V, logits,
                     nt, rstat, labels, scale, logits, loss_rows, rows, ul, ur);
}

void head_bwd_prep(hipStream_t s, int B, int V, const float *dlog, void *dl_bf, float *db_o, bool first) {
  hipLaunchKernelGGL(k_head_bwd_prep, dim3((V + 31) / 32), dim3(512), 0, s, B, V, dlog,
                     static_cast<__bf16 *>(dl_bf), db_o, first ? 1 : 0);
}

void lstm_bwd_point(hipStream_t s, int B, int H, const float *dhpart, int ns, const float *dc_in,
                    const float *gates, const float *c_t, const float *c_prev, const void *h_prev,
                    const void *h_t, void *dz, float *dc_prev, void *hp_copy, void *hc_copy,
                    float *dbp) {
  hipLaunchKernelGGL(k_lstm_bwd_point, dim3((H + 63) / 64, (B + 3) / 4), dim3(256), 0, s, B, H, dhpart,
                     ns, dc_in, gates, c_t, c_prev, static_cast<const __bf16 *>(h_prev),
                     static_cast<const __bf16 *>(h_t), static_cast<__bf16 *>(dz), dc_prev,
                     static_cast<__bf16 *>(hp_copy), static_cast<__bf16 *>(hc_copy), dbp);
}

void db_chunk(hipStream_t s, int N, int nrec, const float *rec, float *db, bool first) {
  hipLaunchKernelGGL(k_db_chunk, dim3((N + 63) / 64), dim3(256), 0, s, N, nrec, rec, db, first ? 1 : 0);
}

void loss_reduce(hipStream_t s, int64_t rows, const float *v, float scale, float *loss) {
  hipLaunchKernelGGL(k_loss_reduce, dim3(1), dim3(1024), 0, s, rows, v, scale, loss);
}

void fill_f32(hipStream_t s, int64_t n, float *p, float v) {
  hipLaunchKernelGGL(k_fill_f32, dim3(grid_for(n)), dim3(256), 0, s, n, p, v);
}

}  // namespace ckpt
