// Pointwise and row kernels of the LSTM step with its softmax head.
//   gates  i, f, g, o = sigma(z_i), sigma(z_f), tanh(z_g), sigma(z_o)
//          (z columns [0,H), [H,2H), [2H,3H), [3H,4H))
//   cell   c_t = f c_{t-1} + i g,   h_t = o tanh(c_t)   (c fp32, h rounded to bf16)
//   head   softmax cross-entropy of a [B, V] row block; the gradient
//          (p - onehot) * scale is kept in fp32
// Every sum (split-K slices, bias-gradient columns) runs in an order fixed by
// the shapes alone, so a step is bit-reproducible whatever the schedule.
#include <hip/hip_runtime.h>

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

// One workgroup per row: loss_row = log sum exp(l - max) + max - l[label];
// dlog = (softmax - onehot) * scale.  A label outside [0, V) gives a NaN loss
// for the row and no one-hot term.
// One workgroup of 1024 threads per row: each thread keeps its (at most
// SM_PER) logits in registers; max and sum are reduced by wavefront
// butterflies and then across the 16 wavefronts in a fixed order.
constexpr int SM_THREADS = 1024, SM_PER = 16;

__device__ __forceinline__ float wave_max(float v) {
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// logits = sum of the ns partial slices [rows, V] + bias
__global__ __launch_bounds__(SM_THREADS) void k_softmax_ce_rows(int V, const float *__restrict__ lpart,
                                                                int ns, size_t slice,
                                                                const float *__restrict__ bias,
                                                                const int *__restrict__ labels, float scale,
                                                                float *__restrict__ dlog,
                                                                float *__restrict__ loss_rows) {
  __shared__ float red[SM_THREADS / 64];
  __shared__ float lab_logit;
  const int row = blockIdx.x, t = threadIdx.x, lane = t & 63, w = t >> 6;
  const size_t r0 = size_t(row) * V;
  const int lab = labels[row];
  float x[SM_PER];
  size_t o[SM_PER];
  // columns past V read column V - 1 (in bounds) and are dropped below
#pragma unroll
  for (int k = 0; k < SM_PER; ++k) o[k] = r0 + min(t + k * SM_THREADS, V - 1);
  slices_sum<SM_PER, 1>(lpart, ns, slice, o, x);
  float mx = -INFINITY;
#pragma unroll
  for (int k = 0; k < SM_PER; ++k) {
    const int v = t + k * SM_THREADS;
    x[k] = v < V ? x[k] + bias[v] : -INFINITY;
    if (v == lab) lab_logit = x[k];
    mx = fmaxf(mx, x[k]);
  }
  mx = wave_max(mx);
  if (lane == 0) red[w] = mx;
  __syncthreads();
  mx = red[0];
  for (int k = 1; k < SM_THREADS / 64; ++k) mx = fmaxf(mx, red[k]);
  __syncthreads();
  float se = 0.f;
#pragma unroll
  for (int k = 0; k < SM_PER; ++k) {
    const int v = t + k * SM_THREADS;
    x[k] = v < V ? expf(x[k] - mx) : 0.f;
    se += x[k];
  }
  se = wave_sum(se);
  if (lane == 0) red[w] = se;
  __syncthreads();
  se = 0.f;
  for (int k = 0; k < SM_THREADS / 64; ++k) se += red[k];
  const bool ok = lab >= 0 && lab < V;
  if (t == 0) loss_rows[row] = ok ? (logf(se) + mx) - lab_logit : NAN;
  const float inv = 1.0f / se;
  float *d = dlog + size_t(row) * V;
#pragma unroll
  for (int k = 0; k < SM_PER; ++k) {
    const int v = t + k * SM_THREADS;
    if (v < V) d[v] = (x[k] * inv - (v == lab ? 1.f : 0.f)) * scale;
  }
}

// Workgroup = 64 columns x 4 row groups (rows b = rg, rg + 4, ...); the
// column sums of the groups are combined in order ((s0 + s1) + s2) + s3.

// dl_bf[b][v] = bf16(dlog[b][v]);  db_o[v] (+)= sum_b dlog[b][v]
__global__ __launch_bounds__(256) void k_head_bwd_prep(int B, int V, const float *__restrict__ dlog,
                                                       __bf16 *__restrict__ dl_bf,
                                                       float *__restrict__ db_o, int first) {
  __shared__ float part[4][64];
  const int cx = threadIdx.x & 63, rg = threadIdx.x >> 6;
  const int v = blockIdx.x * 64 + cx;
  float s = 0.f;
  if (v < V)
    for (int b = rg; b < B; b += 4) {
      const float d = dlog[size_t(b) * V + v];
      dl_bf[size_t(b) * V + v] = (__bf16)d;
      s += d;
    }
  part[rg][cx] = s;
  __syncthreads();
  if (rg == 0 && v < V) {
    const float t = ((part[0][cx] + part[1][cx]) + part[2][cx]) + part[3][cx];
    db_o[v] = first ? t : db_o[v] + t;
  }
}

// Gate backward, one thread per (b, j): workgroup = 64 hidden units x 4
// batch rows (blockIdx.y = row block).  dh = the ns partial slices [B, H] of
// the head gradient's product, in order, + the incoming dh (dh_in, [B, H]).
// The workgroup's bias-gradient column sums over its 4 rows, ((r0 + r1) + r2)
// + r3, go to dbp[blockIdx.y][4H]; k_db_chunk adds them up.
__global__ __launch_bounds__(256) void k_lstm_bwd_point(int B, int H, const float *__restrict__ dhpart,
                                                        int ns, const float *__restrict__ dh_in,
                                                        const float *__restrict__ dc_in,
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
    const float dhv = dh[0] + dh_in[e];
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

void cvt_bf16(hipStream_t s, int64_t n, const float *src, void *dst) {
  hipLaunchKernelGGL(k_cvt_bf16, dim3(grid_for(n)), dim3(256), 0, s, n, src, static_cast<__bf16 *>(dst));
}

void lstm_fwd_point(hipStream_t s, int B, int H, const float *zpart, int ns, const float *bias,
                    const float *c_prev, float *gates, void *h_out, float *c_out) {
  hipLaunchKernelGGL(k_lstm_fwd_point, dim3((B * H + 255) / 256), dim3(256), 0, s, B, H, zpart, ns,
                     bias, c_prev, gates, static_cast<__bf16 *>(h_out), c_out);
}

void softmax_ce_rows(hipStream_t s, int rows, int V, const float *lpart, int ns, const float *bias,
                     const int *labels, float scale, float *dlog, float *loss_rows) {
  hipLaunchKernelGGL(k_softmax_ce_rows, dim3(rows), dim3(SM_THREADS), 0, s, V, lpart, ns,
                     size_t(rows) * V, bias, labels, scale, dlog, loss_rows);
}

void head_bwd_prep(hipStream_t s, int B, int V, const float *dlog, void *dl_bf, float *db_o, bool first) {
  hipLaunchKernelGGL(k_head_bwd_prep, dim3((V + 63) / 64), dim3(256), 0, s, B, V, dlog,
                     static_cast<__bf16 *>(dl_bf), db_o, first ? 1 : 0);
}

void lstm_bwd_point(hipStream_t s, int B, int H, const float *dhpart, int ns, const float *dh_in,
                    const float *dc_in, const float *gates, const float *c_t, const float *c_prev,
                    const void *h_prev, const void *h_t, void *dz, float *dc_prev, void *hp_copy,
                    void *hc_copy, float *dbp) {
  hipLaunchKernelGGL(k_lstm_bwd_point, dim3((H + 63) / 64, (B + 3) / 4), dim3(256), 0, s, B, H, dhpart,
                     ns, dh_in, dc_in, gates, c_t, c_prev, static_cast<const __bf16 *>(h_prev),
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
