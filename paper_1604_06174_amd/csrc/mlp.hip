// Elementwise and reduction kernels of the residual-MLP unit and the MSE head.
// Reductions are fixed-order trees (no atomics), so every result is
// reproducible bit for bit.
#include <hip/hip_runtime.h>

#include "kernels.h"

namespace ckpt {
namespace {

// Workgroup = 64 columns x 4 row groups over a block of 16 rows (blockIdx.y);
// MASK: dr = g * [z > 0], else the sums are of g itself; the workgroup's
// column sums over its rows, ((s0 + s1) + s2) + s3 with s_j = rows j, j+4, ..
// in order, go to pdb[blockIdx.y][cols].
template <bool MASK>
__global__ __launch_bounds__(256) void k_mlp_relu_bwd(int rows, int cols, const float *__restrict__ g,
                                                      const float *__restrict__ z,
                                                      float *__restrict__ dr, float *__restrict__ pdb) {
  __shared__ float part[4][64];
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  const int n = blockIdx.x * 64 + tx, r0 = blockIdx.y * 16 + ty;
  float s = 0.f;
  if (n < cols) {
    float gv[4], zv[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m = r0 + 4 * i;
      const size_t e = size_t(m < rows ? m : 0) * cols + n;
      gv[i] = g[e];
      zv[i] = MASK ? z[e] : 0.f;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m = r0 + 4 * i;
      if (m < rows) {
        const float v = MASK ? (zv[i] > 0.f ? gv[i] : 0.f) : gv[i];
        if (MASK) dr[size_t(m) * cols + n] = v;
        s += v;
      }
    }
  }
  part[ty][tx] = s;
  __syncthreads();
  if (ty == 0 && n < cols)
    pdb[size_t(blockIdx.y) * cols + n] = ((part[0][tx] + part[1][tx]) + part[2][tx]) + part[3][tx];
}

// db[n] = sum over r < R of pdb[r][n], in order of r
__global__ __launch_bounds__(256) void k_colsum_rows(int R, int cols, const float *__restrict__ pdb,
                                                     float *__restrict__ db) {
  const int n = blockIdx.x * 256 + threadIdx.x;
  if (n >= cols) return;
  float s = 0.f;
  int r = 0;
  for (; r + 8 <= R; r += 8) {
    float t[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) t[u] = pdb[size_t(r + u) * cols + n];
#pragma unroll
    for (int u = 0; u < 8; ++u) s += t[u];
  }
  for (; r < R; ++r) s += pdb[size_t(r) * cols + n];
  db[n] = s;
}

// Single block of 1024 threads: thread t sums elements t, t+1024, ...; then a
// fixed binary tree in LDS.
__global__ __launch_bounds__(1024) void k_mse_head(int64_t count, const float *__restrict__ y,
                                                   const float *__restrict__ t, float *__restrict__ g,
                                                   float *__restrict__ loss_out) {
  __shared__ float red[1024];
  const float inv = 1.0f / float(count);
  float s = 0.f;
  for (int64_t i = threadIdx.x; i < count; i += 1024) {
    float d = y[i] - t[i];
    g[i] = 2.0f * d * inv;
    s += d * d;
  }
  red[threadIdx.x] = s;
  __syncthreads();
  for (int w = 512; w > 0; w >>= 1) {
    if (threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) loss_out[0] = red[0] * inv;
}

__global__ void k_copy_scalar(const float *src, float *dst) { dst[0] = src[0]; }

// Elementwise operators of the node-level graph (any of the pointers may
// alias the output: every thread reads its element before writing it).
enum { EW_RELU = 0, EW_ADD = 1, EW_RELU_BWD = 2, EW_COPY = 3 };
template <int OP>
__global__ __launch_bounds__(256) void k_elementwise(int64_t n, const float *a, const float *b, float *y) {
  for (int64_t e = blockIdx.x * int64_t(256) + threadIdx.x; e < n; e += int64_t(gridDim.x) * 256) {
    const float x = a[e];
    float v;
    if (OP == EW_RELU) v = fmaxf(x, 0.f);
    else if (OP == EW_ADD) v = x + b[e];
    else if (OP == EW_RELU_BWD) v = b[e] > 0.f ? x : 0.f;
    else v = x;
    y[e] = v;
  }
}

int ew_blocks(int64_t n) {
  const int64_t b = (n + 255) / 256;
  return int(b < 4096 ? (b > 0 ? b : 1) : 4096);
}

}  // namespace

int mlp_relu_row_blocks(int rows) { return (rows + 15) / 16; }

void mlp_relu_bwd(hipStream_t s, int rows, int cols, const float *g, const float *z, float *dr,
                  float *db, float *pdb) {
  const int R = mlp_relu_row_blocks(rows);
  hipLaunchKernelGGL(k_mlp_relu_bwd<true>, dim3((cols + 63) / 64, R), dim3(256), 0, s, rows, cols, g, z,
                     dr, pdb);
  hipLaunchKernelGGL(k_colsum_rows, dim3((cols + 255) / 256), dim3(256), 0, s, R, cols, pdb, db);
}

void mlp_colsum(hipStream_t s, int rows, int cols, const float *g, float *db, float *pdb) {
  const int R = mlp_relu_row_blocks(rows);
  hipLaunchKernelGGL(k_mlp_relu_bwd<false>, dim3((cols + 63) / 64, R), dim3(256), 0, s, rows, cols, g,
                     nullptr, nullptr, pdb);
  hipLaunchKernelGGL(k_colsum_rows, dim3((cols + 255) / 256), dim3(256), 0, s, R, cols, pdb, db);
}

void ew_relu(hipStream_t s, int64_t n, const float *x, float *y) {
  hipLaunchKernelGGL(k_elementwise<EW_RELU>, dim3(ew_blocks(n)), dim3(256), 0, s, n, x, nullptr, y);
}
void ew_add(hipStream_t s, int64_t n, const float *a, const float *b, float *y) {
  hipLaunchKernelGGL(k_elementwise<EW_ADD>, dim3(ew_blocks(n)), dim3(256), 0, s, n, a, b, y);
}
void ew_relu_bwd(hipStream_t s, int64_t n, const float *dy, const float *y, float *dx) {
  hipLaunchKernelGGL(k_elementwise<EW_RELU_BWD>, dim3(ew_blocks(n)), dim3(256), 0, s, n, dy, y, dx);
}
void ew_copy(hipStream_t s, int64_t n, const float *x, float *y) {
  hipLaunchKernelGGL(k_elementwise<EW_COPY>, dim3(ew_blocks(n)), dim3(256), 0, s, n, x, nullptr, y);
}

void mse_head(hipStream_t s, int64_t count, const float *y, const float *t, float *g, float *loss_out) {
  hipLaunchKernelGGL(k_mse_head, dim3(1), dim3(1024), 0, s, count, y, t, g, loss_out);
}

void copy_scalar(hipStream_t s, const float *src, float *dst) {
  hipLaunchKernelGGL(k_copy_scalar, dim3(1), dim3(1), 0, s, src, dst);
}

}  // namespace ckpt
