// Elementwise and reduction kernels of the residual-MLP unit and the MSE head.
// Reductions are fixed-order trees (no atomics), so every result is
// reproducible bit for bit.
#include <hip/hip_runtime.h>

#include "kernels.h"

namespace ckpt {
namespace {

// One block per 64 columns; 4 row groups per block.  dr = g * [z > 0];
// db[n] = ((s0 + s1) + s2) + s3 where s_j sums rows j, j+4, ... in order.
__global__ __launch_bounds__(256) void k_mlp_relu_bwd(int rows, int cols, const float *__restrict__ g,
                                                      const float *__restrict__ z,
                                                      float *__restrict__ dr, float *__restrict__ db) {
  __shared__ float part[4][64];
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  const int n = blockIdx.x * 64 + tx;
  float s = 0.f;
  if (n < cols) {
    for (int m = ty; m < rows; m += 4) {
      size_t i = size_t(m) * cols + n;
      float v = z[i] > 0.f ? g[i] : 0.f;
      dr[i] = v;
      s += v;
    }
  }
  part[ty][tx] = s;
  __syncthreads();
  if (ty == 0 && n < cols) db[n] = ((part[0][tx] + part[1][tx]) + part[2][tx]) + part[3][tx];
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

}  // namespace

void mlp_relu_bwd(hipStream_t s, int rows, int cols, const float *g, const float *z, float *dr,
                  float *db) {
  hipLaunchKernelGGL(k_mlp_relu_bwd, dim3((cols + 63) / 64), dim3(256), 0, s, rows, cols, g, z, dr, db);
}

void mse_head(hipStream_t s, int64_t count, const float *y, const float *t, float *g, float *loss_out) {
  hipLaunchKernelGGL(k_mse_head, dim3(1), dim3(1024), 0, s, count, y, t, g, loss_out);
}

void copy_scalar(hipStream_t s, const float *src, float *dst) {
  hipLaunchKernelGGL(k_copy_scalar, dim3(1), dim3(1), 0, s, src, dst);
}

}  // namespace ckpt
