// Attainable matrix-core and HBM throughput of the device the roofline
// fractions are quoted against (a measurement aid, not part of the step).
//
//   fp32 v_mfma_f32_16x16x4f32 and v_mfma_f32_32x32x2f32, bf16
//   v_mfma_f32_16x16x32_bf16: every wavefront runs `iters` rounds of its
//   accumulator chains on register operands, 256 threads per workgroup, for
//   several grid sizes; throughput = MFMA flops / event time.
//   HBM: a float4 device-to-device copy of 1 GiB (bytes read + written).
//
// Build and run (not part of the library build):
//   hipcc -O3 -std=c++17 --offload-arch=gfx950 -Xclang -target-feature \
//     -Xclang -packed-fp32-ops -o _build/peaks peaks.hip && _build/peaks
#include <hip/hip_runtime.h>

#include <cstdio>

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

#define CHECK(x)                                                              \
  do {                                                                        \
    hipError_t e_ = (x);                                                      \
    if (e_ != hipSuccess) {                                                   \
      fprintf(stderr, "%s: %s\n", #x, hipGetErrorString(e_));                 \
      return 1;                                                               \
    }                                                                         \
  } while (0)

template <int NACC>
__global__ __launch_bounds__(256) void k_f32_16(int iters, float *out) {
  floatx4 acc[NACC];
  for (int i = 0; i < NACC; ++i) acc[i] = floatx4{0, 0, 0, 0};
  const float a = threadIdx.x * 1e-3f, b = 1.0f + blockIdx.x * 1e-6f;
  for (int it = 0; it < iters; ++it)
#pragma unroll
    for (int i = 0; i < NACC; ++i) acc[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, acc[i], 0, 0, 0);
  float s = 0;
  for (int i = 0; i < NACC; ++i) s += acc[i][0] + acc[i][1] + acc[i][2] + acc[i][3];
  out[blockIdx.x * 256 + threadIdx.x] = s;
}

__global__ __launch_bounds__(256) void k_f32_32(int iters, float *out) {
  floatx16 acc[2];
  for (int i = 0; i < 2; ++i)
    for (int r = 0; r < 16; ++r) acc[i][r] = 0;
  const float a = threadIdx.x * 1e-3f, b = 1.0f + blockIdx.x * 1e-6f;
  for (int it = 0; it < iters; ++it)
#pragma unroll
    for (int i = 0; i < 2; ++i) acc[i] = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, acc[i], 0, 0, 0);
  float s = 0;
  for (int i = 0; i < 2; ++i)
    for (int r = 0; r < 16; ++r) s += acc[i][r];
  out[blockIdx.x * 256 + threadIdx.x] = s;
}

__global__ __launch_bounds__(256) void k_bf16(int iters, float *out) {
  floatx4 acc[4];
  for (int i = 0; i < 4; ++i) acc[i] = floatx4{0, 0, 0, 0};
  bf16x8 a, b;
  for (int i = 0; i < 8; ++i) {
    a[i] = (__bf16)(threadIdx.x * 1e-3f + i);
    b[i] = (__bf16)(1.0f + i * 1e-2f);
  }
  for (int it = 0; it < iters; ++it)
#pragma unroll
    for (int i = 0; i < 4; ++i) acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc[i], 0, 0, 0);
  float s = 0;
  for (int i = 0; i < 4; ++i) s += acc[i][0] + acc[i][1] + acc[i][2] + acc[i][3];
  out[blockIdx.x * 256 + threadIdx.x] = s;
}

__global__ __launch_bounds__(256) void k_copy(const float4 *__restrict__ a, float4 *__restrict__ b, size_t n) {
  for (size_t i = blockIdx.x * size_t(256) + threadIdx.x; i < n; i += size_t(gridDim.x) * 256) b[i] = a[i];
}

// TFLOP/s of one timed launch (after one untimed one)
template <class L>
static double rate(L launch, double flops) {
  hipEvent_t e0, e1;
  if (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess) return -1;
  launch();
  hipEventRecord(e0);
  launch();
  hipEventRecord(e1);
  if (hipEventSynchronize(e1) != hipSuccess) return -1;
  float ms = 0;
  hipEventElapsedTime(&ms, e0, e1);
  hipEventDestroy(e0);
  hipEventDestroy(e1);
  return flops / (ms * 1e-3) / 1e12;
}

int main() {
  constexpr int kMaxBlocks = 2048;
  float *out = nullptr;
  CHECK(hipMalloc(&out, size_t(kMaxBlocks) * 256 * sizeof(float)));
  hipDeviceProp_t p;
  CHECK(hipGetDeviceProperties(&p, 0));
  printf("device: %d compute units, %d MHz, %zu B LDS per workgroup\n", p.multiProcessorCount,
         p.clockRate / 1000, p.sharedMemPerBlock);
  const int it = 20000;
  for (int blocks : {256, 512, 1024, kMaxBlocks}) {
    const double waves = double(blocks) * 4;
    const double f16c1 = rate([&] { hipLaunchKernelGGL(k_f32_16<1>, dim3(blocks), dim3(256), 0, 0, it, out); },
                              waves * it * 1 * 16 * 16 * 4 * 2.0);
    const double f16c4 = rate([&] { hipLaunchKernelGGL(k_f32_16<4>, dim3(blocks), dim3(256), 0, 0, it, out); },
                              waves * it * 4 * 16 * 16 * 4 * 2.0);
    const double f32 = rate([&] { hipLaunchKernelGGL(k_f32_32, dim3(blocks), dim3(256), 0, 0, it, out); },
                            waves * it * 2 * 32 * 32 * 2 * 2.0);
    const double bf = rate([&] { hipLaunchKernelGGL(k_bf16, dim3(blocks), dim3(256), 0, 0, it, out); },
                           waves * it * 4 * 16 * 16 * 32 * 2.0);
    printf("%5d workgroups: fp32 16x16x4 %6.1f TFLOP/s (1 chain), %6.1f (4 chains); fp32 32x32x2 %6.1f; "
           "bf16 16x16x32 %7.1f TFLOP/s\n", blocks, f16c1, f16c4, f32, bf);
  }
  const size_t bytes = size_t(1) << 30, n = bytes / 16;
  float4 *a = nullptr, *b = nullptr;
  CHECK(hipMalloc(&a, bytes));
  CHECK(hipMalloc(&b, bytes));
  CHECK(hipMemset(a, 0, bytes));
  CHECK(hipMemset(b, 0, bytes));
  for (int g : {1024, 4096, 16384}) {
    const double tb = rate([&] { hipLaunchKernelGGL(k_copy, dim3(g), dim3(256), 0, 0, a, b, n); }, 2.0 * bytes);
    printf("copy of 1 GiB, %5d workgroups: %.0f GB/s read + written\n", g, tb * 1e3);
  }
  CHECK(hipDeviceSynchronize());
  CHECK(hipFree(a));
  CHECK(hipFree(b));
  CHECK(hipFree(out));
  return 0;
}
