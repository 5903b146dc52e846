// Achieved HBM bandwidth of the batch-norm element passes at the tensor sizes
// of the step's workloads (a measurement aid, not part of the step).
//
// For each size, 200 back-to-back launches on one stream are timed with HIP
// events; a launch moves its algorithmic bytes (each operand read once, each
// result written once).  Next to every kernel: a device-to-device copy of one
// tensor of the same size, which shows what any single launch reaches at that
// size (the fixed cost of a launch is a large share of a few-megabyte pass).
//   fp32 (CIFAR-shaped net, [N*H*W, C] of 2^21, 2^20, 2^19 elements):
//     bn_apply (relu; + identity residual), bn_backward (3 launches: partial
//     sums, finalize, element pass; with the ReLU mask)
//   bf16 (bottleneck net, batch 32: 56x56x256 .. 7x7x2048 activations):
//     bnb_apply (relu; + identity residual), bnb_backward (3 launches)
#include <hip/hip_runtime.h>

#include <cstdio>
#include <vector>

#include "../csrc/kernels.h"

#define CHECK(x)                                                              \
  do {                                                                        \
    hipError_t e_ = (x);                                                      \
    if (e_ != hipSuccess) {                                                   \
      fprintf(stderr, "%s: %s\n", #x, hipGetErrorString(e_));                 \
      return 1;                                                               \
    }                                                                         \
  } while (0)

namespace {

constexpr int REPS = 200;
constexpr double HBM_PEAK_GBS = 8000.0;

struct Timer {
  hipEvent_t a, b;
  hipStream_t s;
};

template <class F>
double time_us(Timer &t, F f) {
  for (int i = 0; i < 10; ++i) f();
  if (hipEventRecord(t.a, t.s) != hipSuccess) return -1;
  for (int i = 0; i < REPS; ++i) f();
  if (hipEventRecord(t.b, t.s) != hipSuccess || hipEventSynchronize(t.b) != hipSuccess) return -1;
  float ms = 0;
  if (hipEventElapsedTime(&ms, t.a, t.b) != hipSuccess) return -1;
  return ms * 1e3 / REPS;
}

void row(const char *what, double bytes, double us, double copy_gbs) {
  const double gbs = bytes / (us * 1e-6) / 1e9;
  printf("  %-34s %8.2f us  %7.1f GB/s  %5.1f%% of 8 TB/s  %5.1f%% of same-size copy\n", what, us, gbs,
         100.0 * gbs / HBM_PEAK_GBS, 100.0 * gbs / copy_gbs);
}

}  // namespace

int main() {
  hipStream_t s;
  CHECK(hipStreamCreate(&s));
  Timer t{nullptr, nullptr, s};
  CHECK(hipEventCreate(&t.a));
  CHECK(hipEventCreate(&t.b));
  hipDeviceProp_t prop;
  CHECK(hipGetDeviceProperties(&prop, 0));
  printf("device: %s, %d compute units\n", prop.gcnArchName, prop.multiProcessorCount);

  // largest tensor: 32*56*56*256 bf16 or 2^21 fp32 elements; every buffer is
  // sized for the largest case of its kind
  const size_t max_el = size_t(32) * 56 * 56 * 256;
  std::vector<void *> bufs;
  auto dev = [&](size_t bytes) -> void * {
    void *p = nullptr;
    if (hipMalloc(&p, bytes) != hipSuccess) return nullptr;
    bufs.push_back(p);
    (void)hipMemset(p, 0, bytes);
    return p;
  };
  float *A = static_cast<float *>(dev(max_el * 4)), *B = static_cast<float *>(dev(max_el * 4));
  float *Cc = static_cast<float *>(dev(max_el * 4)), *D = static_cast<float *>(dev(max_el * 4));
  const int maxJ = 2048;
  float *st = static_cast<float *>(dev(2 * maxJ * 4)), *gam = static_cast<float *>(dev(maxJ * 4));
  float *bet = static_cast<float *>(dev(maxJ * 4)), *sums = static_cast<float *>(dev(2 * maxJ * 4));
  float *dg = static_cast<float *>(dev(maxJ * 4)), *db = static_cast<float *>(dev(maxJ * 4));
  double *part = static_cast<double *>(dev(size_t(1024) * 2 * maxJ * 8));
  for (void *p : bufs)
    if (!p) {
      fprintf(stderr, "allocation failed\n");
      return 1;
    }
  {  // statistics: mean 0, rstd 1, gamma 1, beta 0
    std::vector<float> h(2 * maxJ, 0.f);
    for (int j = 0; j < maxJ; ++j) h[maxJ + j] = 1.f;
    CHECK(hipMemcpy(st, h.data(), 2 * maxJ * 4, hipMemcpyHostToDevice));
    std::vector<float> one(maxJ, 1.f);
    CHECK(hipMemcpy(gam, one.data(), maxJ * 4, hipMemcpyHostToDevice));
  }

  struct Shape {
    const char *name;
    int64_t P;
    int J;
  };
  printf("fp32 batch norm, CIFAR-shaped net (batch 128):\n");
  for (Shape sh : {Shape{"32x32x16", 128 * 32 * 32, 16}, Shape{"16x16x32", 128 * 16 * 16, 32},
                   Shape{"8x8x64", 128 * 8 * 8, 64}}) {
    const double el = double(sh.P) * sh.J;
    if (el > double(max_el) || sh.J > maxJ || ckpt::bn_partial_blocks(sh.P, sh.J) > 1024) return 1;
    printf(" %s (%.1f MB per tensor)\n", sh.name, el * 4 / 1e6);
    const double cu = time_us(t, [&] { (void)hipMemcpyAsync(B, A, size_t(el) * 4, hipMemcpyDeviceToDevice, s); });
    const double copy_gbs = 2 * el * 4 / (cu * 1e-6) / 1e9;
    printf("  %-34s %8.2f us  %7.1f GB/s\n", "device copy (read + write)", cu, copy_gbs);
    row("bn_apply, relu", 2 * el * 4,
        time_us(t, [&] { ckpt::bn_apply(s, ckpt::BN_RES_NONE, sh.P, sh.J, A, st, gam, bet, nullptr, 0, 0, 0, B); }),
        copy_gbs);
    row("bn_apply, + identity, relu", 3 * el * 4,
        time_us(t, [&] { ckpt::bn_apply(s, ckpt::BN_RES_ID, sh.P, sh.J, A, st, gam, bet, Cc, 0, 0, 0, B); }),
        copy_gbs);
    // partial sums read G, Ym, Cv; the element pass reads them again and writes D
    row("bn_backward, masked (3 launches)", 7 * el * 4,
        time_us(t, [&] { ckpt::bn_backward(s, sh.P, sh.J, A, B, Cc, st, gam, part, sums, dg, db, D); }),
        copy_gbs);
  }
  printf("bf16 batch norm, bottleneck net (batch 32):\n");
  for (Shape sh : {Shape{"56x56x256", 32 * 56 * 56, 256}, Shape{"28x28x512", 32 * 28 * 28, 512},
                   Shape{"14x14x1024", 32 * 14 * 14, 1024}, Shape{"7x7x2048", 32 * 7 * 7, 2048}}) {
    const double el = double(sh.P) * sh.J;
    if (el > double(max_el) || sh.J > maxJ || ckpt::bnb_partial_blocks(sh.P, sh.J) > 1024) return 1;
    printf(" %s (%.1f MB per bf16 tensor)\n", sh.name, el * 2 / 1e6);
    const double cu = time_us(t, [&] { (void)hipMemcpyAsync(B, A, size_t(el) * 2, hipMemcpyDeviceToDevice, s); });
    const double copy_gbs = 2 * el * 2 / (cu * 1e-6) / 1e9;
    printf("  %-34s %8.2f us  %7.1f GB/s\n", "device copy (read + write)", cu, copy_gbs);
    row("bnb_apply, relu", 2 * el * 2,
        time_us(t, [&] { ckpt::bnb_apply(s, ckpt::BNB_RES_NONE, sh.P, sh.J, A, st, gam, bet, nullptr, nullptr, nullptr, nullptr, B); }),
        copy_gbs);
    row("bnb_apply, + identity, relu", 3 * el * 2,
        time_us(t, [&] { ckpt::bnb_apply(s, ckpt::BNB_RES_ID, sh.P, sh.J, A, st, gam, bet, Cc, nullptr, nullptr, nullptr, B); }),
        copy_gbs);
    // fp32 G (4 B), bf16 Ym and Cv (2 B each) read twice; bf16 D written
    row("bnb_backward, masked (3 launches)", el * (2 * (4 + 2 + 2) + 2),
        time_us(t, [&] { ckpt::bnb_backward(s, sh.P, sh.J, A, B, Cc, st, gam, part, sums, dg, db, D); }),
        copy_gbs);
  }
  CHECK(hipStreamSynchronize(s));
  CHECK(hipGetLastError());
  for (void *p : bufs) (void)hipFree(p);
  printf("done\n");
  return 0;
}
