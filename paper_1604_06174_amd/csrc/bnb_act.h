// The batch-norm apply of the bf16 bottleneck units, written once for every
// kernel that forms it (the element pass, and the GEMM epilogue that forms it
// on a unit's re-run from the statistics of its first forward), so that all
// of them give the same bits: gamma times (c - mean) * rstd plus beta as one
// fused multiply-add.
#pragma once

#include <hip/hip_runtime.h>

namespace ckpt {

__device__ __forceinline__ float bnb_affine(float c, float mean, float rstd, float gamma, float beta) {
  return __builtin_fmaf(gamma, (c - mean) * rstd, beta);
}

}  // namespace ckpt
