// Implicit-GEMM convolutions on the bf16 GEMM (gather modes of
// gemm_bf16_kernel.h): forward, data gradient and weight gradient of an R x R
// convolution with stride S in {1, 2} over NHWC bf16 tensors.
#include "common.h"
#include "gemm_bf16_kernel.h"

namespace ckpt {

using namespace gb;

namespace {

int log2_exact(int c) {
  int k = 0;
  while ((1 << k) < c) ++k;
  return (1 << k) == c ? k : -1;
}

// the tap-uniform gathers apply: the gathered channels and the k range per
// workgroup are multiples of the k slice (every slice in one tap, no slice
// past the range), and the tap mask fits 32 bits
bool tap_uniform(const Args &a) {
  return a.cshift >= 0 && (1 << a.cshift) % KS == 0 && a.R * a.R <= 32 && a.K % KS == 0 && a.kper % KS == 0;
}

Args conv_args(const ConvGeo &g, int M, int N, int K, int gathered_c) {
  Args a{};
  a.M = M; a.N = N; a.K = K;
  a.H = g.H; a.W = g.W; a.Ho = g.Ho; a.Wo = g.Wo; a.R = g.R; a.S = g.S; a.P = g.P;
  a.rmagic = (65536 + g.R - 1) / g.R;
  a.cshift = log2_exact(gathered_c);
  a.inv_wo = 1.0f / float(g.Wo);
  a.inv_ho = 1.0f / float(g.Ho);
  a.kper = (K + KS - 1) / KS * KS;
  return a;
}

}  // namespace

bool conv_bf16_supported(const ConvGeo &g) {
  auto ok_c = [](int c) { return c >= 8 && log2_exact(c) >= 0; };
  return ok_c(g.Ci) && ok_c(g.Co) && (g.S == 1 || g.S == 2) && g.R >= 1 && g.R <= 16 && g.P >= 0 &&
         g.Ho == (g.H + 2 * g.P - g.R) / g.S + 1 && g.Wo == (g.W + 2 * g.P - g.R) / g.S + 1;
}

void conv_bf16_fwd(hipStream_t s, const ConvGeo &g, const void *X, const void *Wt, void *Yb,
                   double *stats, const GemmX *act) {
  if (act && act->Rb && (!act->act_st || !act->act_g || !act->act_b || act->Xr))
    fail(CKPT_E_INVALID, "conv_bf16_fwd: the batch-norm apply output needs the statistics, gamma and beta "
                         "(no residual)");
  const int M = g.N * g.Ho * g.Wo, N = g.Co, K = g.R * g.R * g.Ci;
  Args a = conv_args(g, M, N, K, g.Ci);
  a.A = X;
  a.B = static_cast<const __bf16 *>(Wt);
  a.ldb = K;
  a.ldc = N;
  a.Cb = static_cast<__bf16 *>(Yb);
  a.stats = stats;
  if (act && act->Rb) {
    a.Rb = static_cast<__bf16 *>(act->Rb);
    a.ast = act->act_st;
    a.ag = act->act_g;
    a.ab = act->act_b;
  }
  if (tap_uniform(a))
    pick_tile<true, true, __bf16, GA_FWDT, G_DENSE, true>(a, GEMM_EPI_BF16STATS, 1, s);
  else
    pick_tile<true, true, __bf16, GA_FWD, G_DENSE, true>(a, GEMM_EPI_BF16STATS, 1, s);
}

void conv_bf16_dgrad(hipStream_t s, const ConvGeo &g, const void *DY, const void *Wt, float *DX,
                     int epi, const float *D, const void *mask, const void *Cv, const float *bst,
                     double *stats) {
  if (epi == GEMM_EPI_BNBWD && (!mask || !Cv || !bst || !stats))
    fail(CKPT_E_INVALID, "conv_bf16_dgrad: BNBWD needs the mask, input, statistics and partial buffers");
  const int M = g.N * g.H * g.W, N = g.Ci, K = g.R * g.R * g.Co;
  Args a = conv_args(g, M, N, K, g.Co);
  a.A = DY;
  a.B = static_cast<const __bf16 *>(Wt);
  a.C = DX;
  a.ldc = N;
  a.D = D;
  a.ldd = N;
  a.Ym = static_cast<const __bf16 *>(mask);
  a.Cv = static_cast<const __bf16 *>(Cv);
  a.bst = bst;
  a.stats = stats;
  if (g.S == 1 && tap_uniform(a))
    pick_tile<true, false, __bf16, GA_DGRADT, GB_WDGRAD, true>(a, epi, 1, s);
  else
    pick_tile<true, false, __bf16, GA_DGRAD, GB_WDGRAD, true>(a, epi, 1, s);
}

void conv_bf16_wgrad(hipStream_t s, const ConvGeo &g, const void *X, const void *DY, float *part,
                     int splits, float *dW) {
  const int M = g.Co, N = g.R * g.R * g.Ci, K = g.N * g.Ho * g.Wo;
  if (splits < 1) splits = 1;
  Args a = conv_args(g, M, N, K, g.Ci);
  int kper = ((K + splits - 1) / splits + KS - 1) / KS * KS;
  a.kper = kper < KS ? KS : kper;
  a.A = DY;
  a.lda = g.Co;
  a.B = static_cast<const __bf16 *>(X);
  a.C = splits > 1 ? part : dW;
  a.ldc = N;
  pick_tile<false, false, __bf16, G_DENSE, GB_WGRAD, true>(a, GEMM_EPI_STORE, splits, s);
  if (splits > 1) sum_partials(s, part, splits, M * N, dW);
}

}  // namespace ckpt
