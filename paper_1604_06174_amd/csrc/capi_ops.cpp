// extern "C" operator calls: the single kernels the bf16 bottleneck units are
// built from, each behind its own validated entry point (declared in
// include/ckpt.h, "operator calls").  They run exactly the launchers the
// training step runs, so a caller can check one operator on inputs of its
// choice.  Every argument is validated before anything is launched.
#include <hip/hip_runtime.h>

#include <string>

#include "kernels.h"
#include "net.h"

static_assert(CKPT_EPI_STORE == ckpt::GEMM_EPI_STORE && CKPT_EPI_ADD == ckpt::GEMM_EPI_ADD &&
                  CKPT_EPI_BF16STATS == ckpt::GEMM_EPI_BF16STATS &&
                  CKPT_EPI_ADDMASK == ckpt::GEMM_EPI_ADDMASK && CKPT_EPI_BNBWD == ckpt::GEMM_EPI_BNBWD,
              "epilogue codes of the C ABI and the kernels agree");
static_assert(CKPT_BNB_RES_NONE == ckpt::BNB_RES_NONE && CKPT_BNB_RES_ID == ckpt::BNB_RES_ID &&
                  CKPT_BNB_RES_BN == ckpt::BNB_RES_BN,
              "shortcut codes of the C ABI and the kernels agree");

namespace {

template <class F>
int guarded_op(F &&f) {
  try {
    f();
    ckpt::set_last_error("");
    return CKPT_OK;
  } catch (const ckpt::Error &e) {
    ckpt::set_last_error(e.msg);
    return e.code;
  } catch (const std::exception &e) {
    ckpt::set_last_error(e.what());
    return CKPT_E_INVALID;
  }
}

void need(const void *p, const std::string &what) {
  if (!p) ckpt::fail(CKPT_E_INVALID, what + ": null pointer");
}

bool pow2_at_least8(int64_t c) { return c >= 8 && (c & (c - 1)) == 0; }

void launched(const char *fn) {
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) ckpt::fail(CKPT_E_HIP, std::string(fn) + ": " + hipGetErrorString(e));
}

ckpt::ConvGeo geo_of(const ckpt_conv_geo *g, const char *fn) {
  need(g, std::string(fn) + "(geo)");
  const ckpt::ConvGeo c{g->n, g->h, g->w, g->ci, g->ho, g->wo, g->co, g->r, g->s, g->p};
  if (c.N <= 0 || c.H <= 0 || c.W <= 0 || c.Ho <= 0 || c.Wo <= 0)
    ckpt::fail(CKPT_E_INVALID, std::string(fn) + ": sizes must be positive");
  if (!ckpt::conv_bf16_supported(c))
    ckpt::fail(CKPT_E_UNSUPPORTED, std::string(fn) +
                                       ": channels must be powers of two >= 8, stride 1 or 2, "
                                       "1 <= r <= 16, and ho/wo must follow from h, w, r, s, p");
  if (int64_t(c.N) * c.H * c.W >= (int64_t(1) << 24) || int64_t(c.N) * c.Ho * c.Wo >= (int64_t(1) << 24))
    ckpt::fail(CKPT_E_UNSUPPORTED, std::string(fn) + ": n*h*w must stay below 2^24");
  return c;
}

}  // namespace

extern "C" {

int op_gemm_bf16_blocks(int32_t m, int32_t n, int32_t *row_blocks, int32_t *col_blocks) {
  return guarded_op([&] {
    if (m <= 0 || n <= 0) ckpt::fail(CKPT_E_INVALID, "op_gemm_bf16_blocks: m and n must be positive");
    if (row_blocks) *row_blocks = ckpt::gemm_bf16_row_blocks(m, n);
    if (col_blocks) *col_blocks = ckpt::gemm_bf16_col_blocks(m, n);
  });
}

int op_gemm_bf16(int32_t m, int32_t n, int32_t k, const void *a, int32_t a_fp32, int32_t lda,
                 int32_t ak, const void *b, int32_t ldb, int32_t bk, float *c, int32_t ldc,
                 int32_t epi, const float *d, int32_t ldd, const float *bias, int32_t splits,
                 const void *mask, void *cb, double *stats, const void *cv, const float *bst,
                 void *stream) {
  return guarded_op([&] {
    if (m <= 0 || n <= 0 || k <= 0 || splits < 1)
      ckpt::fail(CKPT_E_INVALID, "op_gemm_bf16: m, n, k and splits must be positive");
    need(a, "op_gemm_bf16(a)");
    need(b, "op_gemm_bf16(b)");
    if (lda < (ak ? k : m) || ldb < (bk ? k : n) || ldc < n)
      ckpt::fail(CKPT_E_INVALID, "op_gemm_bf16: a leading dimension is smaller than its row");
    if (epi != CKPT_EPI_STORE && epi != CKPT_EPI_ADD && epi != CKPT_EPI_ADDMASK &&
        epi != CKPT_EPI_BF16STATS && epi != CKPT_EPI_BNBWD)
      ckpt::fail(CKPT_E_INVALID, "op_gemm_bf16: unknown epilogue");
    if (splits > 1 && epi != CKPT_EPI_STORE)
      ckpt::fail(CKPT_E_INVALID, "op_gemm_bf16: split-K products take the STORE epilogue");
    if (a_fp32 && epi != CKPT_EPI_STORE && epi != CKPT_EPI_ADD)
      ckpt::fail(CKPT_E_INVALID, "op_gemm_bf16: an fp32 A takes the STORE or ADD epilogue");
    if (epi == CKPT_EPI_BF16STATS) {
      need(cb, "op_gemm_bf16(cb)");
      need(stats, "op_gemm_bf16(stats)");
    } else {
      need(c, "op_gemm_bf16(c)");
    }
    if (epi == CKPT_EPI_ADD || epi == CKPT_EPI_ADDMASK) {
      need(d, "op_gemm_bf16(d)");
      if (ldd < n) ckpt::fail(CKPT_E_INVALID, "op_gemm_bf16: ldd is smaller than n");
    }
    if (epi == CKPT_EPI_ADDMASK) need(mask, "op_gemm_bf16(mask)");
    ckpt::GemmX x;
    x.splits = splits;
    x.mask = mask;
    x.Cb = cb;
    x.stats = stats;
    x.cv = cv;
    x.bst = bst;
    ckpt::gemm_bf16x(static_cast<hipStream_t>(stream), m, n, k, a, a_fp32 != 0, lda, ak != 0, b, ldb,
                     bk != 0, c, ldc, epi, d, ldd, bias, x);
    launched("op_gemm_bf16");
  });
}

int op_sum_partials(const float *part, int32_t nb, int64_t count, float *out, void *stream) {
  return guarded_op([&] {
    need(part, "op_sum_partials(part)");
    need(out, "op_sum_partials(out)");
    if (nb < 1 || count <= 0 || count >= (int64_t(1) << 31))
      ckpt::fail(CKPT_E_INVALID, "op_sum_partials: nb >= 1 and 0 < count < 2^31");
    ckpt::sum_partials(static_cast<hipStream_t>(stream), part, nb, int(count), out);
    launched("op_sum_partials");
  });
}

int op_conv_bf16_fwd(const ckpt_conv_geo *geo, const void *x, const void *w, void *y, double *stats,
                     void *stream) {
  return guarded_op([&] {
    const ckpt::ConvGeo g = geo_of(geo, "op_conv_bf16_fwd");
    need(x, "op_conv_bf16_fwd(x)");
    need(w, "op_conv_bf16_fwd(w)");
    need(y, "op_conv_bf16_fwd(y)");
    need(stats, "op_conv_bf16_fwd(stats)");
    ckpt::conv_bf16_fwd(static_cast<hipStream_t>(stream), g, x, w, y, stats);
    launched("op_conv_bf16_fwd");
  });
}

int op_conv_bf16_dgrad(const ckpt_conv_geo *geo, const void *dy, const void *w, float *dx, int32_t epi,
                       const float *d, const void *mask, const void *cv, const float *bst,
                       double *stats, void *stream) {
  return guarded_op([&] {
    const ckpt::ConvGeo g = geo_of(geo, "op_conv_bf16_dgrad");
    need(dy, "op_conv_bf16_dgrad(dy)");
    need(w, "op_conv_bf16_dgrad(w)");
    need(dx, "op_conv_bf16_dgrad(dx)");
    if (epi != CKPT_EPI_STORE && epi != CKPT_EPI_ADD && epi != CKPT_EPI_ADDMASK && epi != CKPT_EPI_BNBWD)
      ckpt::fail(CKPT_E_INVALID, "op_conv_bf16_dgrad: epilogue must be STORE, ADD, ADDMASK or BNBWD");
    if (epi == CKPT_EPI_ADD || epi == CKPT_EPI_ADDMASK) need(d, "op_conv_bf16_dgrad(d)");
    if (epi == CKPT_EPI_ADDMASK || epi == CKPT_EPI_BNBWD) need(mask, "op_conv_bf16_dgrad(mask)");
    if (epi == CKPT_EPI_BNBWD) {
      need(cv, "op_conv_bf16_dgrad(cv)");
      need(bst, "op_conv_bf16_dgrad(bst)");
      need(stats, "op_conv_bf16_dgrad(stats)");
    }
    ckpt::conv_bf16_dgrad(static_cast<hipStream_t>(stream), g, dy, w, dx, epi, d, mask, cv, bst, stats);
    launched("op_conv_bf16_dgrad");
  });
}

int op_conv_bf16_wgrad(const ckpt_conv_geo *geo, const void *x, const void *dy, float *part,
                       int32_t splits, float *dw, void *stream) {
  return guarded_op([&] {
    const ckpt::ConvGeo g = geo_of(geo, "op_conv_bf16_wgrad");
    need(x, "op_conv_bf16_wgrad(x)");
    need(dy, "op_conv_bf16_wgrad(dy)");
    need(dw, "op_conv_bf16_wgrad(dw)");
    if (splits < 1) ckpt::fail(CKPT_E_INVALID, "op_conv_bf16_wgrad: splits must be positive");
    if (splits > 1) need(part, "op_conv_bf16_wgrad(part)");
    if (int64_t(g.Co) * g.R * g.R * g.Ci >= (int64_t(1) << 31) / splits)
      ckpt::fail(CKPT_E_UNSUPPORTED, "op_conv_bf16_wgrad: partials exceed 2^31 floats");
    ckpt::conv_bf16_wgrad(static_cast<hipStream_t>(stream), g, x, dy, part, splits, dw);
    launched("op_conv_bf16_wgrad");
  });
}

int op_bn_finalize(int32_t backward, const double *part, int32_t nb, int32_t j, int64_t m, float *out,
                   float *dgamma, float *dbeta, int32_t channel_major, void *stream) {
  return guarded_op([&] {
    need(part, "op_bn_finalize(part)");
    need(out, "op_bn_finalize(out)");
    if (nb < 1 || j < 1 || m < 1) ckpt::fail(CKPT_E_INVALID, "op_bn_finalize: nb, j and m must be positive");
    if (backward) {
      need(dgamma, "op_bn_finalize(dgamma)");
      need(dbeta, "op_bn_finalize(dbeta)");
      ckpt::bn_finalize_bwd(static_cast<hipStream_t>(stream), part, nb, j, m, out, dgamma, dbeta,
                            channel_major != 0);
    } else {
      ckpt::bn_finalize_fwd(static_cast<hipStream_t>(stream), part, nb, j, m, out, channel_major != 0);
    }
    launched("op_bn_finalize");
  });
}

int op_bnb_partial_blocks(int64_t p, int32_t j, int32_t *nb) {
  return guarded_op([&] {
    need(nb, "op_bnb_partial_blocks(nb)");
    if (p < 1 || !pow2_at_least8(j)) ckpt::fail(CKPT_E_INVALID, "op_bnb_partial_blocks: p >= 1, j a power of two >= 8");
    *nb = ckpt::bnb_partial_blocks(p, j);
  });
}

int op_bnb_apply(int32_t res, int64_t p, int32_t j, const void *c, const float *st, const float *gamma,
                 const float *beta, const void *x, const float *stp, const float *gp, const float *bp,
                 void *y, void *stream) {
  return guarded_op([&] {
    if (p < 1 || !pow2_at_least8(j)) ckpt::fail(CKPT_E_INVALID, "op_bnb_apply: p >= 1, j a power of two >= 8");
    need(c, "op_bnb_apply(c)");
    need(st, "op_bnb_apply(st)");
    need(gamma, "op_bnb_apply(gamma)");
    need(beta, "op_bnb_apply(beta)");
    need(y, "op_bnb_apply(y)");
    if (res != CKPT_BNB_RES_NONE && res != CKPT_BNB_RES_ID && res != CKPT_BNB_RES_BN)
      ckpt::fail(CKPT_E_INVALID, "op_bnb_apply: unknown shortcut kind");
    if (res != CKPT_BNB_RES_NONE) need(x, "op_bnb_apply(x)");
    if (res == CKPT_BNB_RES_BN) {
      need(stp, "op_bnb_apply(stp)");
      need(gp, "op_bnb_apply(gp)");
      need(bp, "op_bnb_apply(bp)");
    }
    ckpt::bnb_apply(static_cast<hipStream_t>(stream), res, p, j, c, st, gamma, beta, x, stp, gp, bp, y);
    launched("op_bnb_apply");
  });
}

int op_bnb_backward(int64_t p, int32_t j, const float *g, const void *ym, const void *c, const float *st,
                    const float *gamma, double *part, float *sums, float *dgamma, float *dbeta, void *d,
                    void *stream) {
  return guarded_op([&] {
    if (p < 1 || p >= (int64_t(1) << 31) || !pow2_at_least8(j))
      ckpt::fail(CKPT_E_INVALID, "op_bnb_backward: 1 <= p < 2^31, j a power of two >= 8");
    need(g, "op_bnb_backward(g)");
    need(c, "op_bnb_backward(c)");
    need(st, "op_bnb_backward(st)");
    need(gamma, "op_bnb_backward(gamma)");
    need(part, "op_bnb_backward(part)");
    need(sums, "op_bnb_backward(sums)");
    need(dgamma, "op_bnb_backward(dgamma)");
    need(dbeta, "op_bnb_backward(dbeta)");
    need(d, "op_bnb_backward(d)");
    ckpt::bnb_backward(static_cast<hipStream_t>(stream), p, j, g, ym, c, st, gamma, part, sums, dgamma,
                       dbeta, d);
    launched("op_bnb_backward");
  });
}

int op_bnb_backward_apply(int64_t p, int32_t j, const float *g, const void *ym, const void *c,
                          const float *st, const float *gamma, const float *sums, void *d,
                          void *stream) {
  return guarded_op([&] {
    if (p < 1 || !pow2_at_least8(j))
      ckpt::fail(CKPT_E_INVALID, "op_bnb_backward_apply: p >= 1, j a power of two >= 8");
    need(g, "op_bnb_backward_apply(g)");
    need(c, "op_bnb_backward_apply(c)");
    need(st, "op_bnb_backward_apply(st)");
    need(gamma, "op_bnb_backward_apply(gamma)");
    need(sums, "op_bnb_backward_apply(sums)");
    need(d, "op_bnb_backward_apply(d)");
    ckpt::bnb_backward_apply(static_cast<hipStream_t>(stream), p, j, g, ym, c, st, gamma, sums, d);
    launched("op_bnb_backward_apply");
  });
}

int op_im2col7(int32_t n, int32_t h, int32_t w, int32_t ho, int32_t wo, int32_t kp, const void *x,
               void *col, void *stream) {
  return guarded_op([&] {
    need(x, "op_im2col7(x)");
    need(col, "op_im2col7(col)");
    if (n < 1 || h < 1 || w < 1 || ho != (h + 6 - 7) / 2 + 1 || wo != (w + 6 - 7) / 2 + 1)
      ckpt::fail(CKPT_E_INVALID, "op_im2col7: positive sizes, ho/wo of a 7x7 stride-2 pad-3 window");
    if (kp != 147 && (kp < 147 || kp % 8 != 0))
      ckpt::fail(CKPT_E_INVALID, "op_im2col7: kp = 147 or a multiple of 8 above it");
    ckpt::im2col7(static_cast<hipStream_t>(stream), n, h, w, ho, wo, kp, x, col);
    launched("op_im2col7");
  });
}

int op_maxpool(int32_t backward, int32_t n, int32_t h, int32_t w, int32_t c, int32_t ho, int32_t wo,
               const float *g, const void *r, const void *y, void *out, void *arg, void *stream) {
  return guarded_op([&] {
    need(r, "op_maxpool(r)");
    need(out, "op_maxpool(out)");
    if (n < 1 || h < 1 || w < 1 || !pow2_at_least8(c) || ho != (h + 2 - 3) / 2 + 1 ||
        wo != (w + 2 - 3) / 2 + 1)
      ckpt::fail(CKPT_E_INVALID,
                 "op_maxpool: positive sizes, c a power of two >= 8, ho/wo of a 3x3 stride-2 pad-1 window");
    if (backward) {
      need(g, "op_maxpool(g)");
      need(y, "op_maxpool(y)");
      ckpt::maxpool_bwd(static_cast<hipStream_t>(stream), n, h, w, c, ho, wo, g, r, y,
                        static_cast<float *>(out), arg);
    } else {
      ckpt::maxpool_fwd(static_cast<hipStream_t>(stream), n, h, w, c, ho, wo, r, out);
    }
    launched("op_maxpool");
  });
}

}  // extern "C"
