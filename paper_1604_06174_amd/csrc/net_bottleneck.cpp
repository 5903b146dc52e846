// ImageNet-shaped bottleneck ResNet chain in bf16 (NHWC): the deep residual
// network of the paper's section 5.2 built from bottleneck units.
//   unit 0    stem: conv7x7/2 (pad 3) 3 -> C0, BN, ReLU, max pool 3x3/2 (pad 1)
//   units 1.. bottleneck blocks: conv1x1 - BN - ReLU - conv3x3 (stride s) - BN -
//             ReLU - conv1x1 - BN, + shortcut, ReLU.  Stage t has inner width
//             w0 2^t and E w0 2^t output channels; its first block has stride
//             2 (t > 0) and a projection shortcut conv1x1 (stride s) - BN,
//             the others the identity
//   head      global average pool, FC, softmax cross-entropy over the batch
//
// Precision: activations, convolution outputs and the gradients fed to the
// convolutions are bf16; every convolution accumulates in fp32; batch-norm
// statistics are float64 sums of the bf16 values; the gradients between
// units (the gradient slots) and the parameter gradients are fp32.  The bf16
// roundings sit at: the input, each convolution output c, each ReLU output
// r, the block output y, and each batch-norm input gradient dc.
//
// Static layout (B(c, s) = one bf16 [N, s, s, c] tensor, F = fp32, SB = a
// mean/rstd pair, each rounded up to 256 bytes):
//   stem   a = c | r                               q = dr (F) | dc
//   block  a = c1 | r1 | c2 | r2 | c3 | [cp]
//          q = dc3/dc1 | dr2/dr1 (F) | dc2 | [dcp]
//   fixed  every unit's batch-norm statistics (mean | rstd per BN), held for
//          the whole step (the gradient region's fixed buffers)
// With drop_bn_relu (the "drop bn-relu" plan of section 4.2: keep the
// convolution outputs, form batch norm + ReLU again when needed) a block
// keeps a = c1 | c2 | c3 | [cp] and q = r1 | r2 | (the above):
// its forward forms r1 and r2 in the gradient scratch (which no unit uses
// outside its backward), and its backward forms them there again from c1,
// c2 and the statistics with the same kernel, so every value and gradient
// is the standard layout's bit for bit.
// A unit's first forward of the step forms its statistics and its re-runs,
// which see the same input bits, reuse them instead of finalizing the same
// sums again.
// The boundary b_i is the unit's input (b_0 = the bf16 image batch).
#include <algorithm>

#include "kernels.h"
#include "net.h"

namespace ckpt {
namespace {

struct BUnit {
  bool stem;
  int cin, w, cout, stride, hin, hout;
  bool proj;
  int W1, g1, b1, W2 = -1, g2 = -1, b2 = -1, W3 = -1, g3 = -1, b3 = -1, Wp = -1, gp = -1, bp = -1;
};

class Bottleneck : public Net {
 public:
  int N, S, side, C0, K;
  bool drop;  // blocks keep no relu(bn(.)) outputs
  std::vector<BUnit> u;
  int hw, hb;
  // the stem's patch rows: 147 values padded to 160 (16-byte aligned rows, so
  // its product takes the direct loop), its weights padded the same way
  static constexpr int kStemK = 160;
  uint64_t ks_w7 = 0, ks_parg = 0;
  uint64_t ks_wbf = 0, ks_col = 0, ks_stats = 0, ks_bnpart = 0, ks_sums = 0, ks_wpart = 0,
           ks_pooled = 0, ks_dlog = 0, ks_lossn = 0, ks_loss = 0, ks_dpool = 0;
  std::vector<uint64_t> kst_off;  // each unit's batch-norm statistics in the fixed buffers
  uint64_t wpart_floats = 0;

  static uint64_t bf(int64_t m, int c) { return align256(uint64_t(m) * c * 2); }
  static uint64_t f32(int64_t m, int c) { return align256(uint64_t(m) * c * 4); }

  // weight-gradient split-K: about 512 workgroups (two per compute unit),
  // at least 8 k-slices each, partials capped at 16M floats
  static int wsplits(int M, int Nn, int64_t Kd) {
    const int tiles = gemm_bf16_tiles(M, Nn);
    int64_t s = (512 + tiles - 1) / tiles;
    s = std::min<int64_t>(s, Kd / 256);
    s = std::min<int64_t>(s, (int64_t(16) << 20) / (int64_t(M) * Nn));
    return int(std::max<int64_t>(s, 1));
  }

  explicit Bottleneck(const ckpt_net_desc &d) {
    desc = d;
    N = d.batch;
    S = d.image;
    C0 = d.stem_channels;
    K = d.n_classes;
    drop = d.drop_bn_relu != 0;
    side = (S + 2 * 3 - 7) / 2 + 1;
    const int pooled = (side + 2 - 3) / 2 + 1;
    b.push_back(bf(int64_t(N) * S * S, 3));
    {
      BUnit s{true, 3, 0, C0, 2, S, pooled, false, 0, 0, 0};
      s.W1 = add_param("u0.W", uint64_t(C0) * 49 * 3);
      s.g1 = add_param("u0.gamma", C0);
      s.b1 = add_param("u0.beta", C0);
      u.push_back(s);
      const int64_t m = int64_t(N) * side * side;
      a.push_back(2 * bf(m, C0));
      q.push_back(f32(m, C0) + bf(m, C0));
      b.push_back(bf(int64_t(N) * pooled * pooled, C0));
    }
    int cin = C0, h = pooled;
    for (int t = 0; t < d.depth; ++t) {
      const int w = d.width << t, cout = w * d.expansion;
      for (int j = 0; j < d.stage_blocks[t]; ++j) {
        const int stride = (t > 0 && j == 0) ? 2 : 1;
        const int i = int(u.size());
        const std::string p = "u" + std::to_string(i) + ".";
        BUnit k{false, cin, w, cout, stride, h, h / stride, j == 0, 0, 0, 0};
        k.W1 = add_param(p + "W1", uint64_t(w) * cin);
        k.g1 = add_param(p + "gamma1", w);
        k.b1 = add_param(p + "beta1", w);
        k.W2 = add_param(p + "W2", uint64_t(w) * 9 * w);
        k.g2 = add_param(p + "gamma2", w);
        k.b2 = add_param(p + "beta2", w);
        k.W3 = add_param(p + "W3", uint64_t(cout) * w);
        k.g3 = add_param(p + "gamma3", cout);
        k.b3 = add_param(p + "beta3", cout);
        if (k.proj) {
          k.Wp = add_param(p + "Wp", uint64_t(cout) * cin);
          k.gp = add_param(p + "gammap", cout);
          k.bp = add_param(p + "betap", cout);
        }
        u.push_back(k);
        const int64_t mi = int64_t(N) * k.hin * k.hin, mo = int64_t(N) * k.hout * k.hout;
        const uint64_t relus = bf(mi, w) + bf(mo, w);  // r1, r2
        uint64_t av = bf(mi, w) + bf(mo, w) + bf(mo, cout) + (drop ? 0 : relus);
        if (k.proj) av += bf(mo, cout);
        a.push_back(av);
        q.push_back(std::max(bf(mo, cout), bf(mi, w)) + f32(mi, w) + bf(mo, w) +
                    (k.proj ? bf(mo, cout) : 0) + (drop ? relus : 0));
        b.push_back(bf(mo, cout));
        cin = cout;
        h = k.hout;
      }
    }
    hw = add_param("head.W", uint64_t(cin) * K);
    hb = add_param("head.b", uint64_t(K));
    n = int32_t(u.size());
    // gradient slot: the largest fp32 boundary gradient
    for (size_t i = 0; i < u.size(); ++i)
      gslot_bytes = std::max(gslot_bytes, f32(int64_t(N) * u[i].hout * u[i].hout, u[i].cout));

    // operator workspace
    uint64_t stats = 0, bnpart = 0, wpart = 0;
    int jmax = 0;
    auto st_need = [&](int64_t m, int j) {
      stats = std::max<uint64_t>(stats, uint64_t(gemm_bf16_row_blocks(int(m), j)) * 2 * j * 8);
      bnpart = std::max<uint64_t>(bnpart, uint64_t(bnb_partial_blocks(m, j)) * 2 * j * 8);
      // the data-gradient GEMMs that form the batch-norm backward's partials
      bnpart = std::max<uint64_t>(bnpart, uint64_t(gemm_bf16_row_blocks(int(m), j)) * 2 * j * 8);
      jmax = std::max(jmax, j);
    };
    auto wp_need = [&](int M, int Nn, int64_t Kd) {
      const int s = wsplits(M, Nn, Kd);
      if (s > 1) wpart = std::max<uint64_t>(wpart, uint64_t(s) * M * Nn);
    };
    for (const BUnit &k : u) {
      if (k.stem) {
        const int64_t m = int64_t(N) * side * side;
        st_need(m, C0);
        wp_need(C0, 147, m);
        continue;
      }
      const int64_t mi = int64_t(N) * k.hin * k.hin, mo = int64_t(N) * k.hout * k.hout;
      st_need(mi, k.w);
      st_need(mo, k.w);
      st_need(mo, k.cout);
      wp_need(k.w, k.cin, mi);
      wp_need(k.w, 9 * k.w, mo);
      wp_need(k.cout, k.w, mo);
      if (k.proj) wp_need(k.cout, k.cin, mo);
    }
    uint64_t off = 0;
    auto take = [&](uint64_t bytes) {
      uint64_t o = off;
      off += align256(bytes);
      return o;
    };
    ks_wbf = take(param_bytes / 2);
    ks_col = take(uint64_t(N) * side * side * kStemK * 2);
    ks_w7 = take(uint64_t(C0) * kStemK * 2);
    ks_parg = take(uint64_t(N) * u[0].hout * u[0].hout * C0);
    ks_stats = take(stats);
    ks_bnpart = take(bnpart);
    ks_sums = take(8ull * jmax);
    ks_wpart = take(wpart * 4);
    ks_pooled = take(4ull * N * cin);
    ks_dpool = take(4ull * N * cin);
    ks_dlog = take(4ull * N * K);
    ks_lossn = take(4ull * N);
    ks_loss = take(4);
    // every unit's batch-norm statistics (st1 | st2 | st3 [| stp], the stem's
    // st), formed by its first forward of the step and read by its re-runs
    // and its backward: held for the whole step, so they are fixed buffers
    // of the static layout (counted in the peak), not operator workspace
    uint64_t kst = 0;
    for (const BUnit &k : u) {
      kst_off.push_back(kst);
      kst += k.stem ? align256(8ull * C0)
                    : 2 * align256(8ull * k.w) + (k.proj ? 2 : 1) * align256(8ull * k.cout);
    }
    grad_extra = kst;
    ks_bytes = off;
    timed_family = "k_gemm_bf16";
    uses_side = true;
  }

  // bf16 mirror of parameter k (same element offset as in the f32 buffer)
  const void *Wb(const StepCtx &c, int k) const {
    return c.ks + ks_wbf + params[size_t(k)].off / 2;
  }
  double *statsbuf(StepCtx &c) const { return reinterpret_cast<double *>(c.ks + ks_stats); }
  double *bnpart(StepCtx &c) const { return reinterpret_cast<double *>(c.ks + ks_bnpart); }
  // unit i's statistics: st1, st2, st3, stp at 0, S, 2 S, 2 S + align256(8 cout),
  // S = align256(8 w) (the stem's st at 0)
  float *kst(const StepCtx &c, int32_t i, int which) const {
    const BUnit &k = u[size_t(i)];
    const uint64_t o = which == 0   ? 0
                       : which == 1 ? align256(8ull * k.w)
                       : which == 2 ? 2 * align256(8ull * k.w)
                                    : 2 * align256(8ull * k.w) + align256(8ull * k.cout);
    return reinterpret_cast<float *>(c.gextra + kst_off[size_t(i)] + o);
  }
  float *ksf(StepCtx &c, uint64_t o) const { return reinterpret_cast<float *>(c.ks + o); }

  // timed GEMM-family launches: 2 M N K flops; bytes = operands read once +
  // result written once (+ a re-run's batch-norm output, and the shortcut it
  // reads, when the epilogue forms them)
  void tbeg(StepCtx &c) { timer.begin(c.s); }
  static double act_bytes(const GemmX *act, double m, double co) {
    if (!act || !act->Rb) return 0.0;
    return 2.0 * m * co * (act->Xr ? 2.0 : 1.0);
  }
  void tend(StepCtx &c, double M, double Nn, double Kd, double in_b, double out_b) {
    timer.end(c.s, 2.0 * M * Nn * Kd, in_b + out_b);
    c.launches += 1;
  }

  // forward 1x1 convolution (stride 1) with BN statistics, then the stats
  // (not on a re-run, which reuses the unit's kept statistics and forms no
  // sums).  act (a re-run only): the epilogue also writes the BN apply's
  // output, relu(bn(out) [+ residual]).
  void fwd_1x1(StepCtx &c, int64_t m, int ci, int co, const void *x, int wk, void *out, float *st,
               const GemmX *act = nullptr) {
    tbeg(c);
    GemmX gx = act ? *act : GemmX{};
    gx.Cb = out;
    gx.stats = c.rerun ? nullptr : statsbuf(c);
    gemm_bf16x(c.s, int(m), co, ci, x, false, ci, true, Wb(c, wk), ci, true, nullptr, co,
               GEMM_EPI_BF16STATS, nullptr, 0, nullptr, gx);
    tend(c, double(m), co, ci, 2.0 * (double(m) * ci + double(ci) * co),
         2.0 * double(m) * co + act_bytes(act, double(m), co));
    if (!c.rerun) {
      bn_finalize_fwd(c.s, statsbuf(c), gemm_bf16_row_blocks(int(m), co), co, m, st, false);
      c.launches += 1;
    }
  }

  void fwd_conv(StepCtx &c, const ConvGeo &g, const void *x, int wk, void *out, float *st,
                const GemmX *act = nullptr) {
    const int64_t m = int64_t(g.N) * g.Ho * g.Wo;
    const double kd = double(g.R) * g.R * g.Ci;
    tbeg(c);
    conv_bf16_fwd(c.s, g, x, Wb(c, wk), out, c.rerun ? nullptr : statsbuf(c), act);
    tend(c, double(m), g.Co, kd, 2.0 * (double(g.N) * g.H * g.W * g.Ci + kd * g.Co),
         2.0 * double(m) * g.Co + act_bytes(act, double(m), g.Co));
    if (!c.rerun) {
      bn_finalize_fwd(c.s, statsbuf(c), gemm_bf16_row_blocks(int(m), g.Co), g.Co, m, st, false);
      c.launches += 1;
    }
  }

  // dW [M, Nn] = sum over k of A(m, k) B(k, n), A = dY^T ([Kd, M] bf16), B = X ([Kd, Nn] bf16),
  // on stream st (with its split-K partials)
  // (ldx: X's row pitch, Nn when 0)
  void wgrad_1x1(StepCtx &c, hipStream_t st, int M, int Nn, int64_t Kd, const void *dy, const void *x,
                 float *dW, int ldx = 0) {
    const int s = wsplits(M, Nn, Kd);
    GemmX gx;
    gx.splits = s;
    tbeg(c);
    gemm_bf16x(st, M, Nn, int(Kd), dy, false, M, false, x, ldx ? ldx : Nn, false,
               s > 1 ? ksf(c, ks_wpart) : dW, Nn, GEMM_EPI_STORE, nullptr, 0, nullptr, gx);
    tend(c, M, Nn, double(Kd), 2.0 * double(Kd) * (M + Nn), 4.0 * M * Nn);
    if (s > 1) {
      sum_partials(st, ksf(c, ks_wpart), s, M * Nn, dW);
      c.launches += 1;
    }
  }

  void wgrad_conv(StepCtx &c, hipStream_t st, const ConvGeo &g, const void *x, const void *dy, float *dW) {
    const int M = g.Co, Nn = g.R * g.R * g.Ci;
    const int64_t Kd = int64_t(g.N) * g.Ho * g.Wo;
    const int s = wsplits(M, Nn, Kd);
    tbeg(c);
    conv_bf16_wgrad(st, g, x, dy, ksf(c, ks_wpart), s, dW);
    tend(c, M, Nn, double(Kd), 2.0 * (double(g.N) * g.H * g.W * g.Ci + double(Kd) * g.Co),
         4.0 * M * Nn);
    if (s > 1) c.launches += 1;
  }

  void begin_step(StepCtx &c) override {
    cvt_bf16(c.s, int64_t(param_bytes / 4), c.params, c.ks + ks_wbf);
    cvt_pad_rows(c.s, C0, 147, kStemK, P(c, u[0].W1), c.ks + ks_w7);
    c.launches += 2;
  }

  void fwd(int32_t i, const void *xv, void *yv, void *saved, StepCtx &c) override {
    const BUnit &k = u[size_t(i)];
    char *sv = static_cast<char *>(saved);
    // A re-run writes the arena, which the weight gradients a backward left on
    // the side stream may read (a unit's backward does not wait for its own).
    // Only the first unit's conv1 weight gradient may then still be running
    // after the mark set before it: it reads the gradient scratch (which a
    // forward writes only in the drop bn-relu layout) and the unit's input,
    // the segment's kept boundary (which only a recursive plan rewrites
    // during the backward), so otherwise the forward waits for the mark only.
    if (drop || c.recursive) c.to_main();
    else c.main_after_mark2();
    if (k.stem) {
      const int64_t m = int64_t(N) * side * side;
      char *cv = sv, *r = sv + bf(m, C0);
      float *st = kst(c, i, 0);
      im2col7(c.s, N, S, S, side, side, kStemK, xv, c.ks + ks_col);
      tbeg(c);
      GemmX gx;
      gx.Cb = cv;
      gx.stats = c.rerun ? nullptr : statsbuf(c);
      gemm_bf16x(c.s, int(m), C0, kStemK, c.ks + ks_col, false, kStemK, true, c.ks + ks_w7, kStemK, true,
                 nullptr, C0, GEMM_EPI_BF16STATS, nullptr, 0, nullptr, gx);
      tend(c, double(m), C0, 147, 2.0 * (double(m) * 147 + 147.0 * C0), 2.0 * double(m) * C0);
      if (!c.rerun) bn_finalize_fwd(c.s, statsbuf(c), gemm_bf16_row_blocks(int(m), C0), C0, m, st, false);
      bnb_apply(c.s, BNB_RES_NONE, m, C0, cv, st, P(c, k.g1), P(c, k.b1), nullptr, nullptr,
                nullptr, nullptr, r);
      maxpool_fwd(c.s, N, side, side, C0, k.hout, k.hout, r, yv);
      c.launches += c.rerun ? 3 : 4;
      return;
    }
    const int64_t mi = int64_t(N) * k.hin * k.hin, mo = int64_t(N) * k.hout * k.hout;
    char *c1, *r1, *c2, *r2, *c3, *cp;
    if (drop) {  // r1, r2 transient, in the gradient scratch
      c1 = sv, c2 = c1 + bf(mi, k.w), c3 = c2 + bf(mo, k.w), cp = c3 + bf(mo, k.cout);
      r1 = c.q, r2 = r1 + bf(mi, k.w);
    } else {
      c1 = sv, r1 = c1 + bf(mi, k.w), c2 = r1 + bf(mi, k.w), r2 = c2 + bf(mo, k.w);
      c3 = r2 + bf(mo, k.w), cp = c3 + bf(mo, k.cout);
    }
    float *st1 = kst(c, i, 0), *st2 = kst(c, i, 1), *st3 = kst(c, i, 2), *stp = kst(c, i, 3);
    // a re-run knows the unit's statistics: each convolution's epilogue
    // forms its batch norm + ReLU output itself (the identity block's last
    // one with the shortcut), so no element pass runs
    const bool fuse = c.rerun;
    auto act = [&](void *r, int g, int b, const float *st, const void *res) {
      GemmX a;
      a.Rb = r;
      a.Xr = res;
      a.act_st = st;
      a.act_g = P(c, g);
      a.act_b = P(c, b);
      return a;
    };
    const GemmX a1 = act(r1, k.g1, k.b1, st1, nullptr), a2 = act(r2, k.g2, k.b2, st2, nullptr),
                a3 = act(yv, k.g3, k.b3, st3, xv);
    fwd_1x1(c, mi, k.cin, k.w, xv, k.W1, c1, st1, fuse ? &a1 : nullptr);
    if (!fuse) {
      bnb_apply(c.s, BNB_RES_NONE, mi, k.w, c1, st1, P(c, k.g1), P(c, k.b1), nullptr, nullptr,
                nullptr, nullptr, r1);
      c.launches += 1;
    }
    fwd_conv(c, ConvGeo{N, k.hin, k.hin, k.w, k.hout, k.hout, k.w, 3, k.stride, 1}, r1, k.W2, c2, st2,
             fuse ? &a2 : nullptr);
    if (!fuse) {
      bnb_apply(c.s, BNB_RES_NONE, mo, k.w, c2, st2, P(c, k.g2), P(c, k.b2), nullptr, nullptr,
                nullptr, nullptr, r2);
      c.launches += 1;
    }
    fwd_1x1(c, mo, k.w, k.cout, r2, k.W3, c3, st3, fuse && !k.proj ? &a3 : nullptr);
    if (k.proj) {
      if (k.stride == 1)
        fwd_1x1(c, mo, k.cin, k.cout, xv, k.Wp, cp, stp);
      else
        fwd_conv(c, ConvGeo{N, k.hin, k.hin, k.cin, k.hout, k.hout, k.cout, 1, k.stride, 0}, xv,
                 k.Wp, cp, stp);
      bnb_apply(c.s, BNB_RES_BN, mo, k.cout, c3, st3, P(c, k.g3), P(c, k.b3), cp, stp, P(c, k.gp),
                P(c, k.bp), yv);
      c.launches += 1;
    } else if (!fuse) {
      bnb_apply(c.s, BNB_RES_ID, mo, k.cout, c3, st3, P(c, k.g3), P(c, k.b3), xv, nullptr, nullptr,
                nullptr, yv);
      c.launches += 1;
    }
  }

  void bwd(int32_t i, const void *gv, void *dxv, const void *xv, const void *yv, const void *saved,
           void *qv, StepCtx &c) override {
    const BUnit &k = u[size_t(i)];
    const float *g = static_cast<const float *>(gv);
    const char *sv = static_cast<const char *>(saved);
    char *qb = static_cast<char *>(qv);
    float *sums = ksf(c, ks_sums);
    // The weight gradients a unit's backward leaves on the side stream read the
    // gradient scratch and the unit's activations; the next backward waits for
    // them just before it first writes the scratch (so its first batch norm's
    // sums run beside them), a re-run forward at its start, the step at its end.
    if (k.stem) {  // no input gradient
      c.to_main();
      const int64_t m = int64_t(N) * side * side;
      const char *cv = sv, *r = sv + bf(m, C0);
      const float *st = kst(c, i, 0);
      float *dr = reinterpret_cast<float *>(qb);
      char *dc = qb + f32(m, C0);
      maxpool_bwd(c.s, N, side, side, C0, k.hout, k.hout, g, r, yv, dr, c.ks + ks_parg);
      bnb_backward(c.s, m, C0, dr, r, cv, st, P(c, k.g1), bnpart(c), sums, G(c, k.g1), G(c, k.b1), dc);
      im2col7(c.s, N, S, S, side, side, kStemK, xv, c.ks + ks_col);
      c.launches += 6;
      wgrad_1x1(c, c.s, C0, 147, m, dc, c.ks + ks_col, G(c, k.W1), kStemK);
      return;
    }
    const int64_t mi = int64_t(N) * k.hin * k.hin, mo = int64_t(N) * k.hout * k.hout;
    const char *c1, *r1, *c2, *r2, *c3, *cp;
    const float *st1 = kst(c, i, 0), *st2 = kst(c, i, 1), *st3 = kst(c, i, 2), *stp = kst(c, i, 3);
    if (drop) {
      c1 = sv, c2 = c1 + bf(mi, k.w), c3 = c2 + bf(mo, k.w), cp = c3 + bf(mo, k.cout);
      r1 = r2 = nullptr;
    } else {
      c1 = sv, r1 = c1 + bf(mi, k.w), c2 = r1 + bf(mi, k.w), r2 = c2 + bf(mo, k.w);
      c3 = r2 + bf(mo, k.w), cp = c3 + bf(mo, k.cout);
    }
    // third BN (input gradient: g masked by the block's final ReLU): its sums
    // first; everything after writes the gradient scratch, so it waits for the
    // previous unit's weight gradients
    bnb_backward_sums(c.s, mo, k.cout, g, yv, c3, st3, bnpart(c), sums, G(c, k.g3), G(c, k.b3));
    c.to_main();
    if (drop) {
      // r1, r2 formed again from c1, c2 and their statistics (the forward's
      // kernel on the same bits) at the front of the gradient scratch
      char *rr1 = qb, *rr2 = rr1 + bf(mi, k.w);
      bnb_apply(c.s, BNB_RES_NONE, mi, k.w, c1, st1, P(c, k.g1), P(c, k.b1), nullptr, nullptr,
                nullptr, nullptr, rr1);
      bnb_apply(c.s, BNB_RES_NONE, mo, k.w, c2, st2, P(c, k.g2), P(c, k.b2), nullptr, nullptr,
                nullptr, nullptr, rr2);
      c.launches += 2;
      r1 = rr1, r2 = rr2;
      qb = rr2 + bf(mo, k.w);
    }
    // The weight gradients go to c.ws() (the side stream when there is one),
    // each after a to_side that orders it behind the writes of the gradient it
    // reads.  The write of dc1 over dc3 waits for the mark set after conv3's
    // weight gradient; the next unit's backward waits for all of them before it
    // writes the scratch (it reuses the scratch and the split-K partials).
    char *qA = qb;                                         // dc3, then dc1
    float *qB = reinterpret_cast<float *>(qA + std::max(bf(mo, k.cout), bf(mi, k.w)));  // dr2, dr1
    char *qC = reinterpret_cast<char *>(qB) + f32(mi, k.w);  // dc2
    char *qD = qC + bf(mo, k.w);                             // dcp
    bnb_backward_apply(c.s, mo, k.cout, g, yv, c3, st3, P(c, k.g3), sums, qA);
    if (k.proj)
      bnb_backward(c.s, mo, k.cout, g, yv, cp, stp, P(c, k.gp), bnpart(c), sums, G(c, k.gp),
                   G(c, k.bp), qD);
    c.launches += k.proj ? 6 : 3;
    // conv3 (1x1): weight and data gradients (and the projection's weights)
    c.to_side();
    if (k.proj) {
      const ConvGeo gp{N, k.hin, k.hin, k.cin, k.hout, k.hout, k.cout, 1, k.stride, 0};
      if (k.stride == 1)
        wgrad_1x1(c, c.ws(), k.cout, k.cin, mo, qD, xv, G(c, k.Wp));
      else
        wgrad_conv(c, c.ws(), gp, xv, qD, G(c, k.Wp));
    }
    wgrad_1x1(c, c.ws(), k.cout, k.w, mo, qA, r2, G(c, k.W3));
    c.mark_side();
    // its epilogue masks the product by the second ReLU and adds up the second
    // BN's backward sums (partials per row tile of the GEMM)
    tbeg(c);
    {
      GemmX gx;
      gx.mask = r2;
      gx.cv = c2;
      gx.bst = st2;
      gx.stats = bnpart(c);
      gemm_bf16x(c.s, int(mo), k.w, k.cout, qA, false, k.cout, true, Wb(c, k.W3), k.w, false, qB,
                 k.w, GEMM_EPI_BNBWD, nullptr, 0, nullptr, gx);
    }
    tend(c, double(mo), k.w, k.cout,
         2.0 * (double(mo) * k.cout + double(k.cout) * k.w) + 4.0 * double(mo) * k.w,
         4.0 * double(mo) * k.w);
    // second BN: finalize and element pass
    bn_finalize_bwd(c.s, bnpart(c), gemm_bf16_row_blocks(int(mo), k.w), k.w, mo, sums, G(c, k.g2),
                    G(c, k.b2), false);
    bnb_backward_apply(c.s, mo, k.w, qB, nullptr, c2, st2, P(c, k.g2), sums, qC);
    c.launches += 2;
    // conv2 (3x3, stride s)
    const ConvGeo g2{N, k.hin, k.hin, k.w, k.hout, k.hout, k.w, 3, k.stride, 1};
    c.to_side();
    wgrad_conv(c, c.ws(), g2, r1, qC, G(c, k.W2));
    c.mark2_side();  // all side work but conv1's weight gradient
    // with the first ReLU's mask and the first BN's backward sums in its epilogue
    tbeg(c);
    conv_bf16_dgrad(c.s, g2, qC, Wb(c, k.W2), qB, GEMM_EPI_BNBWD, nullptr, r1, c1, st1, bnpart(c));
    tend(c, double(mi), k.w, 9.0 * k.w,
         2.0 * (double(mo) * k.w + 9.0 * k.w * k.w) + 4.0 * double(mi) * k.w,
         4.0 * double(mi) * k.w);
    // first BN: finalize and element pass
    bn_finalize_bwd(c.s, bnpart(c), gemm_bf16_row_blocks(int(mi), k.w), k.w, mi, sums, G(c, k.g1),
                    G(c, k.b1), false);
    c.main_after_mark();  // dc1 overwrites dc3
    bnb_backward_apply(c.s, mi, k.w, qB, nullptr, c1, st1, P(c, k.g1), sums, qA);
    c.launches += 2;
    // conv1 (1x1)
    c.to_side();
    wgrad_1x1(c, c.ws(), k.w, k.cin, mi, qA, xv, G(c, k.W1));
    if (dxv) {
      float *dx = static_cast<float *>(dxv);
      tbeg(c);
      if (k.proj)
        gemm_bf16(c.s, int(mi), k.cin, k.w, qA, false, k.w, true, Wb(c, k.W1), k.cin, false, dx,
                  k.cin, GEMM_EPI_STORE);
      else {  // + the identity shortcut's gradient, g masked by the final ReLU
        GemmX gx;
        gx.mask = yv;
        gemm_bf16x(c.s, int(mi), k.cin, k.w, qA, false, k.w, true, Wb(c, k.W1), k.cin, false, dx,
                   k.cin, GEMM_EPI_ADDMASK, g, k.cin, nullptr, gx);
      }
      // ADDMASK also reads g (fp32) and the mask (bf16) once
      tend(c, double(mi), k.cin, k.w,
           2.0 * (double(mi) * k.w + double(k.w) * k.cin) + (k.proj ? 0.0 : 6.0 * double(mi) * k.cin),
           4.0 * double(mi) * k.cin);
    }
    if (k.proj) {
      const ConvGeo gp{N, k.hin, k.hin, k.cin, k.hout, k.hout, k.cout, 1, k.stride, 0};
      if (dxv) {
        float *dx = static_cast<float *>(dxv);
        tbeg(c);
        if (k.stride == 1)
          gemm_bf16(c.s, int(mi), k.cin, k.cout, qD, false, k.cout, true, Wb(c, k.Wp), k.cin, false,
                    dx, k.cin, GEMM_EPI_ADD, dx, k.cin);
        else
          conv_bf16_dgrad(c.s, gp, qD, Wb(c, k.Wp), dx, GEMM_EPI_ADD, dx);
        tend(c, double(mi), k.cin, k.cout, 2.0 * (double(mo) * k.cout + double(k.cout) * k.cin),
             8.0 * double(mi) * k.cin);
      }
    }
  }

  void head(const void *xn, void *g, StepCtx &c) override {
    const BUnit &k = u.back();
    pool_fc_ce_head_bf16(c.s, N, k.hout * k.hout, k.cout, K, xn, P(c, hw), P(c, hb),
                         static_cast<const int *>(c.target), ksf(c, ks_pooled), ksf(c, ks_dlog),
                         ksf(c, ks_lossn), ksf(c, ks_dpool), static_cast<float *>(g), G(c, hw),
                         G(c, hb), ksf(c, ks_loss));
    c.launches += 6;
  }

  const float *loss_ptr(const StepCtx &c) const override {
    return reinterpret_cast<const float *>(c.ks + ks_loss);
  }
};

bool pow2_in(int v, int lo, int hi) { return v >= lo && v <= hi && (v & (v - 1)) == 0; }

}  // namespace

std::unique_ptr<Net> make_resnet_bottleneck_net(const ckpt_net_desc &d) {
  if (d.batch <= 0 || d.depth <= 0 || d.depth > 4 || d.width <= 0 || d.image <= 0 ||
      d.n_classes <= 0 || d.expansion <= 0 || d.stem_channels <= 0)
    fail(CKPT_E_INVALID,
         "net_create: RESNET_BOTTLENECK needs positive batch, 1-4 stages, width, expansion, "
         "stem channels, image and classes");
  for (int t = 0; t < 4; ++t) {
    if (t < d.depth && d.stage_blocks[t] <= 0)
      fail(CKPT_E_INVALID, "net_create: RESNET_BOTTLENECK stage_blocks must be positive per stage");
    if (t >= d.depth && d.stage_blocks[t] != 0)
      fail(CKPT_E_INVALID, "net_create: RESNET_BOTTLENECK stage_blocks beyond depth must be zero");
  }
  if (!pow2_in(d.stem_channels, 8, 2048) || !pow2_in(d.expansion, 1, 256))
    fail(CKPT_E_UNSUPPORTED, "net_create: RESNET_BOTTLENECK channel counts must be powers of two in [8, 2048]");
  for (int t = 0; t < d.depth; ++t) {
    const int64_t w = int64_t(d.width) << t;
    if (w > 2048 || !pow2_in(int(w), 8, 2048) || w * d.expansion > 2048)
      fail(CKPT_E_UNSUPPORTED, "net_create: RESNET_BOTTLENECK channel counts must be powers of two in [8, 2048]");
  }
  const int side = (d.image + 2 * 3 - 7) / 2 + 1;
  if (d.image < 4 || side < 2)
    fail(CKPT_E_INVALID, "net_create: RESNET_BOTTLENECK image too small");
  int h = (side + 2 - 3) / 2 + 1;
  for (int t = 1; t < d.depth; ++t) {
    if (h % 2 != 0 || h < 2)
      fail(CKPT_E_UNSUPPORTED, "net_create: RESNET_BOTTLENECK stride-2 stages need an even input side");
    h /= 2;
  }
  if (int64_t(d.batch) * side * side >= (int64_t(1) << 24))
    fail(CKPT_E_INVALID, "net_create: RESNET_BOTTLENECK batch x stem pixels must stay below 2^24");
  return std::make_unique<Bottleneck>(d);
}

}  // namespace ckpt
