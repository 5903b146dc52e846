// CIFAR-shaped residual CNN chain (fp32, NHWC).
//   unit 0      stem: conv3x3 3 -> C0, BN, ReLU
//   units 1..   basic blocks: conv3x3(stride s) - BN - ReLU - conv3x3 - BN,
//               + shortcut (identity, or option A: subsample by 2 and append
//               zero channels), ReLU; three stages of C0, 2 C0, 4 C0 channels,
//               the first block of stages 2 and 3 has stride 2
//   head        global average pool, FC, softmax cross-entropy over the batch
// This is the convolution / batch-norm / activation pipeline of the paper's
// section 4.2 arranged as a residual network (section 5.2).
//
// Static layout per unit (T = one [N, Ho, Ho, Cout] f32 tensor, SB = a BN
// mean/rstd pair of Cout floats each, both rounded up to 256 bytes):
//   stem   a = c                 q = dc
//   block  a = c1 | r1 | c2      q = two T buffers
//   fixed  every unit's SBs, held for the whole step (the gradient region's
//          fixed buffers, counted in the peak)
// The second convolution reads c1 and forms r1 = relu(bn1(c1)) as it loads
// it; when r1 is kept it stores r1 as well (no separate batch-norm pass).
// With drop_bn_relu the blocks keep only the convolution outputs, a = c1 | c2,
// and r1 is formed on the fly from c1 and its statistics
// wherever it is read (the second convolution's input, its data gradient's
// ReLU mask and its weight gradient's input): the "drop bn-relu" memory plan
// the paper applies to the conv-BN-activation pipeline (section 4.2), with the
// same bits as the stored r1.
// A unit's first forward of the step forms its statistics and its re-runs,
// which see the same input bits, reuse them instead of finalizing the same
// sums again.
// The boundary b_i is the unit's input tensor (b_0 = the image batch).
#include <algorithm>

#include "kernels.h"
#include "net.h"

namespace ckpt {
namespace {

struct Blk {
  int cin, cout, stride, hin, hout;
  int w1, g1, b1, w2, g2, b2;  // parameter indices (stem: w1, g1, b1)
};

class ResNetBasic : public Net {
 public:
  int N, S, C0, K, nb;
  bool drop;  // r1 recomputed from c1 instead of kept
  std::vector<Blk> u;
  int hw, hb;  // head parameter indices
  // operator workspace offsets (bytes)
  uint64_t ks_loss = 0, ks_bnpart = 0, ks_sums = 0, ks_wpart = 0, ks_pooled = 0, ks_dlog = 0,
           ks_lossn = 0, ks_nst = 0, ks_fcpart = 0;
  std::vector<uint64_t> kst_off;  // each unit's batch-norm statistics in the fixed buffers

  // ---- the network at operator granularity (node-level graph) ----
  enum { ND_DATA, ND_CONV, ND_BN, ND_RELU, ND_ADD, ND_SHORT, ND_POOL, ND_FC, ND_LOSS };
  struct GNode {
    int op;
    std::vector<int32_t> in;
    uint64_t bytes;
    int h, c;                 // output side and channels (POOL: c features; FC, LOSS: classes)
    int hin, cin, stride;     // CONV, SHORT, POOL, FC: input side, channels, stride
    int w = -1, g = -1, bt = -1;  // parameters (CONV: w; BN: g, bt)
    uint64_t st = 0;          // BN: its statistics' offset in the operator workspace
  };
  std::vector<GNode> gn;
  uint64_t nst_bytes = 0;

  explicit ResNetBasic(const ckpt_net_desc &d) {
    desc = d;
    N = d.batch;
    S = d.image;
    C0 = d.width;
    K = d.n_classes;
    nb = d.depth;
    drop = d.drop_bn_relu != 0;
    auto T = [&](int h, int c) { return align256(uint64_t(N) * h * h * c * 4); };
    b.push_back(align256(uint64_t(N) * S * S * 3 * 4));
    {
      Blk s{3, C0, 1, S, S, 0, 0, 0, -1, -1, -1};
      s.w1 = add_param("u0.W", uint64_t(C0) * 9 * 3);
      s.g1 = add_param("u0.gamma", C0);
      s.b1 = add_param("u0.beta", C0);
      u.push_back(s);
      a.push_back(T(S, C0));
      q.push_back(T(S, C0));
      b.push_back(T(S, C0));
    }
    int cin = C0, side = S;
    for (int st = 0; st < 3; ++st) {
      const int cout = C0 << st;
      for (int j = 0; j < nb; ++j) {
        const int stride = (st > 0 && j == 0) ? 2 : 1;
        const int i = int(u.size());
        const std::string p = "u" + std::to_string(i) + ".";
        Blk k{cin, cout, stride, side, side / stride, 0, 0, 0, 0, 0, 0};
        k.w1 = add_param(p + "W1", uint64_t(cout) * 9 * cin);
        k.g1 = add_param(p + "gamma1", cout);
        k.b1 = add_param(p + "beta1", cout);
        k.w2 = add_param(p + "W2", uint64_t(cout) * 9 * cout);
        k.g2 = add_param(p + "gamma2", cout);
        k.b2 = add_param(p + "beta2", cout);
        u.push_back(k);
        const uint64_t t = T(k.hout, cout);
        a.push_back((drop ? 2 : 3) * t);
        q.push_back(2 * t);
        b.push_back(t);
        cin = cout;
        side = k.hout;
      }
    }
    hw = add_param("head.W", uint64_t(cin) * K);
    hb = add_param("head.b", uint64_t(K));
    n = int32_t(u.size());
    build_nodes();

    // operator workspace: the largest partial-sum buffers any unit needs
    uint64_t bnpart = 0, wpart = 0;
    for (const Blk &k : u) {
      const int64_t np = int64_t(N) * k.hout * k.hout;
      const int conv_in[2] = {k.cin, k.cout};
      const int conv_s[2] = {k.stride, 1};
      for (int c = 0; c < (k.w2 >= 0 ? 2 : 1); ++c) {
        bnpart = std::max<uint64_t>(
            bnpart, uint64_t(conv3x3_blocks(CONV_FWD, conv_s[c], N, k.hout, k.hout, conv_in[c], k.cout)) *
                        2 * k.cout * 8);
        wpart = std::max<uint64_t>(
            wpart, uint64_t(conv3x3_wgrad_blocks(conv_s[c], N, k.hout, k.hout, conv_in[c], k.cout)) *
                       k.cout * 9 * conv_in[c] * 4);
      }
      bnpart = std::max<uint64_t>(bnpart, uint64_t(bn_partial_blocks(np, k.cout)) * 2 * k.cout * 8);
      if (k.w2 >= 0)  // the second convolution's data gradient sums the first BN's backward
        bnpart = std::max<uint64_t>(
            bnpart, uint64_t(conv3x3_blocks(CONV_DGRAD, 1, N, k.hout, k.hout, k.cout, k.cout)) * 2 *
                        k.cout * 8);
    }
    const int CL = u.back().cout;
    uint64_t off = 0;
    auto take = [&](uint64_t bytes) {
      uint64_t o = off;
      off += align256(bytes);
      return o;
    };
    ks_loss = take(4);
    ks_bnpart = take(bnpart);
    ks_sums = take(8ull * (C0 << 2));
    ks_wpart = take(wpart);
    ks_pooled = take(4ull * N * CL);
    ks_dlog = take(4ull * N * K);
    ks_lossn = take(4ull * N);
    ks_nst = take(nst_bytes);                                   // node graph: BN statistics
    ks_fcpart = take(4ull * mlp_relu_row_blocks(N) * K);         // node graph: FC bias sums
    // every unit's batch-norm statistics (mean | rstd per BN, 256-byte
    // aligned), formed by its first forward of the step and read by its
    // re-runs and its backward: held for the whole step, so they are fixed
    // buffers of the static layout (counted in the peak), not operator
    // workspace
    uint64_t kst = 0;
    for (const Blk &k : u) {
      kst_off.push_back(kst);
      kst += (k.w2 >= 0 ? 2 : 1) * align256(8ull * k.cout);
    }
    grad_extra = kst;
    ks_bytes = off;
    timed_family = "k_conv3x3< and k_conv3x3s<";
  }

  double *bnpart(StepCtx &c) const { return reinterpret_cast<double *>(c.ks + ks_bnpart); }
  // unit i's statistics: BN 1 (or the stem's), then BN 2 at + align256(8 cout)
  float *kst(const StepCtx &c, int32_t i) const {
    return reinterpret_cast<float *>(c.gextra + kst_off[size_t(i)]);
  }

  // a block's saved tensors: c1 | [r1] | c2 (then the reserved statistics slots)
  struct Saved {
    float *c1, *r1, *c2;
  };
  Saved saved_of(const Blk &k, char *sv) const {
    const uint64_t t = align256(uint64_t(N) * k.hout * k.hout * k.cout * 4);
    const int nt = drop ? 2 : 3;
    Saved s;
    s.c1 = reinterpret_cast<float *>(sv);
    s.r1 = drop ? nullptr : reinterpret_cast<float *>(sv + t);
    s.c2 = reinterpret_cast<float *>(sv + (nt - 1) * t);
    return s;
  }

  // conv3x3 launch bracketed by the kernel timer.  Algorithmic work of a 3x3
  // convolution with output [N, ho, ho, cout] and input channels cin (the same
  // for its forward and its data gradient): 2 * N*ho*ho * cout * 9*cin flops;
  // bytes = kernel input + weights + kernel output + epilogue tensors read.
  void conv(StepCtx &c, int mode, int s, int epi, const float *X, const float *Wt, float *Y, int H,
            int W, int Hx, int Wx, int C, int J, const float *E0, const float *E1, int Eh, int Ew,
            int Ec, int ho, int cin, int cout, const float *tst = nullptr, const float *tg = nullptr,
            const float *tb = nullptr, float *rout = nullptr) {
    const double fl = 2.0 * N * ho * ho * double(cout) * 9.0 * cin;
    double by = 4.0 * (double(N) * Hx * Wx * C + 9.0 * cin * cout + double(N) * H * W * J);
    if (epi == CONV_EPI_MASK || epi == CONV_EPI_MASKSTATS) by += 4.0 * N * H * W * J;
    if (epi == CONV_EPI_SC1 || epi == CONV_EPI_SC2) by += 2 * 4.0 * N * Eh * Ew * std::min(Ec, J);
    if (rout) by += 4.0 * N * Hx * Wx * C;  // the transformed input, written once
    timer.begin(c.s);
    conv3x3(c.s, mode, s, epi, X, Wt, Y, N, H, W, Hx, Wx, C, J, E0, E1, Eh, Ew, Ec,
            (epi == CONV_EPI_STATS || epi == CONV_EPI_MASKSTATS) ? bnpart(c) : nullptr, tst, tg, tb,
            rout);
    timer.end(c.s, fl, by);
  }
  float *ksf(StepCtx &c, uint64_t off) const { return reinterpret_cast<float *>(c.ks + off); }

  void fwd(int32_t i, const void *xv, void *yv, void *saved, StepCtx &c) override {
    const Blk &k = u[size_t(i)];
    const float *x = static_cast<const float *>(xv);
    float *y = static_cast<float *>(yv);
    char *sv = static_cast<char *>(saved);
    const uint64_t t = align256(uint64_t(N) * k.hout * k.hout * k.cout * 4);
    const int64_t np = int64_t(N) * k.hout * k.hout;
    if (k.w2 < 0) {  // stem
      float *cv = reinterpret_cast<float *>(sv);
      float *st = kst(c, i);
      (void)t;
      conv(c, CONV_FWD, 1, CONV_EPI_STATS, x, P(c, k.w1), cv, S, S, S, S, 3, C0, nullptr, nullptr,
           0, 0, 0, S, 3, C0);
      if (!c.rerun)
        bn_finalize_fwd(c.s, bnpart(c), conv3x3_blocks(CONV_FWD, 1, N, S, S, 3, C0), C0, np, st, true);
      bn_apply(c.s, BN_RES_NONE, np, C0, cv, st, P(c, k.g1), P(c, k.b1), nullptr, 0, 0, 0, y);
      c.launches += c.rerun ? 2 : 3;
      return;
    }
    const Saved sp = saved_of(k, sv);
    float *c1 = sp.c1, *r1 = sp.r1, *c2 = sp.c2;
    // the statistics are formed by the unit's first forward of the step; a
    // re-run (same input bits, so the same sums) reuses them and skips both
    // finalize launches
    float *st1 = kst(c, i), *st2 = st1 + align256(8ull * k.cout) / 4;
    const int ho = k.hout;
    const int epi = c.rerun ? CONV_EPI_STORE : CONV_EPI_STATS;  // no sums on a re-run
    conv(c, CONV_FWD, k.stride, epi, x, P(c, k.w1), c1, ho, ho, k.hin, k.hin, k.cin, k.cout,
         nullptr, nullptr, 0, 0, 0, ho, k.cin, k.cout);
    if (!c.rerun)
      bn_finalize_fwd(c.s, bnpart(c), conv3x3_blocks(CONV_FWD, k.stride, N, ho, ho, k.cin, k.cout),
                      k.cout, np, st1, true);
    // the second convolution forms r1 = relu(bn1(c1)) on its input; when r1
    // is kept it also stores it (the rows each workgroup owns)
    conv(c, CONV_FWD, 1, epi, c1, P(c, k.w2), c2, ho, ho, ho, ho, k.cout, k.cout, nullptr, nullptr, 0,
         0, 0, ho, k.cout, k.cout, st1, P(c, k.g1), P(c, k.b1), drop ? nullptr : r1);
    c.launches -= 1;
    if (!c.rerun)
      bn_finalize_fwd(c.s, bnpart(c), conv3x3_blocks(CONV_FWD, 1, N, ho, ho, k.cout, k.cout), k.cout,
                      np, st2, true);
    bn_apply(c.s, k.stride == 1 ? BN_RES_ID : BN_RES_A, np, k.cout, c2, st2, P(c, k.g2),
             P(c, k.b2), x, ho, ho, k.cin, y);
    c.launches += c.rerun ? 4 : 6;
  }

  void bwd(int32_t i, const void *gv, void *dxv, const void *xv, const void *yv, const void *saved,
           void *qv, StepCtx &c) override {
    const Blk &k = u[size_t(i)];
    const float *g = static_cast<const float *>(gv);
    const float *x = static_cast<const float *>(xv);
    const float *y = static_cast<const float *>(yv);
    const char *sv = static_cast<const char *>(saved);
    const uint64_t t = align256(uint64_t(N) * k.hout * k.hout * k.cout * 4);
    const int64_t np = int64_t(N) * k.hout * k.hout;
    float *sums = ksf(c, ks_sums);
    float *wpart = ksf(c, ks_wpart);
    if (k.w2 < 0) {  // stem: no input gradient
      const float *cv = reinterpret_cast<const float *>(sv);
      const float *st = kst(c, i);
      (void)t;
      float *dc = static_cast<float *>(qv);
      bn_backward(c.s, np, C0, g, y, cv, st, P(c, k.g1), bnpart(c), sums, G(c, k.g1), G(c, k.b1), dc);
      conv3x3_wgrad(c.s, 1, x, dc, wpart, G(c, k.w1), N, S, S, S, S, 3, C0);
      c.launches += 5;
      return;
    }
    const Saved sp = saved_of(k, const_cast<char *>(sv));
    const float *c1 = sp.c1, *r1 = sp.r1, *c2 = sp.c2;
    const float *st1 = kst(c, i), *st2 = st1 + align256(8ull * k.cout) / 4;
    // r1 as read by the second convolution's backward: stored, or c1 with its
    // batch-norm + ReLU transform
    const float *x2 = drop ? c1 : r1;
    const float *tst = drop ? st1 : nullptr, *tg = drop ? P(c, k.g1) : nullptr,
                *tb = drop ? P(c, k.b1) : nullptr;
    float *Pb = static_cast<float *>(qv);
    float *Qb = reinterpret_cast<float *>(static_cast<char *>(qv) + t);
    const int ho = k.hout;
    // second BN (its input gradient is g masked by the block's final ReLU)
    bn_backward(c.s, np, k.cout, g, y, c2, st2, P(c, k.g2), bnpart(c), sums, G(c, k.g2), G(c, k.b2), Qb);
    // conv2: data gradient masked by the first ReLU, formed from c1 and its
    // statistics (the same bits as the stored relu(bn1(c1))), with the first
    // BN backward's partial sums over the masked gradient and c1 in its
    // epilogue; and conv2's weight gradient
    conv(c, CONV_DGRAD, 1, CONV_EPI_MASKSTATS, Qb, P(c, k.w2), Pb, ho, ho, ho, ho, k.cout, k.cout, c1,
         nullptr, 0, 0, 0, ho, k.cout, k.cout, st1, P(c, k.g1), P(c, k.b1));
    conv3x3_wgrad(c.s, 1, x2, Qb, wpart, G(c, k.w2), N, ho, ho, ho, ho, k.cout, k.cout, tst, tg, tb);
    // first BN: finalize those sums, then its element pass
    bn_finalize_bwd(c.s, bnpart(c), conv3x3_blocks(CONV_DGRAD, 1, N, ho, ho, k.cout, k.cout), k.cout,
                    np, sums, G(c, k.g1), G(c, k.b1), true);
    bn_backward_apply(c.s, np, k.cout, Pb, nullptr, c1, st1, P(c, k.g1), sums, Qb);
    c.launches += 8;
    if (dxv) {  // conv1 data gradient plus the shortcut's gradient
      conv(c, CONV_DGRAD, k.stride, k.stride == 1 ? CONV_EPI_SC1 : CONV_EPI_SC2, Qb, P(c, k.w1),
           static_cast<float *>(dxv), k.hin, k.hin, ho, ho, k.cout, k.cin, g, y, ho, ho, k.cout, ho,
           k.cin, k.cout);
      c.launches += 1;
    }
    conv3x3_wgrad(c.s, k.stride, x, Qb, wpart, G(c, k.w1), N, ho, ho, k.hin, k.hin, k.cin, k.cout);
    c.launches += 2;
  }

  void head(const void *xn, void *g, StepCtx &c) override {
    const Blk &k = u.back();
    pool_fc_ce_head(c.s, N, k.hout * k.hout, k.cout, K, static_cast<const float *>(xn), P(c, hw),
                    P(c, hb), static_cast<const int *>(c.target), ksf(c, ks_pooled),
                    ksf(c, ks_dlog), ksf(c, ks_lossn), static_cast<float *>(g), G(c, hw),
                    G(c, hb), ksf(c, ks_loss));
    c.launches += 2;
  }

  const float *loss_ptr(const StepCtx &c) const override {
    return reinterpret_cast<const float *>(c.ks + ks_loss);
  }

  // Node graph, in topological order: 0 data; the stem conv, BN, ReLU; per
  // block conv, BN, ReLU, conv, BN, [option-A shortcut of the block input at
  // stride 2], add (BN output + shortcut), ReLU; then average pool, FC and the
  // softmax cross-entropy loss, whose output is the loss gradient of the
  // logits.  Output bytes are the tensors' exact sizes; the flags give what
  // each operator's backward reads and whether it may run in place (section
  // 3's minimum dependencies).  Every node runs its own operator (the fused
  // chain kernels' arithmetic split into standalone conv, batch-norm,
  // activation, add, pool, FC and loss kernels).
  void build_nodes() {
    auto T = [&](int h, int ch) { return uint64_t(N) * h * h * ch * 4; };
    auto node = [&](GNode d) {
      gn.push_back(std::move(d));
      return int32_t(gn.size()) - 1;
    };
    auto conv_n = [&](int32_t x, int hin, int cin, int h, int cout, int stride, int w) {
      GNode d{ND_CONV, {x}, T(h, cout), h, cout, hin, cin, stride};
      d.w = w;
      return node(d);
    };
    auto bn_n = [&](int32_t x, int h, int ch, int g, int bt) {
      GNode d{ND_BN, {x}, T(h, ch), h, ch, h, ch, 1};
      d.g = g;
      d.bt = bt;
      d.st = nst_bytes;
      nst_bytes += align256(8ull * ch);
      return node(d);
    };
    auto relu_n = [&](int32_t x, int h, int ch) { return node(GNode{ND_RELU, {x}, T(h, ch), h, ch, h, ch, 1}); };
    int32_t x = node(GNode{ND_DATA, {}, T(S, 3), S, 3, S, 3, 1});
    {
      const Blk &k = u[0];
      x = conv_n(x, S, 3, S, C0, 1, k.w1);
      x = bn_n(x, S, C0, k.g1, k.b1);
      x = relu_n(x, S, C0);
    }
    for (size_t i = 1; i < u.size(); ++i) {
      const Blk &k = u[i];
      int32_t y = conv_n(x, k.hin, k.cin, k.hout, k.cout, k.stride, k.w1);
      y = bn_n(y, k.hout, k.cout, k.g1, k.b1);
      y = relu_n(y, k.hout, k.cout);
      y = conv_n(y, k.hout, k.cout, k.hout, k.cout, 1, k.w2);
      y = bn_n(y, k.hout, k.cout, k.g2, k.b2);
      int32_t sc = x;
      if (k.stride != 1)
        sc = node(GNode{ND_SHORT, {x}, T(k.hout, k.cout), k.hout, k.cout, k.hin, k.cin, k.stride});
      y = node(GNode{ND_ADD, {y, sc}, T(k.hout, k.cout), k.hout, k.cout, k.hout, k.cout, 1});
      x = relu_n(y, k.hout, k.cout);
    }
    const Blk &l = u.back();
    const int32_t p = node(GNode{ND_POOL, {x}, uint64_t(N) * l.cout * 4, 1, l.cout, l.hout, l.cout, 1});
    const int32_t f = node(GNode{ND_FC, {p}, uint64_t(N) * K * 4, 1, K, 1, l.cout, 1});
    node(GNode{ND_LOSS, {f}, uint64_t(N) * K * 4, 1, K, 1, K, 1});
  }

  bool node_graph(NodeGraph &g) const override {
    static const int32_t flag[] = {0,                                          // data
                                   CKPT_NODE_GRAD_IN,                          // conv
                                   CKPT_NODE_INPLACE | CKPT_NODE_GRAD_IN,      // bn
                                   CKPT_NODE_INPLACE | CKPT_NODE_GRAD_OUT,     // relu
                                   CKPT_NODE_INPLACE,                          // add
                                   0,                                          // shortcut
                                   0,                                          // pool
                                   CKPT_NODE_GRAD_IN,                          // fc
                                   CKPT_NODE_GRAD_OUT};                        // loss
    g.ptr.assign(1, 0);
    g.idx.clear();
    g.flags.clear();
    g.bytes.clear();
    for (const GNode &d : gn) {
      g.idx.insert(g.idx.end(), d.in.begin(), d.in.end());
      g.ptr.push_back(int32_t(g.idx.size()));
      g.flags.push_back(flag[d.op]);
      g.bytes.push_back(d.bytes);
    }
    return true;
  }

  float *nst(StepCtx &c, const GNode &d) const { return reinterpret_cast<float *>(c.ks + ks_nst + d.st); }

  void node_fwd(int32_t v, const std::vector<const void *> &ins, void *out, StepCtx &c) override {
    const GNode &d = gn[size_t(v)];
    float *y = static_cast<float *>(out);
    const float *x = ins.empty() ? nullptr : static_cast<const float *>(ins[0]);
    const int64_t np = int64_t(N) * d.h * d.h;
    switch (d.op) {
      case ND_DATA:
        if (hipMemcpyAsync(y, c.input, d.bytes, hipMemcpyDeviceToDevice, c.s) != hipSuccess)
          fail(CKPT_E_HIP, "train_step_graph: input copy failed");
        break;
      case ND_CONV:
        conv(c, CONV_FWD, d.stride, CONV_EPI_STORE, x, P(c, d.w), y, d.h, d.h, d.hin, d.hin, d.cin, d.c,
             nullptr, nullptr, 0, 0, 0, d.h, d.cin, d.c);
        break;
      case ND_BN:  // statistics (partials + finalize), then the affine map
        bn_stats(c.s, np, d.c, x, bnpart(c), nst(c, d));
        bn_norm(c.s, np, d.c, x, nst(c, d), P(c, d.g), P(c, d.bt), y);
        c.launches += 2;
        break;
      case ND_RELU:
        ew_relu(c.s, np * d.c, x, y);
        break;
      case ND_ADD:
        ew_add(c.s, np * d.c, x, static_cast<const float *>(ins[1]), y);
        break;
      case ND_SHORT:
        shortcut_a(c.s, N, d.h, d.h, d.c, d.cin, x, y);
        break;
      case ND_POOL:
        avgpool(c.s, N, d.hin * d.hin, d.c, x, y);
        break;
      case ND_FC:
        gemm_f32(c.s, N, K, d.cin, x, d.cin, false, P(c, hw), K, false, y, K, GEMM_EPI_BIAS, nullptr, 0,
                 P(c, hb));
        break;
      case ND_LOSS:
        softmax_ce_rows(c.s, N, K, x, static_cast<const int *>(c.target), y, ksf(c, ks_lossn),
                        ksf(c, ks_loss));
        c.launches += 1;
        break;
    }
    c.launches += 1;
  }

  void node_bwd(int32_t v, const void *dyv, const void *yv, const std::vector<const void *> &ins, void *out,
                StepCtx &c) override {
    const GNode &d = gn[size_t(v)];
    const float *dy = static_cast<const float *>(dyv);
    float *o = static_cast<float *>(out);
    const int64_t np = int64_t(N) * d.h * d.h;
    switch (d.op) {
      case ND_DATA:
        return;  // the input has no gradient to form
      case ND_CONV: {
        const float *x = static_cast<const float *>(ins[0]);
        if (d.in[0] != 0) {  // the stem's input is the image: no data gradient
          conv(c, CONV_DGRAD, d.stride, CONV_EPI_STORE, dy, P(c, d.w), o, d.hin, d.hin, d.h, d.h, d.c,
               d.cin, nullptr, nullptr, 0, 0, 0, d.h, d.cin, d.c);
          c.launches += 1;
        }
        conv3x3_wgrad(c.s, d.stride, x, dy, ksf(c, ks_wpart), G(c, d.w), N, d.h, d.h, d.hin, d.hin, d.cin,
                      d.c);
        c.launches += 2;
        return;
      }
      case ND_BN:
        bn_backward(c.s, np, d.c, dy, nullptr, static_cast<const float *>(ins[0]), nst(c, d), P(c, d.g),
                    bnpart(c), ksf(c, ks_sums), G(c, d.g), G(c, d.bt), o);
        c.launches += 3;
        return;
      case ND_RELU:
        ew_relu_bwd(c.s, np * d.c, dy, static_cast<const float *>(yv), o);
        break;
      case ND_ADD:  // both inputs receive dy
        ew_copy(c.s, np * d.c, dy, o);
        ew_copy(c.s, np * d.c, dy, o + np * d.c);
        c.launches += 1;
        break;
      case ND_SHORT:
        shortcut_a_bwd(c.s, N, d.h, d.h, d.c, d.cin, dy, o);
        break;
      case ND_POOL:
        avgpool_bwd(c.s, N, d.hin * d.hin, d.c, dy, o);
        break;
      case ND_FC: {  // dx = dy W^T, dW = x^T dy, db = column sums of dy
        const float *x = static_cast<const float *>(ins[0]);
        gemm_f32(c.s, N, d.cin, K, dy, K, false, P(c, hw), K, true, o, d.cin, GEMM_EPI_STORE);
        gemm_f32(c.s, d.cin, K, N, x, d.cin, true, dy, K, false, G(c, hw), K, GEMM_EPI_STORE);
        mlp_colsum(c.s, N, K, dy, G(c, hb), ksf(c, ks_fcpart));
        c.launches += 3;
        break;
      }
      case ND_LOSS:  // the loss node's output is dL/d(logits) already
        ew_copy(c.s, int64_t(N) * K, static_cast<const float *>(yv), o);
        break;
    }
    c.launches += 1;
  }
};

bool pow2(int v) { return v > 0 && (v & (v - 1)) == 0; }

}  // namespace

std::unique_ptr<Net> make_resnet_basic_net(const ckpt_net_desc &d) {
  if (d.batch <= 0 || d.depth <= 0 || d.width <= 0 || d.image <= 0 || d.n_classes <= 0)
    fail(CKPT_E_INVALID, "net_create: RESNET_BASIC needs positive batch, depth, width, image, classes");
  if (d.width % 4 != 0 || !pow2(d.width / 4) || (d.width << 2) > 1024)
    fail(CKPT_E_UNSUPPORTED, "net_create: RESNET_BASIC width must be 4 * 2^k and at most 256");
  if (d.image % 4 != 0)
    fail(CKPT_E_INVALID, "net_create: RESNET_BASIC image side must be a multiple of 4");
  if (int64_t(d.batch) * d.image * d.image * (d.width << 2) > (int64_t(1) << 31))
    fail(CKPT_E_INVALID, "net_create: RESNET_BASIC tensors too large");
  for (int st = 0; st < 3; ++st) {
    const int cout = d.width << st, side = d.image >> st;
    const int cin = st == 0 ? d.width : cout / 2;
    if (!conv3x3_supported(CONV_FWD, st == 0 ? 1 : 2, side, side, cin, cout) ||
        !conv3x3_supported(CONV_FWD, 1, side, side, cout, cout) ||
        !conv3x3_supported(CONV_DGRAD, st == 0 ? 1 : 2, side << (st ? 1 : 0), side << (st ? 1 : 0), cout, cin))
      fail(CKPT_E_UNSUPPORTED, "net_create: RESNET_BASIC shape outside the conv kernels' tiling");
  }
  return std::make_unique<ResNetBasic>(d);
}

}  // namespace ckpt
