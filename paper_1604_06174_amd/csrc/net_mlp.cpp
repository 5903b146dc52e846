// Residual-MLP chain: unit i computes y = x + relu(x W_i + b_i) on [batch, width]
// fp32 (the fully connected operator of the paper's Fig. 1, made residual so
// that a deep chain stays trainable); head = mean squared error.
//
// Static layout per unit: boundary b = [B, D] f32; saved internals a = the
// pre-activation z [B, D]; gradient scratch q = the masked gradient dr [B, D].
#include "kernels.h"
#include "net.h"

namespace ckpt {
namespace {

class MlpNet : public Net {
 public:
  int B, D;
  std::vector<int> wi, bi;

  explicit MlpNet(const ckpt_net_desc &d) {
    desc = d;
    n = d.depth;
    B = d.batch;
    D = d.width;
    const uint64_t t = align256(uint64_t(B) * D * 4);
    b.assign(size_t(n) + 1, t);
    a.assign(size_t(n), t);
    q.assign(size_t(n), t);
    for (int i = 0; i < n; ++i) {
      wi.push_back(add_param("u" + std::to_string(i) + ".W", uint64_t(D) * D));
      bi.push_back(add_param("u" + std::to_string(i) + ".b", uint64_t(D)));
    }
    // loss scalar | bias-gradient partial sums of the ReLU backward
    ks_bytes = 256 + align256(uint64_t(mlp_relu_row_blocks(B)) * D * 4);
    timed_family = "k_gemm_f32";
  }

  // algorithmic cost of one [M,K] x [K,N] product: operands read once,
  // result written once (+ the epilogue's extra tensors)
  static double gf(double M, double N, double K) { return 2.0 * M * N * K; }
  static double gb(double M, double N, double K, double extra) {
    return 4.0 * (M * K + K * N + M * N) + extra;
  }

  void fwd(int32_t i, const void *x, void *y, void *saved, StepCtx &c) override {
    timer.begin(c.s);
    gemm_f32(c.s, B, D, D, static_cast<const float *>(x), D, false, P(c, wi[i]), D, false,
             static_cast<float *>(y), D, GEMM_EPI_MLPFWD, nullptr, 0, P(c, bi[i]),
             static_cast<float *>(saved), D);
    timer.end(c.s, gf(B, D, D), gb(B, D, D, 4.0 * D + 4.0 * B * D));
    c.launches += 1;
  }

  void bwd(int32_t i, const void *g, void *dx, const void *x, const void *, const void *saved,
           void *q, StepCtx &c) override {
    const float *gp = static_cast<const float *>(g);
    float *dr = static_cast<float *>(q);
    mlp_relu_bwd(c.s, B, D, gp, static_cast<const float *>(saved), dr, G(c, bi[i]),
                 reinterpret_cast<float *>(c.ks + 256));
    // dW = x^T dr : [D_in, D_out] = [D, B] x [B, D]
    timer.begin(c.s);
    gemm_f32(c.s, D, D, B, static_cast<const float *>(x), D, true, dr, D, false, G(c, wi[i]), D,
             GEMM_EPI_STORE);
    timer.end(c.s, gf(D, D, B), gb(D, D, B, 0));
    c.launches += 3;
    if (dx) {  // dx = g + dr W^T
      timer.begin(c.s);
      gemm_f32(c.s, B, D, D, dr, D, false, P(c, wi[i]), D, true, static_cast<float *>(dx), D,
               GEMM_EPI_ADD, gp, D);
      timer.end(c.s, gf(B, D, D), gb(B, D, D, 4.0 * B * D));
      c.launches += 1;
    }
  }

  void head(const void *xn, void *g, StepCtx &c) override {
    mse_head(c.s, int64_t(B) * D, static_cast<const float *>(xn),
             static_cast<const float *>(c.target), static_cast<float *>(g),
             reinterpret_cast<float *>(c.ks));
    c.launches += 1;
  }

  // Node graph: 0 data; block i: 1 + 3i fully connected (x W + b), 2 + 3i ReLU,
  // 3 + 3i add (ReLU output + block input); 3n + 1 the MSE loss, whose output
  // is the loss gradient.  Every tensor is [B, D] f32.  The operators and their
  // order of arithmetic are those of the fused unit, so any plan of this graph
  // gives the chain's gradients bit for bit.
  bool node_graph(NodeGraph &g) const override {
    const uint64_t t = uint64_t(B) * D * 4;
    g.ptr.assign(1, 0);
    g.idx.clear();
    g.flags.clear();
    g.bytes.clear();
    auto node = [&](std::initializer_list<int32_t> ins, int32_t fl) {
      for (int32_t u : ins) g.idx.push_back(u);
      g.ptr.push_back(int32_t(g.idx.size()));
      g.flags.push_back(fl);
      g.bytes.push_back(t);
    };
    node({}, 0);
    for (int32_t i = 0; i < n; ++i) {
      const int32_t x = 3 * i;
      node({x}, CKPT_NODE_GRAD_IN);                         // fully connected
      node({x + 1}, CKPT_NODE_INPLACE | CKPT_NODE_GRAD_OUT);  // ReLU
      node({x + 2, x}, CKPT_NODE_INPLACE);                   // add
    }
    node({3 * n}, CKPT_NODE_GRAD_OUT);                      // loss
    return true;
  }

  void node_fwd(int32_t v, const std::vector<const void *> &ins, void *out, StepCtx &c) override {
    const int64_t t = int64_t(B) * D;
    float *y = static_cast<float *>(out);
    if (v == 0) {
      if (hipMemcpyAsync(y, c.input, size_t(t) * 4, hipMemcpyDeviceToDevice, c.s) != hipSuccess)
        fail(CKPT_E_HIP, "train_step_graph: input copy failed");
    } else if (v == 3 * n + 1) {
      mse_head(c.s, t, static_cast<const float *>(ins[0]), static_cast<const float *>(c.target), y,
               reinterpret_cast<float *>(c.ks));
    } else {
      const int i = (v - 1) / 3, k = (v - 1) % 3;
      const float *x = static_cast<const float *>(ins[0]);
      if (k == 0) {
        timer.begin(c.s);
        gemm_f32(c.s, B, D, D, x, D, false, P(c, wi[i]), D, false, y, D, GEMM_EPI_BIAS, nullptr, 0,
                 P(c, bi[i]), nullptr, 0);
        timer.end(c.s, gf(B, D, D), gb(B, D, D, 4.0 * D));
      } else if (k == 1) {
        ew_relu(c.s, t, x, y);
      } else {
        ew_add(c.s, t, x, static_cast<const float *>(ins[1]), y);
      }
    }
    c.launches += 1;
  }

  void node_bwd(int32_t v, const void *dyv, const void *yv, const std::vector<const void *> &ins,
                void *out, StepCtx &c) override {
    const int64_t t = int64_t(B) * D;
    const float *dy = static_cast<const float *>(dyv);
    float *o = static_cast<float *>(out);
    if (v == 0) return;  // the input has no gradient to form
    if (v == 3 * n + 1) {  // the loss node's output is dL/dx_n already
      ew_copy(c.s, t, static_cast<const float *>(yv), o);
      c.launches += 1;
      return;
    }
    const int i = (v - 1) / 3, k = (v - 1) % 3;
    if (k == 0) {  // fully connected: dx = dy W^T, dW = x^T dy, db = column sums of dy
      const float *x = static_cast<const float *>(ins[0]);
      timer.begin(c.s);
      gemm_f32(c.s, B, D, D, dy, D, false, P(c, wi[i]), D, true, o, D, GEMM_EPI_STORE);
      timer.end(c.s, gf(B, D, D), gb(B, D, D, 0));
      timer.begin(c.s);
      gemm_f32(c.s, D, D, B, x, D, true, dy, D, false, G(c, wi[i]), D, GEMM_EPI_STORE);
      timer.end(c.s, gf(D, D, B), gb(D, D, B, 0));
      mlp_colsum(c.s, B, D, dy, G(c, bi[i]), reinterpret_cast<float *>(c.ks + 256));
      c.launches += 4;
    } else if (k == 1) {  // ReLU: the mask from its output
      ew_relu_bwd(c.s, t, dy, static_cast<const float *>(yv), o);
      c.launches += 1;
    } else {  // add: both inputs receive dy
      ew_copy(c.s, t, dy, o);
      ew_copy(c.s, t, dy, o + t);
      c.launches += 2;
    }
  }

  const float *loss_ptr(const StepCtx &c) const override {
    return reinterpret_cast<const float *>(c.ks);
  }
};

}  // namespace

std::unique_ptr<Net> make_mlp_net(const ckpt_net_desc &d) {
  if (d.depth <= 0 || d.width <= 0 || d.batch <= 0)
    fail(CKPT_E_INVALID, "net_create: MLP needs positive depth, width and batch");
  if (int64_t(d.batch) * d.width > (int64_t(1) << 31))
    fail(CKPT_E_INVALID, "net_create: MLP tensor too large");
  return std::make_unique<MlpNet>(d);
}

}  // namespace ckpt
