// Single-layer LSTM unrolled over T steps with a softmax head at every step
// (the long-sequence recurrent workload of the paper's section 5.3).  Unit t
// maps the state (h_{t-1}, c_{t-1}) to (h_t, c_t) and adds the step's
// cross-entropy to the loss; the chain's own head is empty (g = 0).
//
//   z_t      = x_t W_x + h_{t-1} W_h + b          bf16 operands, fp32 accumulation
//   gates    i, f, g, o;  c_t = f c_{t-1} + i g;  h_t = o tanh(c_t)   (c fp32, h bf16)
//   logits_t = h_t W_o + b_o;  loss += sum_b CE(logits_t[b], label_t[b]) / (T B)
//
// Shared parameters: their gradients are summed in backward order, T-1 -> 0.
// Weight gradients are computed per fixed chunk of C aligned steps (one GEMM
// over the chunk's C*B rows, accumulated chunk after chunk in backward order);
// the chunk grouping does not depend on the plan, so every plan gives the same
// bytes.  Bias gradients accumulate step by step.
//
// The head of a step (logits, softmax gradient, loss rows) feeds only the
// unit's saved internals and the loss, so a forward whose saved internals are
// discarded (a checkpointed step's forward sweeps) runs the recurrence alone;
// the head runs with the unit's kept forward, once per step in every plan,
// for up to HG steps of a kept segment at once (one batched logits product,
// each step's product computed exactly as its own launch would, written over
// the step's saved softmax-gradient buffer, then one batched softmax pass in
// place), and the loss rows are reduced after the last backward.
//
// Static layout: boundary b = h (bf16 [B,H]) | c (fp32 [B,H]); saved a = gates
// (fp32 [B,4H]) | softmax gradient (fp32 [B,V]); scratch q = total dh (fp32
// [B,H]); gradient slot = dh | dc (fp32; only dc is written: the previous
// step's backward forms dz_t W_h^T itself, in one product with its own head
// gradient); extra gradient buffers = the chunk's
// dz (bf16 [C*B,4H]), head gradient (bf16 [C*B,V]), h_{t-1} and h_t copies
// (bf16 [C*B,H]).
#include <algorithm>

#include "kernels.h"
#include "net.h"

namespace ckpt {
namespace {

class LstmNet : public Net {
 public:
  static constexpr int HG = 64;  // steps per batched head
  int T, B, E, H, V, C;
  int pWx, pWh, pb, pWo, pbo;
  uint64_t hb, cb;  // boundary parts
  uint64_t ga, da;  // saved parts: gates, dlog
  // operator workspace offsets
  uint64_t k_wcat, k_wot, k_wob, k_dbp, k_lossrows, k_loss, k_part, k_rstat;
  bool zcat;  // z = [x_t | h_{t-1}] [W_x; W_h] as one product (same slices as the two)
  // split-K counts: input and recurrent parts of z, the last step's dh (head
  // only), every other step's dh (head and recurrence in one product); the
  // logits are one product (their softmax statistics come from its epilogue)
  int s_x, s_h, s_dh, s_dm;
  // extra gradient buffer offsets
  uint64_t x_dz, x_dl, x_hp, x_hc;

  explicit LstmNet(const ckpt_net_desc &d) {
    desc = d;
    T = d.depth;
    B = d.batch;
    H = d.width;
    E = d.image;
    V = d.n_classes;
    C = d.grad_chunk > 0 ? d.grad_chunk : 32;
    n = T;
    pWx = add_param("W_x", uint64_t(E) * 4 * H);
    pWh = add_param("W_h", uint64_t(H) * 4 * H);
    pb = add_param("b", uint64_t(4) * H);
    pWo = add_param("W_o", uint64_t(H) * V);
    pbo = add_param("b_o", uint64_t(V));
    hb = align256(2ull * B * H);
    cb = align256(4ull * B * H);
    ga = align256(16ull * B * H);
    da = align256(4ull * B * V);
    b.assign(size_t(n) + 1, hb + cb);
    a.assign(size_t(n), ga + da);
    q.assign(size_t(n), align256(4ull * B * H));
    gslot_bytes = 2 * align256(4ull * B * H);
    uint64_t off = 0;
    auto take = [&](uint64_t bytes) {
      uint64_t o = off;
      off += align256(bytes);
      return o;
    };
    x_dz = take(uint64_t(C) * B * 4 * H * 2);
    x_dl = take(uint64_t(C) * B * V * 2);
    x_hp = take(uint64_t(C) * B * H * 2);
    x_hc = take(uint64_t(C) * B * H * 2);
    grad_extra = off;
    off = 0;
    k_wcat = take(uint64_t(E + H) * 4 * H * 2);  // [4H][E + H]: W_x^T | W_h^T

    k_wot = take(uint64_t(H) * V * 2);
    k_wob = take(uint64_t(H) * (V + 4 * H) * 2);  // [H][V + 4H]: W_o | W_h
    // bias-gradient column sums of one chunk: per step, one [4H] record per
    // block of 4 batch rows
    k_dbp = take(uint64_t(C) * ((B + 3) / 4) * 4 * H * 4);
    k_lossrows = take(uint64_t(T) * B * 4);
    k_loss = take(4);
    // z's slices are read back by the pointwise launch right away, so it takes
    // fewer, longer splits (about 128 workgroups per part: 256 for z over
    // [x_t | h_{t-1}] at the 1024/1024/64 shape, 4 slices instead of 16); the
    // backward's products keep about 512 workgroups.
    s_x = gemm_bf16_splits(B, 4 * H, E, 128);
    s_h = gemm_bf16_splits(B, 4 * H, H, 128);
    // one launch for both parts of z when its k splits fall exactly on the two
    // parts' own splits (then every slice holds the same sums in the same order)
    zcat = E == H && s_x == s_h && gemm_bf16_kper(E, s_x) * s_x == E &&
           gemm_bf16_kper(E + H, s_x + s_h) == gemm_bf16_kper(E, s_x) && E % 8 == 0;
    s_dh = gemm_bf16_splits(B, H, V);
    s_dm = gemm_bf16_splits(B, H, V + 4 * H);
    const uint64_t part = std::max({uint64_t(s_x + s_h) * B * 4 * H, uint64_t(B) * V,
                                    uint64_t(std::max(s_dh, s_dm)) * B * H});
    k_part = take(part * 4);
    k_rstat = take(uint64_t(HG) * B * gemm_bf16_col_blocks(B, V) * 2 * 4);
    ks_bytes = off;
    timed_family = "k_gemm_bf16";
  }

  char *K(StepCtx &c, uint64_t o) const { return c.ks + o; }
  float *Kf(StepCtx &c, uint64_t o) const { return reinterpret_cast<float *>(c.ks + o); }
  char *X(StepCtx &c, uint64_t o) const { return c.gextra + o; }

  void gemm(StepCtx &c, int M, int N, int Kd, const void *A, bool a32, int lda, bool ak,
            const void *Bm, int ldb, bool bk, float *Cm, int ldc, int epi, const float *D = nullptr,
            int ldd = 0, const float *bias = nullptr) {
    timer.begin(c.s);
    gemm_bf16(c.s, M, N, Kd, A, a32, lda, ak, Bm, ldb, bk, Cm, ldc, epi, D, ldd, bias);
    // operands and product once; the ADD epilogue also reads D once
    timer.end(c.s, 2.0 * M * N * Kd,
              2.0 * (double(M) * Kd + double(Kd) * N) + (epi == GEMM_EPI_ADD ? 8.0 : 4.0) * M * N);
    c.launches += 1;
  }
  // split-K partial products into slices [z0, z0 + splits) of the partial buffer.
  // Algorithmic bytes: each operand read once and the product written once
  // (the slices are this implementation's, not the product's, traffic).
  void gemm_part(StepCtx &c, int M, int N, int Kd, const void *A, int lda, const void *Bm, int ldb,
                 int z0, int splits) {
    timer.begin(c.s);
    gemm_bf16_part(c.s, M, N, Kd, A, false, lda, true, Bm, ldb, true,
                   Kf(c, k_part) + size_t(z0) * M * N, splits);
    timer.end(c.s, 2.0 * M * N * Kd, 2.0 * (double(M) * Kd + double(Kd) * N) + 4.0 * M * N);
    c.launches += 1;
  }

  void begin_step(StepCtx &c) override {
    // bf16 copies of the weights in the layouts the GEMMs read (k contiguous)
    transpose_bf16(c.s, E, 4 * H, P(c, pWx), K(c, k_wcat), E + H);              // [4H][0, E)
    transpose_bf16(c.s, H, 4 * H, P(c, pWh), K(c, k_wcat) + size_t(E) * 2, E + H);  // [4H][E, E + H)
    cvt_bf16_rows(c.s, H, 4 * H, P(c, pWh), K(c, k_wob) + size_t(V) * 2, V + 4 * H);  // [H][V, V + 4H)
    transpose_bf16(c.s, H, V, P(c, pWo), K(c, k_wot));        // [V][H]
    cvt_bf16_rows(c.s, H, V, P(c, pWo), K(c, k_wob), V + 4 * H);                    // [H][0, V)
    c.launches += 5;
  }

  void fwd(int32_t i, const void *xv, void *yv, void *saved, StepCtx &c) override {
    const char *x = static_cast<const char *>(xv);
    char *y = static_cast<char *>(yv);
    char *sv = static_cast<char *>(saved);
    const void *xt = static_cast<const char *>(c.input) + size_t(i) * B * E * 2;
    // z = x_t W_x + h_{t-1} W_h + b: both products split over k into one
    // slice buffer that the pointwise kernel adds up in order with the bias
    if (i > 0 && zcat) {
      timer.begin(c.s);
      gemm_bf16_part_cat(c.s, B, 4 * H, E, xt, E, H, x, H, K(c, k_wcat), E + H, Kf(c, k_part),
                         s_x + s_h);
      timer.end(c.s, 2.0 * B * 4 * H * (E + H),
                2.0 * (double(B) * (E + H) + double(E + H) * 4 * H) + 4.0 * B * 4 * H);
      c.launches += 1;
    } else {
      gemm_part(c, B, 4 * H, E, xt, E, K(c, k_wcat), E + H, 0, s_x);
      if (i > 0) gemm_part(c, B, 4 * H, H, x, H, K(c, k_wcat) + size_t(E) * 2, E + H, s_x, s_h);
    }
    const float *c_prev = i > 0 ? reinterpret_cast<const float *>(x + hb) : nullptr;
    float *gates = reinterpret_cast<float *>(sv);
    lstm_fwd_point(c.s, B, H, Kf(c, k_part), s_x + (i > 0 ? s_h : 0), P(c, pb), c_prev, gates, y,
                   reinterpret_cast<float *>(y + hb));
    c.launches += 1;
    // the step's head runs after the kept forward of its segment (fwd_segment)
  }

  // the heads of steps i0 .. i0 + nb - 1: h_t at y0 + k sy (bf16 elements),
  // logits and then the softmax gradient at dl0 + k sd (floats)
  void heads(int32_t i0, int nb, const char *y0, int64_t sy, float *dl0, int64_t sd, StepCtx &c) {
    const int nt = gemm_bf16_col_blocks(B, V);
    const int64_t ur = int64_t(B) * nt * 2;
    timer.begin(c.s);
    gemm_bf16_rowsoftmax_batched(c.s, nb, B, V, H, y0, H, sy, K(c, k_wot), H, dl0, sd, P(c, pbo),
                                 Kf(c, k_rstat), ur);
    // each step's h and logits once, the shared W_o once
    timer.end(c.s, 2.0 * nb * B * V * H, nb * (2.0 * B * H + 4.0 * B * V) + 2.0 * H * V);
    softmax_ce_tiles_batched(c.s, nb, B, V, dl0, sd, nt, Kf(c, k_rstat), ur,
                             static_cast<const int *>(c.target) + size_t(i0) * B, 1.0f / (float(T) * float(B)),
                             Kf(c, k_lossrows) + size_t(i0) * B);
    c.launches += 2;
  }

  void fwd_segment(int32_t lo, int32_t hi, const std::vector<void *> &saved, const std::vector<void *> &out,
                   StepCtx &c) override {
    for (int32_t g0 = lo; g0 < hi; g0 += HG) {
      const int nb = int(std::min<int32_t>(hi - g0, HG));
      const char *y0 = static_cast<const char *>(out[size_t(g0 - lo)]);
      char *s0 = static_cast<char *>(saved[size_t(g0 - lo)]);
      // the arena places a segment's units at one stride; batch them when it
      // holds (and the strides are whole elements), else one step at a time
      const int64_t sy = nb > 1 ? static_cast<const char *>(out[size_t(g0 - lo) + 1]) - y0 : 0;
      const int64_t ss = nb > 1 ? static_cast<char *>(saved[size_t(g0 - lo) + 1]) - s0 : 0;
      bool uniform = sy % 16 == 0 && ss % 16 == 0;
      for (int k = 1; uniform && k < nb; ++k)
        uniform = static_cast<const char *>(out[size_t(g0 - lo + k)]) - y0 == k * sy &&
                  static_cast<char *>(saved[size_t(g0 - lo + k)]) - s0 == k * ss;
      if (uniform) {
        heads(g0, nb, y0, sy / 2, reinterpret_cast<float *>(s0 + ga), ss / 4, c);
      } else {
        for (int k = 0; k < nb; ++k)
          heads(g0 + k, 1, static_cast<const char *>(out[size_t(g0 - lo + k)]), 0,
                reinterpret_cast<float *>(static_cast<char *>(saved[size_t(g0 - lo + k)]) + ga), 0, c);
      }
    }
  }

  void bwd(int32_t i, const void *gv, void *dxv, const void *xv, const void *yv, const void *saved,
           void *qv, StepCtx &c) override {
    const char *g = static_cast<const char *>(gv);
    const char *x = static_cast<const char *>(xv);
    const char *y = static_cast<const char *>(yv);
    const char *sv = static_cast<const char *>(saved);
    char *dx = static_cast<char *>(dxv);
    const uint64_t gh = align256(4ull * B * H);  // dh part of a gradient slot
    const int t0 = (i / C) * C;
    const size_t row = size_t(i - t0) * B;
    const bool first_step = i == n - 1;
    const int t_end = std::min(t0 + C, int(n)), rb = (B + 3) / 4;
    char *dl = X(c, x_dl) + row * V * 2;
    char *dz = X(c, x_dz) + row * 4 * H * 2;
    char *hp = X(c, x_hp) + row * H * 2;
    char *hc = X(c, x_hc) + row * H * 2;
    head_bwd_prep(c.s, B, V, reinterpret_cast<const float *>(sv + ga), dl, G(c, pbo), first_step);
    (void)qv;
    // total dh = dl_t W_o^T + dz_{t+1} W_h^T (the incoming dh; none at the
    // last step): one split-K product over [dl_t | dz_{t+1}] and [W_o | W_h],
    // its slices added up by the gate backward.  dz_{t+1} is the next step's
    // row of the chunk buffer (row 0 of it when t + 1 began a chunk; nothing
    // has written that row since).
    int ns = s_dh;
    if (first_step) {
      gemm_part(c, B, H, V, dl, V, K(c, k_wob), V + 4 * H, 0, s_dh);
    } else {
      const int t1 = i + 1;
      const char *dzn = X(c, x_dz) + size_t(t1 - (t1 / C) * C) * B * 4 * H * 2;
      timer.begin(c.s);
      gemm_bf16_part_cat(c.s, B, H, V, dl, V, 4 * H, dzn, 4 * H, K(c, k_wob), V + 4 * H,
                         Kf(c, k_part), s_dm);
      timer.end(c.s, 2.0 * B * H * (V + 4.0 * H),
                2.0 * (double(B) * (V + 4 * H) + double(V + 4 * H) * H) + 4.0 * B * H);
      c.launches += 1;
      ns = s_dm;
    }
    lstm_bwd_point(c.s, B, H, Kf(c, k_part), ns, reinterpret_cast<const float *>(g + gh),
                   reinterpret_cast<const float *>(sv), reinterpret_cast<const float *>(y + hb),
                   i > 0 ? reinterpret_cast<const float *>(x + hb) : nullptr, i > 0 ? x : nullptr, y, dz,
                   dx ? reinterpret_cast<float *>(dx + gh) : nullptr, hp, hc,
                   Kf(c, k_dbp) + size_t(t_end - 1 - i) * rb * 4 * H);
    c.launches += 2;
    if (i == t0) {  // the chunk [t0, t0 + C) is complete: its weight gradients
      const int rows = (t_end - t0) * B;
      const bool first_chunk = t0 + C >= n;
      // b: the chunk's records in backward order of the steps
      db_chunk(c.s, 4 * H, (t_end - t0) * rb, Kf(c, k_dbp), G(c, pb), first_chunk);
      c.launches += 1;
      const int epi = first_chunk ? GEMM_EPI_STORE : GEMM_EPI_ADD;
      const void *xs = static_cast<const char *>(c.input) + size_t(t0) * B * E * 2;
      gemm(c, E, 4 * H, rows, xs, false, E, false, X(c, x_dz), 4 * H, false, G(c, pWx), 4 * H, epi,
           G(c, pWx), 4 * H);
      gemm(c, H, 4 * H, rows, X(c, x_hp), false, H, false, X(c, x_dz), 4 * H, false, G(c, pWh), 4 * H,
           epi, G(c, pWh), 4 * H);
      gemm(c, H, V, rows, X(c, x_hc), false, H, false, X(c, x_dl), V, false, G(c, pWo), V, epi,
           G(c, pWo), V);
    }
  }

  void head(const void *, void *g, StepCtx &c) override {
    fill_f32(c.s, int64_t(gslot_bytes / 4), static_cast<float *>(g), 0.f);
    c.launches += 1;
  }

  // the loss: every step's rows are in place once each unit has run its kept
  // forward, i.e. after the last backward
  void end_step(StepCtx &c) override {
    loss_reduce(c.s, int64_t(T) * B, Kf(c, k_lossrows), 1.0f / (float(T) * float(B)), Kf(c, k_loss));
    c.launches += 1;
  }

  const float *loss_ptr(const StepCtx &c) const override {
    return reinterpret_cast<const float *>(c.ks + k_loss);
  }
};

}  // namespace

std::unique_ptr<Net> make_lstm_net(const ckpt_net_desc &d) {
  if (d.batch <= 0 || d.depth <= 0 || d.width <= 0 || d.image <= 0 || d.n_classes <= 0 ||
      d.grad_chunk < 0)
    fail(CKPT_E_INVALID, "net_create: LSTM needs positive batch, steps, hidden, input and vocabulary");
  if (d.width % 8 != 0 || d.image % 8 != 0 || d.n_classes % 8 != 0)
    fail(CKPT_E_UNSUPPORTED, "net_create: LSTM sizes must be multiples of 8");
  if (d.n_classes > 16384)
    fail(CKPT_E_UNSUPPORTED, "net_create: LSTM vocabulary above 16384");
  if (int64_t(d.depth) * d.batch * d.image > (int64_t(1) << 31) ||
      int64_t(d.batch) * d.n_classes * 32 > (int64_t(1) << 31))
    fail(CKPT_E_INVALID, "net_create: LSTM tensors too large");
  return std::make_unique<LstmNet>(d);
}

}  // namespace ckpt
