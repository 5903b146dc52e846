// The checkpointed training step on one HIP stream.
//
// One-level plans follow Alg. 1 (section 4.1): a forward sweep keeps only the
// boundaries at the plan's cuts; the head gives g = dL/dx_n; then each segment,
// last to first, is re-run from its kept input into the arena (Alg. 1's
// localtemp) and back-propagated unit by unit.  With keep_last the final
// segment's first forward already writes the localtemp layout and is not
// re-run.
//
// RECURSIVE follows section 4.4 with k stored splits per level: the first
// sweep keeps the top-level split boundaries; a range [lo, hi) of length > 1
// runs forward from its input up to its last split point, pushing each split
// boundary on the checkpoint stack, then handles its parts last to first,
// popping each boundary after its part; a single unit is re-run and
// back-propagated.
//
// Workspace layout (each region 256-byte aligned, sizes from the planner's
// accounting so that the reported peak is exactly what is used):
//   [ CKPT | ARENA | GRAD (slot0 | slot1 | q) | operator workspace ]
// Forward sweeps place a unit's input and output at opposite ends of the arena
// (inputs that live in CKPT or are the network input stay where they are), so
// a sweep needs at most b_i + a_i + b_{i+1}.  A re-run segment stacks, per
// unit, its saved internals followed by its output.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "kernels.h"
#include "net.h"

namespace ckpt {
namespace {

enum Where { EXTERNAL, BOTTOM, TOP };

struct Exec {
  Net &net;
  StepCtx &c;
  const Accounting &acc;
  char *ckpt, *arena, *gslot[2], *qbuf;
  int cur = 0;                  // gradient slot holding dL/dx of the current unit
  uint64_t fwd_count = 0, bwd_count = 0;
  std::vector<char> ran = std::vector<char>(size_t(net.n), 0);  // unit has run a forward this step

  // Forward sweep over [lo, hi) starting from x (outside the arena).  Units
  // listed in `stored` write their output to the given address instead of the
  // arena.  Returns the address of x_hi.
  template <class StoreAt>
  const void *sweep(int32_t lo, int32_t hi, const void *x, StoreAt store_at) {
    Where pos = EXTERNAL;
    const void *cur_x = x;
    const uint64_t A = acc.arena;
    for (int32_t i = lo; i < hi; ++i) {
      void *dst = store_at(i);
      const uint64_t bi = net.b[size_t(i)], ai = net.a[size_t(i)], bo = net.b[size_t(i) + 1];
      void *saved;
      void *y;
      Where next;
      if (pos == BOTTOM) {
        saved = arena + bi;
        y = dst ? dst : arena + (A - bo);
        next = dst ? EXTERNAL : TOP;
      } else if (pos == TOP) {
        if (dst) {
          saved = arena;
        } else {
          saved = arena + bo;
        }
        y = dst ? dst : arena;
        next = dst ? EXTERNAL : BOTTOM;
      } else {  // EXTERNAL input
        saved = dst ? arena : arena + bo;
        y = dst ? dst : arena;
        next = dst ? EXTERNAL : BOTTOM;
      }
      (void)ai;
      c.keep_saved = false;
      c.rerun = ran[size_t(i)] != 0;
      net.fwd(i, cur_x, y, saved, c);
      ran[size_t(i)] = 1;
      c.rerun = false;
      c.keep_saved = true;
      ++fwd_count;
      cur_x = y;
      pos = next;
    }
    return cur_x;
  }

  // Re-run [lo, hi) from x into the arena's localtemp layout; fills the
  // per-unit saved/output addresses, then lets the net finish the segment's
  // kept forwards together.
  void localtemp(int32_t lo, int32_t hi, const void *x, std::vector<void *> &saved,
                 std::vector<void *> &out) {
    saved.assign(size_t(hi - lo), nullptr);
    out.assign(size_t(hi - lo), nullptr);
    uint64_t off = 0;
    const void *cur_x = x;
    for (int32_t i = lo; i < hi; ++i) {
      void *s = arena + off;
      void *y = arena + off + net.a[size_t(i)];
      off += net.a[size_t(i)] + net.b[size_t(i) + 1];
      c.rerun = ran[size_t(i)] != 0;
      net.fwd(i, cur_x, y, s, c);
      ran[size_t(i)] = 1;
      c.rerun = false;
      ++fwd_count;
      saved[size_t(i - lo)] = s;
      out[size_t(i - lo)] = y;
      cur_x = y;
    }
    net.fwd_segment(lo, hi, saved, out, c);
  }

  void backward_segment(int32_t lo, int32_t hi, const void *x, const std::vector<void *> &saved,
                        const std::vector<void *> &out) {
    for (int32_t i = hi - 1; i >= lo; --i) {
      const void *xi = (i == lo) ? x : out[size_t(i - lo - 1)];
      void *dx = (i > 0) ? gslot[cur ^ 1] : nullptr;
      net.bwd(i, gslot[cur], dx, xi, out[size_t(i - lo)], saved[size_t(i - lo)], qbuf, c);
      ++bwd_count;
      cur ^= 1;
    }
  }

  void one_level(const Plan &p, const void *x0) {
    auto segs = p.segments();
    const size_t K = segs.size();
    std::vector<char *> kept(K, nullptr);  // input of segment k (kept[0] = x0)
    {
      uint64_t off = 0;
      for (size_t k = 1; k < K; ++k) {
        kept[k] = ckpt + off;
        off += net.b[size_t(segs[k].first)];
      }
    }
    const int32_t fwd_hi = p.keep_last ? segs.back().first : p.n;
    // segment index of each stored output: unit segs[k].second - 1 -> kept[k+1]
    auto store_at = [&](int32_t i) -> void * {
      for (size_t k = 0; k + 1 < K; ++k)
        if (segs[k].second - 1 == i) return kept[k + 1];
      return nullptr;
    };
    std::vector<void *> last_saved, last_out;
    const void *xn = x0;
    if (fwd_hi > 0) xn = sweep(0, fwd_hi, x0, store_at);
    if (p.keep_last) {
      const auto &s = segs.back();
      const void *xin = (K == 1) ? x0 : kept[K - 1];
      localtemp(s.first, s.second, xin, last_saved, last_out);
      xn = last_out.back();
    }
    net.head(xn, gslot[0], c);
    cur = 0;
    for (size_t k = K; k-- > 0;) {
      const auto &s = segs[k];
      const void *xin = (k == 0) ? x0 : kept[k];
      std::vector<void *> saved, out;
      if (p.keep_last && k == K - 1) {
        saved = last_saved;
        out = last_out;
      } else {
        localtemp(s.first, s.second, xin, saved, out);
      }
      backward_segment(s.first, s.second, xin, saved, out);
    }
  }

  uint64_t stack_top = 0;

  int32_t fanout = 1;

  // Forward [lo, sweep_hi) from x keeping the split boundaries of [lo, hi)
  // on the checkpoint stack; returns x_{sweep_hi} and the boundaries' slots.
  const void *push_splits(int32_t lo, int32_t hi, int32_t sweep_hi, const void *x,
                          std::vector<int32_t> &s, std::vector<char *> &slot) {
    s = rec_splits(lo, hi, fanout);
    slot.resize(s.size());
    for (size_t t = 0; t < s.size(); ++t) {
      slot[t] = ckpt + stack_top;
      stack_top += net.b[size_t(s[t])];
    }
    return sweep(lo, sweep_hi, x, [&](int32_t i) -> void * {
      auto it = std::lower_bound(s.begin(), s.end(), i + 1);
      return (it != s.end() && *it == i + 1) ? slot[size_t(it - s.begin())] : nullptr;
    });
  }

  // the parts of [lo, hi), last to first; each split boundary is popped once
  // its part is done
  void parts(int32_t lo, int32_t hi, const void *x, const std::vector<int32_t> &s,
             const std::vector<char *> &slot) {
    for (size_t t = s.size() + 1; t-- > 0;) {
      const int32_t p_lo = t == 0 ? lo : s[t - 1], p_hi = t == s.size() ? hi : s[t];
      rec(p_lo, p_hi, t == 0 ? x : slot[t - 1]);
      if (t > 0) stack_top -= net.b[size_t(s[t - 1])];
    }
  }

  void rec(int32_t lo, int32_t hi, const void *x) {
    if (hi - lo == 1) {
      std::vector<void *> saved, out;
      localtemp(lo, hi, x, saved, out);
      backward_segment(lo, hi, x, saved, out);
      return;
    }
    std::vector<int32_t> s;
    std::vector<char *> slot;
    push_splits(lo, hi, rec_splits(lo, hi, fanout).back(), x, s, slot);
    parts(lo, hi, x, s, slot);
  }

  void recursive(const Plan &p, const void *x0) {
    const int32_t n = p.n;
    fanout = p.fanout;
    stack_top = 0;
    if (n == 1) {
      const void *xn = sweep(0, 1, x0, [](int32_t) -> void * { return nullptr; });
      net.head(xn, gslot[0], c);
      cur = 0;
      rec(0, 1, x0);
      return;
    }
    std::vector<int32_t> s;
    std::vector<char *> slot;
    const void *xn = push_splits(0, n, n, x0, s, slot);  // the first forward: the whole chain
    net.head(xn, gslot[0], c);
    cur = 0;
    parts(0, n, x0, s, slot);
  }
};

}  // namespace

// device of stream s (the current device for the null stream)
hipError_t stream_device(hipStream_t s, int *d) { return s ? hipStreamGetDevice(s, d) : hipGetDevice(d); }

void prepare_side(Net &net, hipStream_t s) {
  if (!net.uses_side || !net.side.wanted || net.side.s) return;
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  int d = -1, cur = -1;
  if (hipStreamIsCapturing(s, &cs) != hipSuccess || cs != hipStreamCaptureStatusNone ||
      stream_device(s, &d) != hipSuccess || hipGetDevice(&cur) != hipSuccess || d != cur) {
    (void)hipGetLastError();  // no side stream: the step runs on its own stream
    return;
  }
  net.side.create(d);
}

uint64_t workspace_bytes(const Net &net, const Accounting &acc) {
  return align256(acc.ckpt) + align256(acc.arena) + align256(acc.grad) + align256(net.ks_bytes);
}

void run_train_step(Net &net, const float *params, float *grads, const ckpt_batch &batch,
                    const Plan &p, char *ws, uint64_t ws_bytes, hipStream_t s, float *loss_dev,
                    float *loss_host, uint64_t *peak, ckpt_step_stats *stats) {
  Accounting acc = net.accounting(p);
  const uint64_t need = workspace_bytes(net, acc);
  if (ws_bytes < need)
    fail(CKPT_E_WORKSPACE, "train_step: workspace has " + std::to_string(ws_bytes) +
                               " bytes, the plan needs " + std::to_string(need));
  StepCtx c;
  c.s = s;
  c.params = params;
  c.grads = grads;
  c.input = batch.input;
  c.target = batch.target;
  char *ckpt = ws;
  char *arena = ckpt + align256(acc.ckpt);
  char *grad = arena + align256(acc.arena);
  c.ks = grad + align256(acc.grad);
  const uint64_t slot = net.slot_bytes();
  uint64_t maxq = 0;
  for (int32_t i = 0; i < net.n; ++i) maxq = std::max(maxq, net.q[size_t(i)]);
  c.gextra = grad + 2 * slot + maxq;
  c.q = grad + 2 * slot;

  if (net.uses_side && net.side.wanted && net.side.s) {
    int d = -1;
    if (stream_device(s, &d) == hipSuccess && d == net.side.dev) {
      c.side = net.side.s;
      c.ev_side = net.side.to_side;
      c.ev_main = net.side.to_main;
      c.ev_mark = net.side.mark;
      c.ev_mark2 = net.side.mark2;
    }
  }

  c.recursive = p.mode == CKPT_RECURSIVE;
  Exec e{net, c, acc, ckpt, arena, {grad, grad + slot}, grad + 2 * slot};
  (void)hipGetLastError();  // clear a stale error left by the caller
  net.begin_step(c);
  if (p.mode == CKPT_RECURSIVE)
    e.recursive(p, batch.input);
  else
    e.one_level(p, batch.input);
  c.to_main();  // the weight gradients the last backward left on the side stream
  net.end_step(c);
  if (loss_dev) {
    copy_scalar(s, net.loss_ptr(c), loss_dev);
    ++c.launches;
  }
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) fail(CKPT_E_HIP, std::string("train_step: ") + hipGetErrorString(err));
  if (loss_host) {
    err = hipMemcpyAsync(loss_host, net.loss_ptr(c), sizeof(float), hipMemcpyDeviceToHost, s);
    if (err == hipSuccess) err = hipStreamSynchronize(s);
    if (err != hipSuccess) fail(CKPT_E_HIP, std::string("train_step: ") + hipGetErrorString(err));
  }
  if (peak) *peak = acc.peak();
  if (stats) {
    stats->unit_forwards = e.fwd_count;
    stats->unit_backwards = e.bwd_count;
    stats->kernel_launches = c.launches;
    stats->ckpt_bytes = acc.ckpt;
    stats->arena_bytes = acc.arena;
    stats->grad_bytes = acc.grad;
  }
}

}  // namespace ckpt
