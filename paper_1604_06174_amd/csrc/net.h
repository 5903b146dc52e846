// Unit chains: static layout tables, parameter layout and per-unit launchers.
#pragma once

#include <hip/hip_runtime.h>

#include <algorithm>
#include <memory>
#include <string>
#include <vector>

#include "common.h"
#include "launch.h"

namespace ckpt {

// Optional HIP-event timing of one kernel family (the net's dominant kernel):
// every launch of the family is bracketed by an event pair on its stream;
// durations are read back (synchronising) only when the totals are requested.
struct KernelTimer {
  bool enabled = false;
  std::vector<std::pair<hipEvent_t, hipEvent_t>> pool;
  std::vector<double> fl, by;
  std::vector<double> lt, lf, lb;  // every harvested launch: ms, flops, bytes
  size_t used = 0;
  uint64_t launches = 0;
  double ms = 0, flops = 0, bytes = 0;
  // time during which at least one launch of the family ran (the union of
  // their intervals; below the summed durations when launches on two streams
  // overlap)
  double busy = 0;

  // begin arms an event pair for the next launch of the timed family (see
  // launch.h: the launch itself stamps the pair with the kernel's start and
  // end); end books the launch's algorithmic work when one took the pair
  void begin(hipStream_t) {
    if (!enabled) return;
    if (used == pool.size()) {
      hipEvent_t a, b;
      if (hipEventCreate(&a) != hipSuccess) fail(CKPT_E_HIP, "hipEventCreate failed");
      if (hipEventCreate(&b) != hipSuccess) fail(CKPT_E_HIP, "hipEventCreate failed");
      pool.emplace_back(a, b);
    }
    TimedLaunch &t = timed_launch();
    t.start = pool[used].first;
    t.stop = pool[used].second;
    t.armed = true;
    t.taken = false;
  }
  void end(hipStream_t, double f, double b) {
    if (!enabled) return;
    TimedLaunch &t = timed_launch();
    if (t.taken) {
      fl.push_back(f);
      by.push_back(b);
      ++used;
    }
    t.armed = t.taken = false;
  }
  void harvest() {
    std::vector<std::pair<double, double>> iv;  // intervals from the first start (ms)
    iv.reserve(used);
    for (size_t k = 0; k < used; ++k) {
      float t = 0.f, a = 0.f;
      if (hipEventSynchronize(pool[k].second) != hipSuccess ||
          hipEventElapsedTime(&t, pool[k].first, pool[k].second) != hipSuccess ||
          hipEventElapsedTime(&a, pool[0].first, pool[k].first) != hipSuccess)
        fail(CKPT_E_HIP, "kernel timing: event query failed");
      iv.emplace_back(double(a), double(a) + double(t));
      ms += t;
      flops += fl[k];
      bytes += by[k];
      lt.push_back(t);
      lf.push_back(fl[k]);
      lb.push_back(by[k]);
      ++launches;
    }
    std::sort(iv.begin(), iv.end());
    double end = -1e300;
    for (const auto &v : iv) {
      if (v.first >= end) {
        busy += v.second - v.first;
        end = v.second;
      } else if (v.second > end) {
        busy += v.second - end;
        end = v.second;
      }
    }
    used = 0;
    fl.clear();
    by.clear();
  }
  void reset() {
    harvest();
    launches = 0;
    ms = flops = bytes = busy = 0;
    lt.clear();
    lf.clear();
    lb.clear();
  }
  // summed max(flops / pf, bytes / pb) over the harvested launches, in ms
  double roofline_ms(double pf, double pb) {
    harvest();
    double r = 0;
    for (size_t k = 0; k < lt.size(); ++k) r += std::max(lf[k] / pf, lb[k] / pb) * 1e3;
    return r;
  }
  ~KernelTimer() {
    for (auto &e : pool) {
      (void)hipEventDestroy(e.first);
      (void)hipEventDestroy(e.second);
    }
  }
};

// A second stream for work that can run beside a unit's chain of data
// gradients (its weight gradients), ordered with the step's stream by
// events.  Created, outside any stream capture, by the first step that may use
// it, on the device of that step's stream; a later step whose stream is on
// another device runs everything on its own stream.
struct SideStream {
  bool wanted = true;  // the net's owner allows it (net_set_side_stream)
  hipStream_t s = nullptr;
  hipEvent_t to_side = nullptr, to_main = nullptr, mark = nullptr, mark2 = nullptr;
  int dev = -1;
  void create(int device) {
    hipStream_t t = nullptr;
    hipEvent_t a = nullptr, b = nullptr, m = nullptr, m2 = nullptr;
    // the events only order the two streams' kernels on this device (each
    // kernel's own completion already releases its writes to device scope):
    // no timing, and a device-scope release instead of a system-scope one
    const unsigned ef = hipEventDisableTiming | hipEventReleaseToDevice;
    hipError_t e = hipStreamCreateWithFlags(&t, hipStreamNonBlocking);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&a, ef);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&b, ef);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&m, ef);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&m2, ef);
    if (e != hipSuccess) {
      if (m2) (void)hipEventDestroy(m2);
      if (m) (void)hipEventDestroy(m);
      if (b) (void)hipEventDestroy(b);
      if (a) (void)hipEventDestroy(a);
      if (t) (void)hipStreamDestroy(t);
      fail(CKPT_E_HIP, std::string("side stream: ") + hipGetErrorString(e));
    }
    s = t, to_side = a, to_main = b, mark = m, mark2 = m2, dev = device;
  }
  ~SideStream() {
    if (mark2) (void)hipEventDestroy(mark2);
    if (mark) (void)hipEventDestroy(mark);
    if (to_main) (void)hipEventDestroy(to_main);
    if (to_side) (void)hipEventDestroy(to_side);
    if (s) (void)hipStreamDestroy(s);
  }
};

// Work enqueued on `after` from here on waits for all work enqueued on
// `before` so far (an event recorded on one, waited for by the other).
inline void order_streams(hipStream_t before, hipStream_t after, hipEvent_t e) {
  hipError_t r = hipEventRecord(e, before);
  if (r == hipSuccess) r = hipStreamWaitEvent(after, e, 0);
  if (r != hipSuccess) fail(CKPT_E_HIP, std::string("stream ordering: ") + hipGetErrorString(r));
}

// Everything a unit launcher needs besides its own tensors.
struct StepCtx {
  hipStream_t s = nullptr;
  // the net's side stream for this step (null: everything on s) and its events
  hipStream_t side = nullptr;
  hipEvent_t ev_side = nullptr, ev_main = nullptr, ev_mark = nullptr, ev_mark2 = nullptr;
  bool recursive = false;          // the step runs a recursive plan
  mutable bool side_busy = false;  // side work enqueued since the last to_main
  mutable bool mark2_set = false;  // mark2_side recorded since the last to_main
  // stream of weight-gradient work, and the orderings around it: to_side
  // before side work that reads what s has written; to_main before s writes
  // what side work still reads; mark_side (mark2_side) then main_after_mark
  // (main_after_mark2) to order s behind only the side work enqueued before
  // the mark
  hipStream_t ws() const { return side ? side : s; }
  void to_side() const {
    if (!side) return;
    order_streams(s, side, ev_side);
    side_busy = true;
  }
  void to_main() const {
    if (!side || !side_busy) return;
    order_streams(side, s, ev_main);
    side_busy = mark2_set = false;
  }
  void mark2_side() const {
    if (!side) return;
    const hipError_t r = hipEventRecord(ev_mark2, side);
    if (r != hipSuccess) fail(CKPT_E_HIP, std::string("stream ordering: ") + hipGetErrorString(r));
    mark2_set = true;
  }
  void main_after_mark2() const {
    if (!side || !mark2_set) return;
    const hipError_t r = hipStreamWaitEvent(s, ev_mark2, 0);
    if (r != hipSuccess) fail(CKPT_E_HIP, std::string("stream ordering: ") + hipGetErrorString(r));
  }
  void mark_side() const {
    if (!side) return;
    const hipError_t r = hipEventRecord(ev_mark, side);
    if (r != hipSuccess) fail(CKPT_E_HIP, std::string("stream ordering: ") + hipGetErrorString(r));
  }
  void main_after_mark() const {
    if (!side) return;
    const hipError_t r = hipStreamWaitEvent(s, ev_mark, 0);
    if (r != hipSuccess) fail(CKPT_E_HIP, std::string("stream ordering: ") + hipGetErrorString(r));
  }
  const float *params = nullptr;  // device, net.param_bytes
  float *grads = nullptr;         // device, net.param_bytes
  const void *input = nullptr;    // device, batch input
  const void *target = nullptr;   // device, batch targets
  char *ks = nullptr;             // device operator workspace (net.ks_bytes)
  char *gextra = nullptr;         // device fixed gradient buffers (net.grad_extra)
  // device unit gradient scratch (the largest q_i): in use only inside a
  // unit's backward, so a unit's forward may keep transient tensors there
  char *q = nullptr;
  uint64_t launches = 0;
  // false while a forward sweep runs whose saved internals are discarded
  // (they are formed again by the unit's re-run before its backward)
  bool keep_saved = true;
  // true when this unit has already run a forward in this step (from the
  // same input bits): per-unit reductions computed then, such as batch-norm
  // statistics kept in operator workspace, may be reused
  bool rerun = false;
};

class Net {
 public:
  struct Tensor {
    std::string name;
    uint64_t off, numel;
  };

  ckpt_net_desc desc{};
  int32_t n = 0;
  std::vector<uint64_t> b, a, q;  // b[n+1], a[n], q[n]: 256-byte aligned bytes
  std::vector<Tensor> params;
  uint64_t param_bytes = 0;
  uint64_t ks_bytes = 0;          // operator workspace (not part of the peak)
  uint64_t gslot_bytes = 0;       // one gradient slot (0: the largest boundary)
  uint64_t grad_extra = 0;        // fixed gradient buffers (part of the peak)
  KernelTimer timer;              // times `timed_family` launches when enabled
  bool uses_side = false;         // its backward can run work on a side stream
  SideStream side;
  std::string timed_family;       // kernel-name prefix of the timed family

  virtual ~Net() = default;

  // Unit i forward: x (x_i) -> y (x_{i+1}); saved internals written to `saved`.
  // Every unit runs exactly one forward with c.keep_saved set before its
  // backward; a forward with it clear may leave out work whose only results
  // are saved internals (and loss terms, which the kept forward then adds),
  // and a kept forward may leave such work to fwd_segment.
  virtual void fwd(int32_t i, const void *x, void *y, void *saved, StepCtx &c) = 0;
  // Unit i backward: g = dL/dx_{i+1} -> dx = dL/dx_i (dx is null for unit 0),
  // reading x, y and saved; q is the unit's gradient scratch.  Writes unit i's
  // parameter gradients.
  virtual void bwd(int32_t i, const void *g, void *dx, const void *x, const void *y,
                   const void *saved, void *q, StepCtx &c) = 0;
  // Called after a kept forward of units [lo, hi) into the arena (unit lo + k's
  // saved internals at saved[k], its output at out[k]) and before their
  // backwards: work of those units that their forwards leave to be done for
  // all of them at once, in no order across the units (products batched over
  // the units).
  virtual void fwd_segment(int32_t, int32_t, const std::vector<void *> &, const std::vector<void *> &,
                           StepCtx &) {}
  // Called once at the start of every step, before any unit runs, and once at
  // its end, after the last backward.
  virtual void begin_step(StepCtx &) {}
  virtual void end_step(StepCtx &) {}
  // Head: x_n -> g = dL/dx_n (+ head parameter gradients), loss into ks.
  virtual void head(const void *xn, void *g, StepCtx &c) = 0;
  // Device address of the f32 loss after the step.
  virtual const float *loss_ptr(const StepCtx &c) const = 0;

  // ---- node-granularity graph (nets that provide one): nodes in a
  // topological order with their inputs (CSR), output bytes and CKPT_NODE_*
  // flags, the form graph_plan takes.
  struct NodeGraph {
    std::vector<int32_t> ptr, idx, flags;
    std::vector<uint64_t> bytes;
  };
  virtual bool node_graph(NodeGraph &) const { return false; }
  // Forward operator of node v: its inputs (in order) -> out.
  virtual void node_fwd(int32_t, const std::vector<const void *> &, void *, StepCtx &) {}
  // Backward operator of node v: dy = dL/d(v's output) (null for the loss
  // node), y = v's output (when its backward reads it), ins = v's inputs
  // (when read) -> out = the gradients of v's inputs, concatenated in input
  // order.  Writes v's parameter gradients.
  virtual void node_bwd(int32_t, const void *, const void *, const std::vector<const void *> &, void *,
                        StepCtx &) {}

  const float *P(const StepCtx &c, int k) const { return c.params + params[size_t(k)].off / 4; }
  float *G(const StepCtx &c, int k) const { return c.grads + params[size_t(k)].off / 4; }

  Accounting accounting(const Plan &p) const { return account(p, b, a, q, gslot_bytes, grad_extra); }
  uint64_t slot_bytes() const {
    if (gslot_bytes) return gslot_bytes;
    uint64_t m = 0;
    for (size_t i = 1; i < b.size(); ++i) m = b[i] > m ? b[i] : m;
    return m;
  }

 protected:
  int add_param(const std::string &name, uint64_t numel) {
    params.push_back({name, param_bytes, numel});
    param_bytes += align256(numel * 4);
    return int(params.size()) - 1;
  }
};

std::unique_ptr<Net> make_mlp_net(const ckpt_net_desc &d);
std::unique_ptr<Net> make_resnet_basic_net(const ckpt_net_desc &d);
std::unique_ptr<Net> make_lstm_net(const ckpt_net_desc &d);
std::unique_ptr<Net> make_resnet_bottleneck_net(const ckpt_net_desc &d);

}  // namespace ckpt
