// extern "C" boundary of libckpt: argument validation, error codes and the
// thread-local error message.  Nothing here launches work before every
// argument has been checked.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>
#include <memory>

#include "capi_internal.h"
#include "net.h"

namespace ckpt {
uint64_t graph_workspace_bytes(const Net &net, const GraphPlan &p);
void run_graph_step(Net &net, const float *params, float *grads, const ckpt_batch &batch,
                    const GraphPlan &p, char *ws, uint64_t ws_bytes, hipStream_t s, float *loss_dev,
                    float *loss_host, uint64_t *peak, ckpt_step_stats *stats);
}  // namespace ckpt

namespace {
thread_local std::string g_err;
}  // namespace

void ckpt::set_last_error(const std::string &msg) { g_err = msg; }

extern "C" {

const char *ckpt_last_error(void) { return g_err.c_str(); }

int plan_checkpoints(int32_t n_layers, const uint64_t *layer_bytes, const uint64_t *cut_bytes,
                     uint64_t budget, int32_t mode, const int32_t *user_cuts, int32_t n_user_cuts,
                     int32_t flags, ckpt_plan **out) {
  return ckpt::guarded([&] {
    ckpt::need(out, "plan_checkpoints(out)");
    *out = nullptr;
    auto p = std::make_unique<ckpt_plan>();
    p->p = ckpt::make_plan(n_layers, layer_bytes, cut_bytes, budget, mode, user_cuts,
                           n_user_cuts, flags);
    *out = p.release();
  });
}

int plan_info(const ckpt_plan *plan, int32_t *mode, int32_t *n_layers, int32_t *n_cuts,
              uint64_t *x, uint64_t *y, uint64_t *extra) {
  return ckpt::guarded([&] {
    ckpt::need(plan, "plan_info");
    if (mode) *mode = plan->p.mode;
    if (n_layers) *n_layers = plan->p.n;
    if (n_cuts) *n_cuts = int32_t(plan->p.cuts.size());
    if (x) *x = plan->p.x;
    if (y) *y = plan->p.y;
    if (extra) *extra = plan->p.extra;
  });
}

int plan_cuts(const ckpt_plan *plan, int32_t *cuts, int32_t cap, int32_t *n_cuts) {
  return ckpt::guarded([&] {
    ckpt::need(plan, "plan_cuts");
    const auto &c = plan->p.cuts;
    if (n_cuts) *n_cuts = int32_t(c.size());
    if (cuts && cap > 0) std::memcpy(cuts, c.data(), sizeof(int32_t) * std::min<size_t>(size_t(cap), c.size()));
  });
}

int plan_serialize(const ckpt_plan *plan, uint8_t *buf, uint64_t cap, uint64_t *len) {
  return ckpt::guarded([&] {
    ckpt::need(plan, "plan_serialize");
    auto v = ckpt::serialize(plan->p);
    if (len) *len = v.size();
    if (buf) {
      if (cap < v.size()) ckpt::fail(CKPT_E_INVALID, "plan_serialize: buffer too small");
      std::memcpy(buf, v.data(), v.size());
    }
  });
}

void plan_free(ckpt_plan *plan) { delete plan; }

int plan_search(int32_t n_layers, const uint64_t *layer_bytes, const uint64_t *cut_bytes,
                const uint64_t *b, const uint64_t *a, const uint64_t *q, uint64_t grad_slot,
                uint64_t grad_extra, int32_t flags, ckpt_plan **out, uint64_t *budget,
                uint64_t *peak) {
  return ckpt::guarded([&] {
    ckpt::need(out, "plan_search(out)");
    *out = nullptr;
    if (n_layers <= 0) ckpt::fail(CKPT_E_INVALID, "plan_search: n_layers must be positive");
    ckpt::need(layer_bytes, "plan_search(layer_bytes)");
    ckpt::need(cut_bytes, "plan_search(cut_bytes)");
    ckpt::need(b, "plan_search(b)");
    ckpt::need(a, "plan_search(a)");
    ckpt::need(q, "plan_search(q)");
    const size_t n = size_t(n_layers);
    std::vector<uint64_t> bv(b, b + n + 1), av(a, a + n), qv(q, q + n);
    auto p = std::make_unique<ckpt_plan>();
    p->p = ckpt::search_plan(n_layers, layer_bytes, cut_bytes, bv, av, qv, grad_slot, grad_extra,
                             flags, budget, peak);
    *out = p.release();
  });
}

int graph_plan(int32_t n_nodes, const int32_t *pred_ptr, const int32_t *pred_idx,
               const uint64_t *out_bytes, const int32_t *flags, const int32_t *mirror,
               int32_t strategy, ckpt_graph_plan **out) {
  return ckpt::guarded([&] {
    ckpt::need(out, "graph_plan(out)");
    *out = nullptr;
    auto p = std::make_unique<ckpt_graph_plan>();
    p->p = ckpt::make_graph_plan(n_nodes, pred_ptr, pred_idx, out_bytes, flags, mirror, strategy);
    *out = p.release();
  });
}

int graph_plan_info(const ckpt_graph_plan *plan, int32_t *n_exec, int32_t *n_mirror,
                    int32_t *n_blocks, uint64_t *peak_bytes) {
  return ckpt::guarded([&] {
    ckpt::need(plan, "graph_plan_info");
    if (n_exec) *n_exec = int32_t(plan->p.order.size());
    if (n_mirror) *n_mirror = plan->p.n_mirror;
    if (n_blocks) *n_blocks = int32_t(plan->p.tag_bytes.size());
    if (peak_bytes) *peak_bytes = plan->p.peak;
  });
}

int graph_plan_schedule(const ckpt_graph_plan *plan, int32_t *kind, int32_t *of, int32_t *block,
                        int32_t cap, int32_t *n_exec) {
  return ckpt::guarded([&] {
    ckpt::need(plan, "graph_plan_schedule");
    if (cap < 0) ckpt::fail(CKPT_E_INVALID, "graph_plan_schedule: negative cap");
    const auto &p = plan->p;
    if (n_exec) *n_exec = int32_t(p.order.size());
    const size_t k = std::min(size_t(cap), p.order.size());
    for (size_t i = 0; i < k; ++i) {
      const int32_t w = p.order[i];
      if (kind) kind[i] = p.nodes[size_t(w)].kind;
      if (of) of[i] = p.nodes[size_t(w)].of;
      if (block) block[i] = p.tag_of[size_t(w)];
    }
  });
}

int graph_plan_blocks(const ckpt_graph_plan *plan, uint64_t *bytes, int32_t cap, int32_t *n_blocks) {
  return ckpt::guarded([&] {
    ckpt::need(plan, "graph_plan_blocks");
    if (cap < 0) ckpt::fail(CKPT_E_INVALID, "graph_plan_blocks: negative cap");
    const auto &tb = plan->p.tag_bytes;
    if (n_blocks) *n_blocks = int32_t(tb.size());
    if (bytes)
      for (size_t i = 0; i < std::min(size_t(cap), tb.size()); ++i) bytes[i] = tb[i];
  });
}

void graph_plan_free(ckpt_graph_plan *plan) { delete plan; }

int net_create(const ckpt_net_desc *desc, ckpt_net **out) {
  return ckpt::guarded([&] {
    ckpt::need(desc, "net_create(desc)");
    ckpt::need(out, "net_create(out)");
    *out = nullptr;
    for (int32_t r : desc->reserved)
      if (r != 0) ckpt::fail(CKPT_E_INVALID, "net_create: reserved fields must be zero");
    if (desc->kind != CKPT_NET_LSTM && desc->grad_chunk != 0)
      ckpt::fail(CKPT_E_INVALID, "net_create: grad_chunk applies to LSTM only");
    if (desc->kind != CKPT_NET_RESNET_BOTTLENECK &&
        (desc->stage_blocks[0] | desc->stage_blocks[1] | desc->stage_blocks[2] |
         desc->stage_blocks[3] | desc->expansion | desc->stem_channels) != 0)
      ckpt::fail(CKPT_E_INVALID,
                 "net_create: stage_blocks, expansion and stem_channels apply to RESNET_BOTTLENECK only");
    if (desc->drop_bn_relu != 0 &&
        ((desc->kind != CKPT_NET_RESNET_BASIC && desc->kind != CKPT_NET_RESNET_BOTTLENECK) ||
         desc->drop_bn_relu != 1))
      ckpt::fail(CKPT_E_INVALID,
                 "net_create: drop_bn_relu is 0 or 1 and applies to RESNET_BASIC and RESNET_BOTTLENECK only");
    auto h = std::make_unique<ckpt_net>();
    switch (desc->kind) {
      case CKPT_NET_MLP: h->net = ckpt::make_mlp_net(*desc); break;
      case CKPT_NET_RESNET_BASIC: h->net = ckpt::make_resnet_basic_net(*desc); break;
      case CKPT_NET_LSTM: h->net = ckpt::make_lstm_net(*desc); break;
      case CKPT_NET_RESNET_BOTTLENECK: h->net = ckpt::make_resnet_bottleneck_net(*desc); break;
      default: ckpt::fail(CKPT_E_INVALID, "net_create: unknown network kind");
    }
    *out = h.release();
  });
}

void net_destroy(ckpt_net *net) { delete net; }

int net_units(const ckpt_net *net, int32_t *n) {
  return ckpt::guarded([&] {
    ckpt::need(net, "net_units");
    ckpt::need(n, "net_units(n)");
    *n = net->net->n;
  });
}

int net_unit_sizes(const ckpt_net *net, uint64_t *b, uint64_t *a, uint64_t *q) {
  return ckpt::guarded([&] {
    ckpt::need(net, "net_unit_sizes");
    const auto &N = *net->net;
    if (b) std::memcpy(b, N.b.data(), N.b.size() * 8);
    if (a) std::memcpy(a, N.a.data(), N.a.size() * 8);
    if (q) std::memcpy(q, N.q.data(), N.q.size() * 8);
  });
}

int net_grad_bytes(const ckpt_net *net, uint64_t *slot, uint64_t *extra) {
  return ckpt::guarded([&] {
    ckpt::need(net, "net_grad_bytes");
    if (slot) *slot = net->net->slot_bytes();
    if (extra) *extra = net->net->grad_extra;
  });
}

int net_layer_sizes(const ckpt_net *net, uint64_t *layer_bytes, uint64_t *cut_bytes) {
  return ckpt::guarded([&] {
    ckpt::need(net, "net_layer_sizes");
    const auto &N = *net->net;
    for (int32_t i = 0; i < N.n; ++i) {
      if (layer_bytes) layer_bytes[i] = N.a[size_t(i)] + N.b[size_t(i) + 1];
      if (cut_bytes) cut_bytes[i] = (i + 1 < N.n) ? N.b[size_t(i) + 1] : 0;
    }
  });
}

int net_param_bytes(const ckpt_net *net, uint64_t *bytes) {
  return ckpt::guarded([&] {
    ckpt::need(net, "net_param_bytes");
    ckpt::need(bytes, "net_param_bytes(bytes)");
    *bytes = net->net->param_bytes;
  });
}

int net_param_count(const ckpt_net *net, int32_t *count) {
  return ckpt::guarded([&] {
    ckpt::need(net, "net_param_count");
    ckpt::need(count, "net_param_count(count)");
    *count = int32_t(net->net->params.size());
  });
}

int net_param_info(const ckpt_net *net, int32_t k, char *name, int32_t cap, uint64_t *offset,
                   uint64_t *numel) {
  return ckpt::guarded([&] {
    ckpt::need(net, "net_param_info");
    const auto &ps = net->net->params;
    if (k < 0 || size_t(k) >= ps.size()) ckpt::fail(CKPT_E_INVALID, "net_param_info: bad index");
    const auto &t = ps[size_t(k)];
    if (name && cap > 0) {
      size_t nlen = std::min(size_t(cap - 1), t.name.size());
      std::memcpy(name, t.name.data(), nlen);
      name[nlen] = 0;
    }
    if (offset) *offset = t.off;
    if (numel) *numel = t.numel;
  });
}

int plan_accounting(const ckpt_net *net, const ckpt_plan *plan, uint64_t *ckpt_b, uint64_t *arena,
                    uint64_t *grad, uint64_t *peak) {
  return ckpt::guarded([&] {
    ckpt::need(net, "plan_accounting(net)");
    ckpt::need(plan, "plan_accounting(plan)");
    if (plan->p.n != net->net->n)
      ckpt::fail(CKPT_E_MISMATCH, "plan_accounting: plan n differs from the net's unit count");
    auto acc = net->net->accounting(plan->p);
    if (ckpt_b) *ckpt_b = acc.ckpt;
    if (arena) *arena = acc.arena;
    if (grad) *grad = acc.grad;
    if (peak) *peak = acc.peak();
  });
}

int net_workspace_bytes(const ckpt_net *net, const ckpt_plan *plan, uint64_t *bytes) {
  return ckpt::guarded([&] {
    ckpt::need(net, "net_workspace_bytes(net)");
    ckpt::need(plan, "net_workspace_bytes(plan)");
    ckpt::need(bytes, "net_workspace_bytes(bytes)");
    if (plan->p.n != net->net->n)
      ckpt::fail(CKPT_E_MISMATCH, "net_workspace_bytes: plan n differs from the net's unit count");
    auto acc = net->net->accounting(plan->p);
    *bytes = ckpt::workspace_bytes(*net->net, acc);
  });
}

int train_step(ckpt_net *net, const void *params, void *grads, const ckpt_batch *batch,
               const ckpt_plan *plan, void *workspace, uint64_t workspace_bytes, void *stream,
               float *loss_dev, float *loss_host, uint64_t *peak, ckpt_step_stats *stats) {
  return ckpt::guarded([&] {
    ckpt::check_step_args("train_step", net, params, grads, batch, plan, workspace);
    ckpt::prepare_side(*net->net, static_cast<hipStream_t>(stream));
    ckpt::run_train_step(*net->net, static_cast<const float *>(params), static_cast<float *>(grads),
                         *batch, plan->p, static_cast<char *>(workspace), workspace_bytes,
                         static_cast<hipStream_t>(stream), loss_dev, loss_host, peak, stats);
  });
}

int step_graph_create(ckpt_net *net, const void *params, void *grads, const ckpt_batch *batch,
                      const ckpt_plan *plan, void *workspace, uint64_t workspace_bytes,
                      void *stream, float *loss_dev, ckpt_step_graph **out,
                      ckpt_step_stats *stats) {
  return ckpt::guarded([&] {
    ckpt::need(out, "step_graph_create(out)");
    *out = nullptr;
    ckpt::check_step_args("step_graph_create", net, params, grads, batch, plan, workspace);
    if (!stream)
      ckpt::fail(CKPT_E_INVALID, "step_graph_create: capture needs a stream other than the default one");
    if (net->net->timer.enabled)
      ckpt::fail(CKPT_E_INVALID, "step_graph_create: turn kernel timing off before recording");
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    hipError_t e = hipStreamIsCapturing(s, &cs);
    if (e != hipSuccess)
      ckpt::fail(CKPT_E_HIP, std::string("step_graph_create: ") + hipGetErrorString(e));
    if (cs != hipStreamCaptureStatusNone)
      ckpt::fail(CKPT_E_INVALID, "step_graph_create: the stream is already being captured");
    auto g = std::make_unique<ckpt_step_graph>();
    ckpt::prepare_side(*net->net, s);  // before the capture: it creates a stream and events
    e = hipStreamBeginCapture(s, hipStreamCaptureModeThreadLocal);
    if (e != hipSuccess)
      ckpt::fail(CKPT_E_HIP, std::string("step_graph_create: ") + hipGetErrorString(e));
    try {
      ckpt::run_train_step(*net->net, static_cast<const float *>(params), static_cast<float *>(grads),
                           *batch, plan->p, static_cast<char *>(workspace), workspace_bytes, s,
                           loss_dev, nullptr, nullptr, stats);
    } catch (...) {
      hipGraph_t partial = nullptr;
      (void)hipStreamEndCapture(s, &partial);
      if (partial) (void)hipGraphDestroy(partial);
      throw;
    }
    e = hipStreamEndCapture(s, &g->graph);
    if (e == hipSuccess) e = hipGraphInstantiate(&g->exec, g->graph, nullptr, nullptr, 0);
    if (e != hipSuccess)
      ckpt::fail(CKPT_E_HIP, std::string("step_graph_create: ") + hipGetErrorString(e));
    *out = g.release();
  });
}

int step_graph_launch(ckpt_step_graph *graph, void *stream) {
  return ckpt::guarded([&] {
    ckpt::need(graph, "step_graph_launch(graph)");
    const hipError_t e = hipGraphLaunch(graph->exec, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) ckpt::fail(CKPT_E_HIP, std::string("step_graph_launch: ") + hipGetErrorString(e));
  });
}

void step_graph_free(ckpt_step_graph *graph) { delete graph; }

int net_node_graph(const ckpt_net *net, int32_t *n_nodes, int32_t *n_edges, int32_t *pred_ptr,
                   int32_t *pred_idx, uint64_t *out_bytes, int32_t *flags, int32_t cap_nodes,
                   int32_t cap_edges) {
  return ckpt::guarded([&] {
    ckpt::need(net, "net_node_graph");
    ckpt::Net::NodeGraph g;
    if (!net->net->node_graph(g))
      ckpt::fail(CKPT_E_UNSUPPORTED, "net_node_graph: this net has no node graph");
    const int32_t n = int32_t(g.bytes.size()), e = int32_t(g.idx.size());
    if (n_nodes) *n_nodes = n;
    if (n_edges) *n_edges = e;
    if (!pred_ptr && !pred_idx && !out_bytes && !flags) return;
    if (cap_nodes < n || cap_edges < e || !pred_ptr || !out_bytes || !flags || (e > 0 && !pred_idx))
      ckpt::fail(CKPT_E_INVALID, "net_node_graph: output arrays missing or too small");
    std::copy(g.ptr.begin(), g.ptr.end(), pred_ptr);
    std::copy(g.idx.begin(), g.idx.end(), pred_idx);
    std::copy(g.bytes.begin(), g.bytes.end(), out_bytes);
    std::copy(g.flags.begin(), g.flags.end(), flags);
  });
}

int graph_workspace_bytes(const ckpt_net *net, const ckpt_graph_plan *plan, uint64_t *bytes) {
  return ckpt::guarded([&] {
    ckpt::need(net, "graph_workspace_bytes(net)");
    ckpt::need(plan, "graph_workspace_bytes(plan)");
    ckpt::need(bytes, "graph_workspace_bytes(bytes)");
    *bytes = ckpt::graph_workspace_bytes(*net->net, plan->p);
  });
}

int train_step_graph(ckpt_net *net, const void *params, void *grads, const ckpt_batch *batch,
                     const ckpt_graph_plan *plan, void *workspace, uint64_t workspace_bytes,
                     void *stream, float *loss_dev, float *loss_host, uint64_t *peak,
                     ckpt_step_stats *stats) {
  return ckpt::guarded([&] {
    ckpt::need(net, "train_step_graph(net)");
    ckpt::need(params, "train_step_graph(params)");
    ckpt::need(grads, "train_step_graph(grads)");
    ckpt::need(batch, "train_step_graph(batch)");
    ckpt::need(batch->input, "train_step_graph(batch.input)");
    ckpt::need(batch->target, "train_step_graph(batch.target)");
    ckpt::need(plan, "train_step_graph(plan)");
    ckpt::need(workspace, "train_step_graph(workspace)");
    if (reinterpret_cast<uintptr_t>(workspace) & 255)
      ckpt::fail(CKPT_E_INVALID, "train_step_graph: workspace must be 256-byte aligned");
    if ((reinterpret_cast<uintptr_t>(params) & 255) || (reinterpret_cast<uintptr_t>(grads) & 255))
      ckpt::fail(CKPT_E_INVALID, "train_step_graph: params and grads must be 256-byte aligned");
    ckpt::run_graph_step(*net->net, static_cast<const float *>(params), static_cast<float *>(grads),
                         *batch, plan->p, static_cast<char *>(workspace), workspace_bytes,
                         static_cast<hipStream_t>(stream), loss_dev, loss_host, peak, stats);
  });
}

int net_set_side_stream(ckpt_net *net, int32_t enable) {
  return ckpt::guarded([&] {
    ckpt::need(net, "net_set_side_stream");
    net->net->side.wanted = enable != 0;
  });
}

int net_timing_enable(ckpt_net *net, int32_t enable) {
  return ckpt::guarded([&] {
    ckpt::need(net, "net_timing_enable");
    auto &t = net->net->timer;
    t.reset();
    t.enabled = enable != 0;
  });
}

int net_timing_read(ckpt_net *net, uint64_t *launches, double *ms, double *flops, double *bytes,
                    char *name, int32_t cap) {
  return ckpt::guarded([&] {
    ckpt::need(net, "net_timing_read");
    auto &t = net->net->timer;
    t.harvest();
    if (launches) *launches = t.launches;
    if (ms) *ms = t.ms;
    if (flops) *flops = t.flops;
    if (bytes) *bytes = t.bytes;
    if (name && cap > 0) {
      const std::string &f = net->net->timed_family;
      size_t k = std::min(size_t(cap - 1), f.size());
      std::memcpy(name, f.data(), k);
      name[k] = 0;
    }
  });
}

int net_timing_roofline(ckpt_net *net, double peak_flops, double peak_bytes_per_s,
                        double *roofline_ms, double *kernel_ms, double *busy_ms) {
  return ckpt::guarded([&] {
    ckpt::need(net, "net_timing_roofline");
    if (!(peak_flops > 0) || !(peak_bytes_per_s > 0))
      ckpt::fail(CKPT_E_INVALID, "net_timing_roofline: peaks must be positive");
    auto &t = net->net->timer;
    const double r = t.roofline_ms(peak_flops, peak_bytes_per_s);
    if (roofline_ms) *roofline_ms = r;
    if (kernel_ms) *kernel_ms = t.ms;
    if (busy_ms) *busy_ms = t.busy;
  });
}

}  // extern "C"
