// Training step over a node-granularity graph planned by graph_plan (Alg. 2
// with mirror nodes, memory blocks from the section-3 allocator), on one HIP
// stream.
//
// Workspace: the plan's memory blocks, each 256-byte aligned, in block order,
// then the net's operator workspace, then one scratch tensor for adding up
// the gradients of a node with several readers (operator workspace in the
// sense of section 5.1, not part of the planned bytes).  Nodes run in the
// plan's order: forward and mirror nodes apply their operator to their
// inputs' blocks; a gradient node first forms dL/d(output) of its forward
// node -- the slice of each reader's gradient output that belongs to this
// node, added in reader order -- then applies the node's backward operator.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "kernels.h"
#include "net.h"

namespace ckpt {

namespace {

void check_graph(const Net &net, const Net::NodeGraph &g, const GraphPlan &p) {
  const int32_t n = int32_t(g.bytes.size());
  if (p.n_forward != n || p.flags != g.flags)
    fail(CKPT_E_MISMATCH, "train_step_graph: the plan is not of this net's graph");
  for (int32_t v = 0; v < n; ++v) {
    const GraphNode &nd = p.nodes[size_t(v)];
    const std::vector<int32_t> ins(g.idx.begin() + g.ptr[size_t(v)], g.idx.begin() + g.ptr[size_t(v) + 1]);
    if (nd.kind != CKPT_GNODE_FORWARD || nd.of != v || nd.bytes != g.bytes[size_t(v)] || nd.inputs != ins ||
        nd.inplace != ((g.flags[size_t(v)] & CKPT_NODE_INPLACE) != 0))
      fail(CKPT_E_MISMATCH, "train_step_graph: the plan is not of this net's graph");
  }
  (void)net;
}

}  // namespace

uint64_t graph_workspace_bytes(const Net &net, const GraphPlan &p) {
  Net::NodeGraph g;
  if (!net.node_graph(g)) fail(CKPT_E_UNSUPPORTED, "graph plans: this net has no node graph");
  check_graph(net, g, p);
  uint64_t w = 0, scratch = 0;
  for (uint64_t b : p.tag_bytes) w += align256(b);
  for (uint64_t b : g.bytes) scratch = std::max(scratch, b);
  return w + align256(net.ks_bytes) + align256(scratch);
}

void run_graph_step(Net &net, const float *params, float *grads, const ckpt_batch &batch,
                    const GraphPlan &p, char *ws, uint64_t ws_bytes, hipStream_t s, float *loss_dev,
                    float *loss_host, uint64_t *peak, ckpt_step_stats *stats) {
  Net::NodeGraph g;
  if (!net.node_graph(g)) fail(CKPT_E_UNSUPPORTED, "train_step_graph: this net has no node graph");
  check_graph(net, g, p);
  const uint64_t need = graph_workspace_bytes(net, p);
  if (ws_bytes < need)
    fail(CKPT_E_WORKSPACE, "train_step_graph: workspace has " + std::to_string(ws_bytes) +
                               " bytes, the plan needs " + std::to_string(need));
  const int32_t n = int32_t(g.bytes.size());
  std::vector<char *> block(p.tag_bytes.size());
  uint64_t off = 0;
  for (size_t t = 0; t < p.tag_bytes.size(); ++t) {
    block[t] = ws + off;
    off += align256(p.tag_bytes[t]);
  }
  StepCtx c;
  c.s = s;
  c.params = params;
  c.grads = grads;
  c.input = batch.input;
  c.target = batch.target;
  c.ks = ws + off;
  float *scratch = reinterpret_cast<float *>(c.ks + align256(net.ks_bytes));
  auto at = [&](int32_t w) -> char * {
    const int32_t t = p.tag_of[size_t(w)];
    return t >= 0 ? block[size_t(t)] : nullptr;
  };
  // readers of each forward node, in first-reference order, and the byte
  // offset of the node within each reader's input gradients
  std::vector<std::vector<std::pair<int32_t, uint64_t>>> succ(static_cast<size_t>(n));
  for (int32_t v = 0; v < n; ++v) {
    uint64_t o = 0;
    for (int32_t e = g.ptr[size_t(v)]; e < g.ptr[size_t(v) + 1]; ++e) {
      const int32_t u = g.idx[size_t(e)];
      auto &su = succ[size_t(u)];
      if (std::none_of(su.begin(), su.end(), [&](const auto &x) { return x.first == v; }))
        su.emplace_back(v, o);
      o += g.bytes[size_t(u)];
    }
  }
  (void)hipGetLastError();
  net.begin_step(c);
  uint64_t fwd = 0, bwd = 0;
  std::vector<const void *> ins;
  for (int32_t w : p.order) {
    const GraphNode &nd = p.nodes[size_t(w)];
    const int32_t v = nd.of;
    if (nd.kind != CKPT_GNODE_GRAD) {
      ins.clear();
      for (int32_t i : nd.inputs) ins.push_back(at(i));
      net.node_fwd(v, ins, at(w), c);
      ++fwd;
      continue;
    }
    if (g.ptr[size_t(v)] == g.ptr[size_t(v) + 1]) {  // a graph input: nothing to propagate to
      ++bwd;
      continue;
    }
    const auto &sv = succ[size_t(v)];
    const size_t k = sv.size();
    const float *dy = nullptr;
    if (k == 1) {
      dy = reinterpret_cast<const float *>(at(nd.inputs[0]) + sv[0].second);
    } else if (k > 1) {
      const int64_t cnt = int64_t(g.bytes[size_t(v)] / 4);
      ew_add(s, cnt, reinterpret_cast<const float *>(at(nd.inputs[0]) + sv[0].second),
             reinterpret_cast<const float *>(at(nd.inputs[1]) + sv[1].second), scratch);
      for (size_t j = 2; j < k; ++j)
        ew_add(s, cnt, scratch, reinterpret_cast<const float *>(at(nd.inputs[j]) + sv[j].second), scratch);
      c.launches += k - 1;
      dy = scratch;
    }
    size_t r = k;
    const void *y = nullptr;
    if (g.flags[size_t(v)] & CKPT_NODE_GRAD_OUT) y = at(nd.inputs[r++]);
    ins.clear();
    if (g.flags[size_t(v)] & CKPT_NODE_GRAD_IN)
      for (; r < nd.inputs.size(); ++r) ins.push_back(at(nd.inputs[r]));
    net.node_bwd(v, dy, y, ins, at(w), c);
    ++bwd;
  }
  net.end_step(c);
  if (loss_dev) {
    copy_scalar(s, net.loss_ptr(c), loss_dev);
    ++c.launches;
  }
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) fail(CKPT_E_HIP, std::string("train_step_graph: ") + hipGetErrorString(err));
  if (loss_host) {
    err = hipMemcpyAsync(loss_host, net.loss_ptr(c), sizeof(float), hipMemcpyDeviceToHost, s);
    if (err == hipSuccess) err = hipStreamSynchronize(s);
    if (err != hipSuccess) fail(CKPT_E_HIP, std::string("train_step_graph: ") + hipGetErrorString(err));
  }
  if (peak) *peak = p.peak;
  if (stats) {
    stats->unit_forwards = fwd;
    stats->unit_backwards = bwd;
    stats->kernel_launches = c.launches;
    stats->ckpt_bytes = 0;
    stats->arena_bytes = p.peak;
    stats->grad_bytes = 0;
  }
}

}  // namespace ckpt
