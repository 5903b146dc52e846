// Gradient-graph construction with mirror nodes (Alg. 2) and the static memory
// allocator of section 3 (liveness counters, in-place writes, shared tags).
// Host integer code, no HIP calls.
//
// Alg. 2 as implemented: a[v] starts as v; in round k = 1 .. max m(v), in
// topological order, each v with m(v) >= k gets a mirror of its operator
// reading the current a[] of its predecessors, and a[v] becomes the mirror.
// The execution order begins with the forward graph; then, for v from last to
// first, the gradient node g[v] reads the gradient nodes of v's successors,
// a[v] when v's backward reads its output, a[u] of v's predecessors when it
// reads its inputs, and produces the gradients of v's inputs; the ancestors
// of g[v] not yet scheduled, then g[v], are appended in creation order (which
// is topological), so a mirror runs right before the first gradient that
// needs it.  Graph inputs (no predecessors) are never mirrored.
//
// Allocator: one pass over the execution order, one liveness counter per
// output (its pending readers).  NONE gives every output its own tag;
// INPLACE lets an in-place-capable node write over its first input when that
// input's counter is 1 and its tag is large enough; SHARE adds a pool of the
// tags whose output's counter reached 0, from which a new output takes the
// smallest tag that fits (lowest id on ties).  A node's inputs are released
// after its output is placed; an output nobody reads is released after its
// node.  The plan's peak is the sum of the tag sizes.
#include <algorithm>
#include <set>
#include <utility>
#include <vector>

#include "common.h"

namespace ckpt {

GraphPlan make_graph_plan(int32_t n, const int32_t *pred_ptr, const int32_t *pred_idx,
                          const uint64_t *out_bytes, const int32_t *flags, const int32_t *mirror,
                          int32_t strategy) {
  if (n <= 0) fail(CKPT_E_INVALID, "graph_plan: the graph needs at least one node");
  if (!pred_ptr || !out_bytes || !flags || (pred_ptr[n] > 0 && !pred_idx))
    fail(CKPT_E_INVALID, "graph_plan: null array");
  if (strategy < CKPT_ALLOC_NONE || strategy > CKPT_ALLOC_SHARE)
    fail(CKPT_E_INVALID, "graph_plan: unknown allocation strategy");
  if (pred_ptr[0] != 0) fail(CKPT_E_INVALID, "graph_plan: pred_ptr[0] must be 0");
  std::vector<int32_t> m(static_cast<size_t>(n), 0);
  int32_t mmax = 0;
  for (int32_t v = 0; v < n; ++v) {
    if (pred_ptr[v + 1] < pred_ptr[v]) fail(CKPT_E_INVALID, "graph_plan: pred_ptr must not decrease");
    for (int32_t e = pred_ptr[v]; e < pred_ptr[v + 1]; ++e)
      if (pred_idx[e] < 0 || pred_idx[e] >= v)
        fail(CKPT_E_INVALID, "graph_plan: nodes must be listed in topological order");
    if (flags[v] & ~(CKPT_NODE_INPLACE | CKPT_NODE_GRAD_OUT | CKPT_NODE_GRAD_IN))
      fail(CKPT_E_INVALID, "graph_plan: unknown node flag bits");
    const int32_t mv = mirror ? mirror[v] : 0;
    if (mv < 0) fail(CKPT_E_INVALID, "graph_plan: mirror counts are non-negative");
    m[size_t(v)] = pred_ptr[v + 1] > pred_ptr[v] ? mv : 0;
    mmax = std::max(mmax, m[size_t(v)]);
  }
  GraphPlan p;
  p.n_forward = n;
  p.flags.assign(flags, flags + n);
  auto add = [&](int32_t kind, int32_t of, std::vector<int32_t> ins, uint64_t bytes, bool inplace) {
    p.nodes.push_back(GraphNode{kind, of, std::move(ins), bytes, inplace});
    return int32_t(p.nodes.size() - 1);
  };
  for (int32_t v = 0; v < n; ++v)
    add(CKPT_GNODE_FORWARD, v, std::vector<int32_t>(pred_idx + pred_ptr[v], pred_idx + pred_ptr[v + 1]),
        out_bytes[v], (flags[v] & CKPT_NODE_INPLACE) != 0);
  std::vector<int32_t> a(static_cast<size_t>(n));
  for (int32_t v = 0; v < n; ++v) a[size_t(v)] = v;
  for (int32_t k = 1; k <= mmax; ++k)
    for (int32_t v = 0; v < n; ++v)
      if (k <= m[size_t(v)]) {
        std::vector<int32_t> ins;
        for (int32_t e = pred_ptr[v]; e < pred_ptr[v + 1]; ++e) ins.push_back(a[size_t(pred_idx[e])]);
        a[size_t(v)] = add(CKPT_GNODE_MIRROR, v, std::move(ins), out_bytes[v],
                           (flags[v] & CKPT_NODE_INPLACE) != 0);
      }
  // successors in first-reference order
  std::vector<std::vector<int32_t>> succ(static_cast<size_t>(n));
  for (int32_t v = 0; v < n; ++v)
    for (int32_t e = pred_ptr[v]; e < pred_ptr[v + 1]; ++e) {
      auto &s = succ[size_t(pred_idx[e])];
      if (std::find(s.begin(), s.end(), v) == s.end()) s.push_back(v);
    }
  std::vector<char> sched(p.nodes.size() + size_t(n), 0);
  for (int32_t v = 0; v < n; ++v) {
    p.order.push_back(v);
    sched[size_t(v)] = 1;
  }
  std::vector<int32_t> g(static_cast<size_t>(n), -1), stack, need;
  for (int32_t v = n - 1; v >= 0; --v) {
    std::vector<int32_t> ins;
    for (int32_t s : succ[size_t(v)]) ins.push_back(g[size_t(s)]);
    if (flags[v] & CKPT_NODE_GRAD_OUT) ins.push_back(a[size_t(v)]);
    if (flags[v] & CKPT_NODE_GRAD_IN)
      for (int32_t e = pred_ptr[v]; e < pred_ptr[v + 1]; ++e) ins.push_back(a[size_t(pred_idx[e])]);
    uint64_t bytes = 0;
    for (int32_t e = pred_ptr[v]; e < pred_ptr[v + 1]; ++e) bytes += out_bytes[pred_idx[e]];
    g[size_t(v)] = add(CKPT_GNODE_GRAD, v, std::move(ins), bytes, (flags[v] & CKPT_NODE_INPLACE) != 0);
    if (sched.size() < p.nodes.size()) sched.resize(p.nodes.size(), 0);
    need.clear();
    stack.assign(1, g[size_t(v)]);
    while (!stack.empty()) {  // unscheduled ancestors of g[v] (and g[v])
      const int32_t w = stack.back();
      stack.pop_back();
      if (sched[size_t(w)] == 1 || sched[size_t(w)] == 2) continue;
      sched[size_t(w)] = 2;
      need.push_back(w);
      for (int32_t i : p.nodes[size_t(w)].inputs) stack.push_back(i);
    }
    std::sort(need.begin(), need.end());
    for (int32_t w : need) {
      p.order.push_back(w);
      sched[size_t(w)] = 1;
    }
  }

  // ---- static allocation over the execution order
  const size_t N = p.nodes.size();
  std::vector<int64_t> count(N, 0);
  for (int32_t w : p.order)
    for (int32_t i : p.nodes[size_t(w)].inputs) ++count[size_t(i)];
  p.tag_of.assign(N, -1);
  std::set<std::pair<uint64_t, int32_t>> pool;  // free blocks by (bytes, id)
  auto release = [&](int32_t i) {
    const int32_t t = p.tag_of[size_t(i)];
    if (strategy == CKPT_ALLOC_SHARE && t >= 0) pool.emplace(p.tag_bytes[size_t(t)], t);
  };
  for (int32_t w : p.order) {
    const GraphNode &nd = p.nodes[size_t(w)];
    int32_t tag = -1;
    if (nd.bytes > 0) {
      const int32_t first = nd.inputs.empty() ? -1 : nd.inputs[0];
      if (strategy != CKPT_ALLOC_NONE && nd.inplace && first >= 0 && count[size_t(first)] == 1 &&
          p.tag_of[size_t(first)] >= 0 && p.tag_bytes[size_t(p.tag_of[size_t(first)])] >= nd.bytes) {
        tag = p.tag_of[size_t(first)];
        count[size_t(first)] = 0;  // taken over by the in-place write, not released
      } else if (strategy == CKPT_ALLOC_SHARE) {
        // smallest free block that fits, lowest id among equal sizes
        auto it = pool.lower_bound({nd.bytes, INT32_MIN});
        if (it != pool.end()) {
          tag = it->second;
          pool.erase(it);
        }
      }
      if (tag < 0) {
        tag = int32_t(p.tag_bytes.size());
        p.tag_bytes.push_back(nd.bytes);
      }
    }
    p.tag_of[size_t(w)] = tag;
    for (int32_t i : nd.inputs)
      if (count[size_t(i)] > 0 && --count[size_t(i)] == 0) release(i);
    if (count[size_t(w)] == 0 && tag >= 0) release(w);  // an output nobody reads
  }
  for (uint64_t b : p.tag_bytes) p.peak += b;
  for (int32_t w : p.order)
    if (p.nodes[size_t(w)].kind == CKPT_GNODE_MIRROR) ++p.n_mirror;
  return p;
}

}  // namespace ckpt
