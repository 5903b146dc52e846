// Internal to the C boundary: the opaque objects behind the ABI's handles,
// the error guard and the argument checks the training-step entry points
// share.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <memory>
#include <new>
#include <string>

#include "net.h"

struct ckpt_plan {
  ckpt::Plan p;
};
struct ckpt_net {
  std::unique_ptr<ckpt::Net> net;
};
struct ckpt_graph_plan {
  ckpt::GraphPlan p;
};
// a recorded training step: the captured graph and its executable form
struct ckpt_step_graph {
  hipGraph_t graph = nullptr;
  hipGraphExec_t exec = nullptr;
  ~ckpt_step_graph() {
    if (exec) (void)hipGraphExecDestroy(exec);
    if (graph) (void)hipGraphDestroy(graph);
  }
};

namespace ckpt {
uint64_t workspace_bytes(const Net &net, const Accounting &acc);
void run_train_step(Net &net, const float *params, float *grads, const ckpt_batch &batch,
                    const Plan &p, char *ws, uint64_t ws_bytes, hipStream_t s, float *loss_dev,
                    float *loss_host, uint64_t *peak, ckpt_step_stats *stats);
// Creates the net's side stream when the net uses one, its owner allows it,
// none exists yet, s is not being captured and s is on the current device;
// otherwise does nothing (steps then run on their own stream alone).
void prepare_side(Net &net, hipStream_t s);

// Runs f; returns CKPT_OK, or the code of the error it threw (message kept for
// ckpt_last_error).
template <class F>
int guarded(F &&f) {
  try {
    f();
    set_last_error("");
    return CKPT_OK;
  } catch (const Error &e) {
    set_last_error(e.msg);
    return e.code;
  } catch (const std::bad_alloc &) {
    set_last_error("host allocation failed");
    return CKPT_E_INVALID;
  } catch (const std::exception &e) {
    set_last_error(e.what());
    return CKPT_E_INVALID;
  }
}

inline void need(const void *p, const char *what) {
  if (!p) fail(CKPT_E_INVALID, std::string(what) + ": null pointer");
}

// the argument checks train_step and step_graph_create share
inline void check_step_args(const char *fn, const ckpt_net *net, const void *params,
                            const void *grads, const ckpt_batch *batch, const ckpt_plan *plan,
                            const void *workspace) {
  const std::string f(fn);
  need(net, (f + "(net)").c_str());
  need(params, (f + "(params)").c_str());
  need(grads, (f + "(grads)").c_str());
  need(batch, (f + "(batch)").c_str());
  need(batch->input, (f + "(batch.input)").c_str());
  need(batch->target, (f + "(batch.target)").c_str());
  need(plan, (f + "(plan)").c_str());
  need(workspace, (f + "(workspace)").c_str());
  if (reinterpret_cast<uintptr_t>(workspace) & 255)
    fail(CKPT_E_INVALID, f + ": workspace must be 256-byte aligned");
  if ((reinterpret_cast<uintptr_t>(params) & 255) || (reinterpret_cast<uintptr_t>(grads) & 255))
    fail(CKPT_E_INVALID, f + ": params and grads must be 256-byte aligned");
  if (plan->p.n != net->net->n)
    fail(CKPT_E_MISMATCH, f + ": plan n differs from the net's unit count");
}
}  // namespace ckpt
