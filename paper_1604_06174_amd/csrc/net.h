// Unit chains: static layout tables, parameter layout and per-unit launchers.
#pragma once

#include <hip/hip_runtime.h>

#include <memory>
#include <string>
#include <vector>

#include "common.h"

namespace ckpt {

// Everything a unit launcher needs besides its own tensors.
struct StepCtx {
  hipStream_t s = nullptr;
  const float *params = nullptr;  // device, net.param_bytes
  float *grads = nullptr;         // device, net.param_bytes
  const void *input = nullptr;    // device, batch input
  const void *target = nullptr;   // device, batch targets
  char *ks = nullptr;             // device operator workspace (net.ks_bytes)
  uint64_t launches = 0;
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

  virtual ~Net() = default;

  // Unit i forward: x (x_i) -> y (x_{i+1}); saved internals written to `saved`.
  virtual void fwd(int32_t i, const void *x, void *y, void *saved, StepCtx &c) = 0;
  // Unit i backward: g = dL/dx_{i+1} -> dx = dL/dx_i (dx is null for unit 0),
  // reading x, y and saved; q is the unit's gradient scratch.  Writes unit i's
  // parameter gradients.
  virtual void bwd(int32_t i, const void *g, void *dx, const void *x, const void *y,
                   const void *saved, void *q, StepCtx &c) = 0;
  // Head: x_n -> g = dL/dx_n (+ head parameter gradients), loss into ks.
  virtual void head(const void *xn, void *g, StepCtx &c) = 0;
  // Device address of the f32 loss after the step.
  virtual const float *loss_ptr(const StepCtx &c) const = 0;

  const float *P(const StepCtx &c, int k) const { return c.params + params[size_t(k)].off / 4; }
  float *G(const StepCtx &c, int k) const { return c.grads + params[size_t(k)].off / 4; }

 protected:
  int add_param(const std::string &name, uint64_t numel) {
    params.push_back({name, param_bytes, numel});
    param_bytes += align256(numel * 4);
    return int(params.size()) - 1;
  }
};

std::unique_ptr<Net> make_mlp_net(const ckpt_net_desc &d);
std::unique_ptr<Net> make_resnet_basic_net(const ckpt_net_desc &d);

}  // namespace ckpt
