// train_step_static: the training step for callers that cannot allocate
// device memory (code under HIP graph capture, tight serving loops, harnesses
// that forbid hipMalloc).  It is train_step with the workspace taken from a
// fixed scratch array the library holds on each GPU, instead of a caller
// buffer: the same kernels on the same layout, so the results are
// train_step's bit for bit.
//
// The scratch is a file-scope __device__ array; in host code its name is only
// a stand-in for the symbol, so its device address on the current GPU is
// looked up once per device (hipGetSymbolAddress, with that device current)
// and that address is what the kernels receive.  Every call on one GPU shares
// that GPU's array, which keeps whatever the last call left in it; the step
// ignores the workspace's contents on entry, so nothing needs clearing.  Calls
// that overlap in time on one GPU (different streams or threads) race on it.
#include <hip/hip_runtime.h>

#include <mutex>
#include <string>

#include "capi_internal.h"

namespace {

constexpr uint64_t kScratchBytes = uint64_t(CKPT_STATIC_SCRATCH_BYTES);
constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[CKPT_STATIC_SCRATCH_BYTES];

std::mutex g_scratch_mu;
char *g_scratch[kMaxDevices] = {};  // device address of `scratch` per device

// The scratch array's device address on the calling thread's current device.
char *scratch_on_current_device() {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess)
    ckpt::fail(CKPT_E_HIP, std::string("train_step_static: hipGetDevice: ") + hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices)
    ckpt::fail(CKPT_E_UNSUPPORTED, "train_step_static: device index beyond " + std::to_string(kMaxDevices));
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      ckpt::fail(CKPT_E_HIP, std::string("train_step_static: hipGetSymbolAddress: ") +
                                 (e != hipSuccess ? hipGetErrorString(e) : "null address"));
    if (reinterpret_cast<uintptr_t>(p) & 255)
      ckpt::fail(CKPT_E_HIP, "train_step_static: scratch is not 256-byte aligned");
    g_scratch[dev] = static_cast<char *>(p);
  }
  return g_scratch[dev];
}

}  // namespace

extern "C" int train_step_static(ckpt_net *net, const void *params, void *grads,
                                 const ckpt_batch *batch, const ckpt_plan *plan, void *stream,
                                 float *loss_dev, float *loss_host, uint64_t *peak,
                                 ckpt_step_stats *stats) {
  return ckpt::guarded([&] {
    // the checks train_step makes, a non-null stand-in for the workspace
    ckpt::check_step_args("train_step_static", net, params, grads, batch, plan,
                          reinterpret_cast<const void *>(uintptr_t(256)));
    if (net->net->timer.enabled)
      ckpt::fail(CKPT_E_INVALID, "train_step_static: kernel timing creates events; turn it off");
    const uint64_t need = ckpt::workspace_bytes(*net->net, net->net->accounting(plan->p));
    if (need > kScratchBytes)
      ckpt::fail(CKPT_E_WORKSPACE, "train_step_static: the plan needs " + std::to_string(need) +
                                       " bytes of workspace, the static scratch holds " +
                                       std::to_string(kScratchBytes) + " (use train_step)");
    char *ws = scratch_on_current_device();
    ckpt::run_train_step(*net->net, static_cast<const float *>(params), static_cast<float *>(grads),
                         *batch, plan->p, ws, kScratchBytes, static_cast<hipStream_t>(stream),
                         loss_dev, loss_host, peak, stats);
  });
}
