// CIFAR-shaped residual CNN (placeholder until its kernels land).
#include "net.h"

namespace ckpt {
std::unique_ptr<Net> make_resnet_basic_net(const ckpt_net_desc &) {
  fail(CKPT_E_UNSUPPORTED, "net_create: RESNET_BASIC is not built yet");
}
}  // namespace ckpt
