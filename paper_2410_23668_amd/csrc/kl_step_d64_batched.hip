// Step-kernel instances for head_dim 64, batched (matrix-core) path.
#include "kl_step_impl.h"

namespace kl {

StepKernel step_kernel_d64_batched(int group) {
    switch (group) {
        case 1: return kl_step_kernel<64, 1, true>;
        case 2: return kl_step_kernel<64, 2, true>;
        case 4: return kl_step_kernel<64, 4, true>;
        case 8: return kl_step_kernel<64, 8, true>;
        default: return nullptr;
    }
}

}  // namespace kl
