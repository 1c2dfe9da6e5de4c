// Step-kernel instances for head_dim 64, GEMV path.
#include "kl_step_impl.h"

namespace kl {

StepKernel step_kernel_d64(int group) {
    switch (group) {
        case 1: return kl_step_kernel<64, 1, false>;
        case 2: return kl_step_kernel<64, 2, false>;
        case 4: return kl_step_kernel<64, 4, false>;
        case 8: return kl_step_kernel<64, 8, false>;
        default: return nullptr;
    }
}

}  // namespace kl
