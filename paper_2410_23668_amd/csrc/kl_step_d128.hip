// Step-kernel instances for head_dim 128, GEMV path.
#include "kl_step_impl.h"

namespace kl {

StepKernel step_kernel_d128(int group) {
    switch (group) {
        case 1: return kl_step_kernel<128, 1, false>;
        case 2: return kl_step_kernel<128, 2, false>;
        case 3: return kl_step_kernel<128, 3, false>;
        case 4: return kl_step_kernel<128, 4, false>;
        case 8: return kl_step_kernel<128, 8, false>;
        default: return nullptr;
    }
}

}  // namespace kl
