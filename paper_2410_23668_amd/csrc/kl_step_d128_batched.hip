// Step-kernel instances for head_dim 128, batched (matrix-core) path.
#include "kl_step_impl.h"

namespace kl {

StepKernel step_kernel_d128_batched(int group) {
    switch (group) {
        case 1: return kl_step_kernel<128, 1, true>;
        case 2: return kl_step_kernel<128, 2, true>;
        case 3: return kl_step_kernel<128, 3, true>;
        case 4: return kl_step_kernel<128, 4, true>;
        case 8: return kl_step_kernel<128, 8, true>;
        default: return nullptr;
    }
}

}  // namespace kl
