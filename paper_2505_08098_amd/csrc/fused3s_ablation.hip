// Ablation build of the fused forward: K and V gathered in 4-byte words
// instead of 16-byte chunks (the access granularity the register remapping
// of Section 3.4 removes); selected by a plan built with F3S_NARROW_GATHER=1.
#include "fused3s_kernel.h"

namespace f3s {

hipError_t launch_fused_narrow(const f3s_plan_s &p, const void *Q, const void *K,
                               const void *V, void *O, float *lse, int32_t H, int32_t d,
                               float sl2, hipStream_t s)
{
    return launch_in<kInF16, false, true>(p, Q, K, V, O, lse, H, d, sl2, s);
}

}  // namespace f3s
