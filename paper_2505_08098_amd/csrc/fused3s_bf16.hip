// Fused 3S forward with bfloat16 inputs (scores on the bf16 matrix
// instruction, probabilities as a two-term bf16 split; see fused3s_kernel.h).
#include "fused3s_kernel.h"

namespace f3s {

hipError_t launch_fused_bf16(const f3s_plan_s &p, const void *Q, const void *K,
                             const void *V, void *O, bool out_f16, float *lse, int32_t H,
                             int32_t d, float sl2, hipStream_t s)
{
    return out_f16 ? launch_in<kInBF16, true>(p, Q, K, V, O, lse, H, d, sl2, s)
                   : launch_in<kInBF16, false>(p, Q, K, V, O, lse, H, d, sl2, s);
}

}  // namespace f3s
