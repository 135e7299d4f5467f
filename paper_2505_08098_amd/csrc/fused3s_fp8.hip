// Fused 3S forward with fp8 (OCP e4m3) inputs: half the gathered bytes of
// the fp16 scheme; rows are widened to fp16 (exactly) as they are staged, so
// the products and the probabilities follow the fp16 path (see
// fused3s_kernel.h).
#include "fused3s_kernel.h"

namespace f3s {

hipError_t launch_fused_fp8(const f3s_plan_s &p, const void *Q, const void *K,
                            const void *V, void *O, bool out_f16, float *lse, int32_t H,
                            int32_t d, float sl2, hipStream_t s)
{
    return out_f16 ? launch_in<kInFP8, true>(p, Q, K, V, O, lse, H, d, sl2, s)
                   : launch_in<kInFP8, false>(p, Q, K, V, O, lse, H, d, sl2, s);
}

}  // namespace f3s
