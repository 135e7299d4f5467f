// Backward pass, fp16 inputs (the kernels: backward_kernel.h).
#include "backward_kernel.h"

namespace f3s {

hipError_t launch_backward(const f3s_plan_s &p, const f3s_plan_s &pt, const void *Q,
                           const void *K, const void *V, const float *O, const void *G,
                           const float *lse, float *row_stats, float *dQ, float *dK, float *dV,
                           int32_t H, int32_t d, float scale, hipStream_t s)
{
    return launch_bwd_in<false>(p, pt, Q, K, V, O, G, lse, row_stats, dQ, dK, dV, H, d, scale,
                                s);
}

}  // namespace f3s
