// Fused 3S forward, fp16 inputs (the precision scheme of Table 5), and the
// dispatch over input storage types.  The kernels are in fused3s_kernel.h.
#include "fused3s_kernel.h"

namespace f3s {

hipError_t launch_fused(const f3s_plan_s &p, const void *Q, const void *K,
                        const void *V, int in_type, void *O, bool out_f16, float *lse,
                        int32_t H, int32_t d, float sl2, hipStream_t s)
{
    if (in_type == kInBF16) return launch_fused_bf16(p, Q, K, V, O, out_f16, lse, H, d, sl2, s);
    if (in_type == kInFP8) return launch_fused_fp8(p, Q, K, V, O, out_f16, lse, H, d, sl2, s);
    if (in_type != kInF16) return hipErrorInvalidValue;
    if (p.flags & 2) {
        if (out_f16) return hipErrorInvalidValue;
        return launch_fused_narrow(p, Q, K, V, O, lse, H, d, sl2, s);
    }
    if (p.flags & 8) {
        if (out_f16) return hipErrorInvalidValue;
        return launch_fused_split_row(p, Q, K, V, static_cast<float *>(O), lse, H, d, sl2, s);
    }
    return out_f16 ? launch_in<kInF16, true>(p, Q, K, V, O, lse, H, d, sl2, s)
                   : launch_in<kInF16, false>(p, Q, K, V, O, lse, H, d, sl2, s);
}

hipError_t launch_fused_trace(const f3s_plan_s &p, const void *Q, const void *K,
                              const void *V, void *O, int32_t d, float sl2, uint32_t *trace,
                              hipStream_t s)
{
    if (p.flags & 10) return hipErrorInvalidValue;
    return launch_in<kInF16, false>(p, Q, K, V, O, nullptr, 1, d, sl2, s, trace);
}

}  // namespace f3s
