// f3s_backward_noalloc: the backward pass with its per-row (lse, delta)
// records kept in a fixed device array of this library instead of a buffer
// the caller passes, for callers that cannot allocate device memory.
#include <mutex>

#include "f3s_internal.h"

namespace {

// (row, head) records the array holds: 2^21 records of two floats, 16 MiB
// per device, held from the first call on a device until the process ends.
constexpr int64_t kMaxRecords = int64_t(1) << 21;
constexpr int kMaxDevices = 64;

static __device__ __align__(256) float scratch[2 * kMaxRecords];

std::mutex g_scratch_mu;
// Device address of `scratch` on each device (null until the first call on
// that device looks it up).  Host code uses these, never the array's name,
// which on the host only stands in for the device symbol.
void *g_scratch_ptr[kMaxDevices] = {};

// Address of the array on `device`, looked up once per device with that
// device current.
f3s_status_t scratch_on(int device, float **out)
{
    if (device < 0 || device >= kMaxDevices) return F3S_ERR_UNSUPPORTED;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[device]) {
        int cur = -1;
        if (hipGetDevice(&cur) != hipSuccess) return F3S_ERR_HIP;
        if (cur != device && hipSetDevice(device) != hipSuccess) return F3S_ERR_HIP;
        void *ptr = nullptr;
        const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (cur != device) (void)hipSetDevice(cur);
        if (e != hipSuccess || !ptr) return F3S_ERR_HIP;
        g_scratch_ptr[device] = ptr;
    }
    *out = static_cast<float *>(g_scratch_ptr[device]);
    return F3S_OK;
}

}  // namespace

extern "C" {

f3s_status_t f3s_backward_noalloc(f3s_plan_t p, f3s_plan_t pt, const void *Q,
                                  const void *K, const void *V, f3s_dtype_t in_dtype,
                                  const float *O, const void *dO, const float *lse,
                                  float *dQ, float *dK, float *dV, int32_t n_heads,
                                  int32_t d, float scale, hipStream_t stream)
{
    // Argument errors that need no device go through the full check below;
    // only the size limit and the array lookup are this entry point's own.
    if (p && n_heads >= 1 && (int64_t)p->N * n_heads > kMaxRecords)
        return f3s::record_error(F3S_ERR_TOO_LARGE);
    float *row_stats = nullptr;
    if (p && p->N > 0) {
        const f3s_status_t st = scratch_on(p->device, &row_stats);
        if (st != F3S_OK) return f3s::record_error(st);
    }
    // The dQ pass writes every record the dK/dV pass reads (same stream,
    // in order), so nothing in the array needs clearing between calls.
    return f3s_backward_typed(p, pt, Q, K, V, in_dtype, O, dO, lse, row_stats, dQ, dK, dV,
                              n_heads, d, scale, stream);
}

int64_t f3s_backward_noalloc_max_records(void) { return kMaxRecords; }

}  // extern "C"
