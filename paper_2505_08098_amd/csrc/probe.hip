// Memory-system probes: plain streaming kernels and the fused kernel's access
// pattern without its arithmetic.  They give the bandwidth ceilings the fused
// kernel is measured against (what HBM delivers to a streaming read or copy
// on this GPU, and what the caches and HBM together deliver to a plan's
// gathers), measured in the same process as the kernel.
#include "f3s_probe.h"
#include "kernel_common.h"

namespace {

typedef uint32_t u4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kUnroll = 16;      // 16-byte loads in flight per thread
constexpr uint32_t kNever = 0x9E3779B9u;

__device__ __forceinline__ uint32_t fold(u4 v) { return v.x ^ v.y ^ v.z ^ v.w; }

// Each workgroup reads one contiguous tile of kThreads * kUnroll 16-byte
// chunks (coalesced: chunk t + kThreads * u).  The loaded values feed a
// store that practically never happens, which keeps every load live.
__global__ __launch_bounds__(kThreads) void k_probe_read(const u4 *__restrict__ src,
                                                         uint64_t n16,
                                                         uint32_t *__restrict__ sink)
{
    const uint64_t base = (uint64_t)blockIdx.x * (kThreads * kUnroll) + threadIdx.x;
    u4 v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
        const uint64_t k = base + (uint64_t)kThreads * u;
        v[u] = k < n16 ? src[k] : u4{0u, 0u, 0u, 0u};
    }
    uint32_t acc = 0;
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) acc ^= fold(v[u]);
    if (acc == kNever) sink[threadIdx.x] = acc;
}

__global__ __launch_bounds__(kThreads) void k_probe_copy(const u4 *__restrict__ src,
                                                         u4 *__restrict__ dst, uint64_t n16)
{
    const uint64_t base = (uint64_t)blockIdx.x * (kThreads * kUnroll) + threadIdx.x;
    u4 v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
        const uint64_t k = base + (uint64_t)kThreads * u;
        if (k < n16) v[u] = src[k];
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
        const uint64_t k = base + (uint64_t)kThreads * u;
        if (k < n16) dst[k] = v[u];
    }
}

__global__ __launch_bounds__(kThreads) void k_probe_write(u4 *__restrict__ dst, uint64_t n16,
                                                          uint32_t value)
{
    const uint64_t base = (uint64_t)blockIdx.x * (kThreads * kUnroll) + threadIdx.x;
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
        const uint64_t k = base + (uint64_t)kThreads * u;
        if (k < n16) dst[k] = u4{value, value ^ (uint32_t)u, value, (uint32_t)k};
    }
}

// A fixed integer hash (xorshift-multiply finaliser) that spreads group and
// step indices uniformly over the table's rows.
__device__ __forceinline__ uint32_t spread(uint32_t x)
{
    x ^= x >> 16;
    x *= 0x7FEB352Du;
    x ^= x >> 15;
    x *= 0x846CA68Bu;
    x ^= x >> 16;
    return x;
}

// Random whole-row gathers: a group of L lanes reads one row of 16 L bytes
// (16 bytes per lane) per step, kInFlight steps in flight, `rounds` times.
template <int L, int kInFlight>
__global__ __launch_bounds__(kThreads) void k_probe_rows(const u4 *__restrict__ table,
                                                         uint32_t rows, int32_t rounds,
                                                         uint32_t *__restrict__ sink)
{
    const uint32_t gid = blockIdx.x * kThreads + threadIdx.x;
    const uint32_t group = gid / L, sub = gid % L;
    uint32_t acc = 0;
    for (int r = 0; r < rounds; ++r) {
        u4 v[kInFlight];
#pragma unroll
        for (int u = 0; u < kInFlight; ++u) {
            const uint32_t step = (uint32_t)r * kInFlight + u;
            const uint32_t row = spread(group * 0x9E3779B1u + step * 0x85EBCA77u) % rows;
            v[u] = table[(uint64_t)row * L + sub];
        }
#pragma unroll
        for (int u = 0; u < kInFlight; ++u) acc ^= fold(v[u]);
    }
    if (acc == kNever) sink[threadIdx.x] = acc;
}

// The fp16 -> fp32 fused kernel's memory accesses for one work item, with no
// arithmetic: the item record, the window's Q rows, per block its 16 column
// ids and 8 bitmap words, the K and V rows of every slot gathered in 16-byte
// chunks laid flat over the lanes (a lane quad reads 64 contiguous bytes of
// one row, padding slots re-read the block's first column), and 16 rows of
// D fp32 written (to O for a whole window, to the piece's partial slot for a
// piece of a split window).  Four waves share an item, wave w taking block
// pairs w, w + 4, ...; each wave has two pairs in flight.  Workgroups take
// items in the fused kernel's order (XCD ranges where it uses them).  The
// written values are the loaded bits folded together (garbage, but they keep
// every load live).
template <int D, bool kWide>
__global__ __launch_bounds__(256) void k_probe_gather(
    const f3s::WorkItem *__restrict__ items, const int32_t *__restrict__ cols,
    const uint32_t *__restrict__ mask, const int32_t *__restrict__ win_row,
    const char *__restrict__ Q, const char *__restrict__ K, const char *__restrict__ V,
    float *__restrict__ O, float *__restrict__ part_o, int32_t N, uint32_t order)
{
    constexpr int LPR = D / 8;   // 16-byte chunks per row
    constexpr int NI = D / 16;   // chunks per lane per 32-row tile
    const int wv = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const f3s::WorkItem it = items[f3s::workgroup_position(order, 1)];
    int32_t r0, nr;
    f3s::window_rows(win_row, N, it.window, &r0, &nr);
    uint32_t acc = 0;
    // Q: rows 4 wv .. 4 wv + 3 of the window (pad rows read its first row)
    for (int f = lane; f < 4 * LPR; f += 64) {
        const int r = 4 * wv + f / LPR;
        const int64_t qrow = r0 + (r < nr ? r : 0);
        acc ^= fold(*reinterpret_cast<const u4 *>(Q + qrow * D * 2 + 16 * (f % LPR)));
    }
    const int b0 = it.blk_begin, b1 = it.blk_end;
    for (int b = b0 + 2 * wv; b < b1; b += 16) {
        // pairs b and b + 8 of this wave (the second one if it exists)
        const int npp = b + 8 < b1 ? 2 : 1;
        u4 kv[2][2 * NI];
        uint32_t mw[2] = {0u, 0u};
#pragma unroll
        for (int pp = 0; pp < 2; ++pp) {
            if (pp >= npp) break;
            const int bb = b + 8 * pp;
            const int slot = lane & 31;
            const int blk = slot < 16 ? bb : min(bb + 1, b1 - 1);
            int c = cols[(int64_t)16 * blk + (slot & 15)];
            const int first = cols[(int64_t)16 * blk];
            c = c < 0 ? first : c;
#pragma unroll
            for (int j = 0; j < NI; ++j) {
                const int f = lane + 64 * j;
                const int col = __shfl(c, f / LPR);
                if constexpr (kWide) {
                    const int64_t off = (int64_t)col * D * 2 + 16 * (f % LPR);
                    kv[pp][2 * j] = *reinterpret_cast<const u4 *>(K + off);
                    kv[pp][2 * j + 1] = *reinterpret_cast<const u4 *>(V + off);
                } else {
                    const uint32_t off = (uint32_t)col * (uint32_t)(2 * D) + 16u * (f % LPR);
                    kv[pp][2 * j] = *reinterpret_cast<const u4 *>(K + off);
                    kv[pp][2 * j + 1] = *reinterpret_cast<const u4 *>(V + off);
                }
            }
            mw[pp] = mask[(int64_t)8 * bb + (lane >> 3)] ^
                     mask[(int64_t)8 * min(bb + 1, b1 - 1) + (lane >> 3)];
        }
#pragma unroll
        for (int pp = 0; pp < 2; ++pp) {
            if (pp >= npp) break;
            acc ^= mw[pp];
#pragma unroll
            for (int j = 0; j < 2 * NI; ++j) acc ^= fold(kv[pp][j]);
        }
    }
    // 16 x D fp32 out: wave wv writes rows 4 wv .. 4 wv + 3
    const float val = __builtin_bit_cast(float, acc & 0x3FFFFFFFu);
    for (int f = lane; f < 4 * (D / 4); f += 64) {
        const int rr = 4 * wv + f / (D / 4), cc = 4 * (f % (D / 4));
        const float4 v4 = make_float4(val, val, val, val);
        if (it.slot < 0) {
            if (rr < nr) *reinterpret_cast<float4 *>(O + (int64_t)(r0 + rr) * D + cc) = v4;
        } else {
            *reinterpret_cast<float4 *>(part_o + ((int64_t)it.slot * 16 + rr) * D + cc) = v4;
        }
    }
}

// The same accesses with the K and V chunks loaded straight into LDS
// (global_load_lds, 16 bytes per lane: one instruction fills a 1 KB run of
// the wave's LDS area, lane l at byte 16 l).  The wave walks pairs w, w + 4,
// ... of the item one after another and never waits for them: every pair
// overwrites the same 2 NI KB area, which nothing reads back until the end
// (one word per lane), so the only limit on the rows in flight is the
// hardware's count of outstanding loads.  This is the rate of the access
// pattern with unbounded depth, an upper bound for any kernel that gathers
// the rows into LDS and has to keep each pair there until it is consumed.
// 32-bit offsets only; D <= 128 (the four waves' areas, 8 D bytes each per
// 16-byte chunk column, fill at most 64 KB).
template <int D>
__global__ __launch_bounds__(256) void k_probe_gather_lds(
    const f3s::WorkItem *__restrict__ items, const int32_t *__restrict__ cols,
    const uint32_t *__restrict__ mask, const int32_t *__restrict__ win_row,
    const char *__restrict__ Q, const char *__restrict__ K, const char *__restrict__ V,
    float *__restrict__ O, float *__restrict__ part_o, int32_t N, uint32_t order)
{
    constexpr int LPR = D / 8;            // 16-byte chunks per row
    constexpr int NI = D / 16;            // chunks per lane per 32-row tile
    constexpr int AREA = 2 * NI * 1024;   // a pair's K and V rows, bytes
    typedef __attribute__((address_space(3))) void lds_void;
    __shared__ __attribute__((aligned(16))) char lds[4][AREA];
    const int wv = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const f3s::WorkItem it = items[f3s::workgroup_position(order, 1)];
    int32_t r0, nr;
    f3s::window_rows(win_row, N, it.window, &r0, &nr);
    uint32_t acc = 0;
    for (int f = lane; f < 4 * LPR; f += 64) {
        const int r = 4 * wv + f / LPR;
        const int64_t qrow = r0 + (r < nr ? r : 0);
        acc ^= fold(*reinterpret_cast<const u4 *>(Q + qrow * D * 2 + 16 * (f % LPR)));
    }
    const int b0 = it.blk_begin, b1 = it.blk_end;
    for (int b = b0 + 2 * wv; b < b1; b += 8) {
        const int slot = lane & 31;
        const int blk = slot < 16 ? b : min(b + 1, b1 - 1);
        int c = cols[(int64_t)16 * blk + (slot & 15)];
        const int first = cols[(int64_t)16 * blk];
        c = c < 0 ? first : c;
#pragma unroll
        for (int j = 0; j < NI; ++j) {
            const int f = lane + 64 * j;
            const int col = __shfl(c, f / LPR);
            const uint32_t off = (uint32_t)col * (uint32_t)(2 * D) + 16u * (f % LPR);
            __builtin_amdgcn_global_load_lds(static_cast<const void *>(K + off),
                                             (lds_void *)&lds[wv][2 * j * 1024], 16, 0, 0);
            __builtin_amdgcn_global_load_lds(static_cast<const void *>(V + off),
                                             (lds_void *)&lds[wv][(2 * j + 1) * 1024], 16, 0,
                                             0);
        }
        acc ^= mask[(int64_t)8 * b + (lane >> 3)] ^
               mask[(int64_t)8 * min(b + 1, b1 - 1) + (lane >> 3)];
    }
    // every load done before the area is read (the compiler does not track
    // loads into LDS)
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    acc ^= reinterpret_cast<const uint32_t *>(lds[wv])[lane];
    const float val = __builtin_bit_cast(float, acc & 0x3FFFFFFFu);
    for (int f = lane; f < 4 * (D / 4); f += 64) {
        const int rr = 4 * wv + f / (D / 4), cc = 4 * (f % (D / 4));
        const float4 v4 = make_float4(val, val, val, val);
        if (it.slot < 0) {
            if (rr < nr) *reinterpret_cast<float4 *>(O + (int64_t)(r0 + rr) * D + cc) = v4;
        } else {
            *reinterpret_cast<float4 *>(part_o + ((int64_t)it.slot * 16 + rr) * D + cc) = v4;
        }
    }
}

template <int D>
hipError_t launch_gather_lds_d(const f3s_plan_s &p, const void *Q, const void *K,
                               const void *V, float *O, hipStream_t s)
{
    k_probe_gather_lds<D><<<p.n_items, 256, 0, s>>>(
        p.items, p.cols, p.mask, p.win_row, static_cast<const char *>(Q),
        static_cast<const char *>(K), static_cast<const char *>(V), O, p.part_o, p.N,
        f3s::xcd_chunks(p, 1) ? f3s::kOrderXcd : 0u);
    return hipGetLastError();
}

template <int D>
hipError_t launch_gather_d(const f3s_plan_s &p, const void *Q, const void *K, const void *V,
                           float *O, hipStream_t s)
{
    const bool wide = (uint64_t)p.N * D * 2 > 0xFFFFFFF0ull;
    auto kern = wide ? k_probe_gather<D, true> : k_probe_gather<D, false>;
    kern<<<p.n_items, 256, 0, s>>>(p.items, p.cols, p.mask, p.win_row,
                                   static_cast<const char *>(Q),
                                   static_cast<const char *>(K),
                                   static_cast<const char *>(V), O, p.part_o, p.N,
                                   f3s::xcd_chunks(p, 1) ? f3s::kOrderXcd : 0u);
    return hipGetLastError();
}

f3s_status_t status(hipError_t e)
{
    return e == hipSuccess ? F3S_OK : F3S_ERR_HIP;
}

template <int U>
f3s_status_t launch_rows(const void *table, int64_t rows, int32_t row_bytes,
                         int32_t workgroups, int32_t rounds, uint32_t *sink, hipStream_t s)
{
    const dim3 grid((unsigned)workgroups);
    const u4 *tab = static_cast<const u4 *>(table);
    const uint32_t n = (uint32_t)rows;
    switch (row_bytes) {
    case 16: k_probe_rows<1, U><<<grid, kThreads, 0, s>>>(tab, n, rounds, sink); break;
    case 32: k_probe_rows<2, U><<<grid, kThreads, 0, s>>>(tab, n, rounds, sink); break;
    case 64: k_probe_rows<4, U><<<grid, kThreads, 0, s>>>(tab, n, rounds, sink); break;
    case 128: k_probe_rows<8, U><<<grid, kThreads, 0, s>>>(tab, n, rounds, sink); break;
    case 256: k_probe_rows<16, U><<<grid, kThreads, 0, s>>>(tab, n, rounds, sink); break;
    case 512: k_probe_rows<32, U><<<grid, kThreads, 0, s>>>(tab, n, rounds, sink); break;
    case 1024: k_probe_rows<64, U><<<grid, kThreads, 0, s>>>(tab, n, rounds, sink); break;
    default: return F3S_ERR_UNSUPPORTED;
    }
    return status(hipGetLastError());
}

bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }

unsigned tiles(uint64_t n16)
{
    return (unsigned)((n16 + kThreads * kUnroll - 1) / (kThreads * kUnroll));
}

}  // namespace

extern "C" {

f3s_status_t f3s_probe_read(const void *src, size_t bytes, uint32_t *sink, hipStream_t stream)
{
    if (!src || !sink || !aligned16(src) || bytes % 16 ||
        bytes / 16 / (kThreads * kUnroll) >= 0x7FFFFFFFull)
        return F3S_ERR_INVALID_VALUE;
    const uint64_t n16 = bytes / 16;
    if (n16 == 0) return F3S_OK;
    k_probe_read<<<tiles(n16), kThreads, 0, stream>>>(static_cast<const u4 *>(src), n16, sink);
    return status(hipGetLastError());
}

f3s_status_t f3s_probe_copy(const void *src, void *dst, size_t bytes, hipStream_t stream)
{
    if (!src || !dst || !aligned16(src) || !aligned16(dst) || bytes % 16 ||
        bytes / 16 / (kThreads * kUnroll) >= 0x7FFFFFFFull)
        return F3S_ERR_INVALID_VALUE;
    const uint64_t n16 = bytes / 16;
    if (n16 == 0) return F3S_OK;
    k_probe_copy<<<tiles(n16), kThreads, 0, stream>>>(static_cast<const u4 *>(src),
                                                       static_cast<u4 *>(dst), n16);
    return status(hipGetLastError());
}

f3s_status_t f3s_probe_write(void *dst, size_t bytes, uint32_t value, hipStream_t stream)
{
    if (!dst || !aligned16(dst) || bytes % 16 ||
        bytes / 16 / (kThreads * kUnroll) >= 0x7FFFFFFFull)
        return F3S_ERR_INVALID_VALUE;
    const uint64_t n16 = bytes / 16;
    if (n16 == 0) return F3S_OK;
    k_probe_write<<<tiles(n16), kThreads, 0, stream>>>(static_cast<u4 *>(dst), n16, value);
    return status(hipGetLastError());
}

f3s_status_t f3s_probe_rows(const void *table, int64_t rows, int32_t row_bytes,
                            int32_t in_flight, int32_t workgroups, int32_t rounds,
                            uint32_t *sink, hipStream_t stream)
{
    if (!table || !sink || !aligned16(table) || rows < 1 || rows > 0xFFFFFFFFll ||
        workgroups < 1 || rounds < 1)
        return F3S_ERR_INVALID_VALUE;
    switch (in_flight) {
    case 1: return launch_rows<1>(table, rows, row_bytes, workgroups, rounds, sink, stream);
    case 2: return launch_rows<2>(table, rows, row_bytes, workgroups, rounds, sink, stream);
    case 4: return launch_rows<4>(table, rows, row_bytes, workgroups, rounds, sink, stream);
    case 8: return launch_rows<8>(table, rows, row_bytes, workgroups, rounds, sink, stream);
    case 16: return launch_rows<16>(table, rows, row_bytes, workgroups, rounds, sink, stream);
    default: return F3S_ERR_UNSUPPORTED;
    }
}

f3s_status_t f3s_probe_gather(f3s_plan_t p, const void *Q, const void *K, const void *V,
                              float *O, int32_t d, hipStream_t stream)
{
    if (!p || !Q || !K || !V || !O) return F3S_ERR_INVALID_VALUE;
    if (!aligned16(Q) || !aligned16(K) || !aligned16(V) || !aligned16(O))
        return F3S_ERR_INVALID_VALUE;
    if (p->N == 0 || p->n_items == 0) return F3S_OK;
    switch (d) {
    case 32: return status(launch_gather_d<32>(*p, Q, K, V, O, stream));
    case 64: return status(launch_gather_d<64>(*p, Q, K, V, O, stream));
    case 128: return status(launch_gather_d<128>(*p, Q, K, V, O, stream));
    case 256: return status(launch_gather_d<256>(*p, Q, K, V, O, stream));
    default: return F3S_ERR_UNSUPPORTED;
    }
}

f3s_status_t f3s_probe_gather_lds(f3s_plan_t p, const void *Q, const void *K,
                                  const void *V, float *O, int32_t d, hipStream_t stream)
{
    if (!p || !Q || !K || !V || !O) return F3S_ERR_INVALID_VALUE;
    if (!aligned16(Q) || !aligned16(K) || !aligned16(V) || !aligned16(O))
        return F3S_ERR_INVALID_VALUE;
    if (d != 32 && d != 64 && d != 128) return F3S_ERR_UNSUPPORTED;
    if ((uint64_t)p->N * (uint64_t)d * 2u > 0xFFFFFFF0ull) return F3S_ERR_UNSUPPORTED;
    if (p->N == 0 || p->n_items == 0) return F3S_OK;
    switch (d) {
    case 32: return status(launch_gather_lds_d<32>(*p, Q, K, V, O, stream));
    case 64: return status(launch_gather_lds_d<64>(*p, Q, K, V, O, stream));
    default: return status(launch_gather_lds_d<128>(*p, Q, K, V, O, stream));
    }
}

}  // extern "C"
