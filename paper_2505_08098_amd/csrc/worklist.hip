// Heavy-first work list of a plan (Section 3.2), in O(T) memory: the windows
// are stably sorted by their key, largest first, the item counts are scanned
// in that order, and every window writes its item (or, if split, its merge
// record and first item position; its pieces are written by k_split_items).
//
// The sort is a least-significant-digit radix sort with 8-bit digits (one
// pass per 8 bits of the largest key, usually one or two): per tile of
// kTile keys a digit histogram, one scan over (digit, tile), then a stable
// scatter in which each tile walks its keys in order, 256 at a time, and
// ranks equal digits with wavefront ballots.  Larger keys first: the digit
// used is 255 - digit.
#include "f3s_internal.h"

namespace f3s {
namespace {

constexpr int kRadixThreads = 256;
constexpr int kRadixSteps = 16;
constexpr int kTile = kRadixThreads * kRadixSteps;  // keys per tile

__device__ __forceinline__ int rdigit(int32_t key, int shift)
{
    return 255 - ((key >> shift) & 255);
}

// counts[d * ntiles + tile] = keys of tile `tile` whose (reversed) digit is d.
__global__ __launch_bounds__(kRadixThreads) void k_digit_count(const int32_t *keys,
                                                               int32_t n, int shift,
                                                               int32_t ntiles,
                                                               int32_t *counts)
{
    __shared__ int32_t h[256];
    const int tid = threadIdx.x;
    h[tid] = 0;
    __syncthreads();
    const int64_t base = (int64_t)blockIdx.x * kTile;
    for (int j = 0; j < kRadixSteps; ++j) {
        const int64_t i = base + j * kRadixThreads + tid;
        if (i < n) atomicAdd(&h[rdigit(keys[i], shift)], 1);
    }
    __syncthreads();
    counts[(int64_t)tid * ntiles + blockIdx.x] = h[tid];
}

// Stable scatter of one tile: keys are taken in index order, 256 per step;
// within a step a key's rank among equal digits comes from ballots (within
// its wavefront) and the counts of the earlier wavefronts of the step.
__global__ __launch_bounds__(kRadixThreads) void k_digit_scatter(
    const int32_t *keys, const int32_t *vals, int32_t n, int shift, int32_t ntiles,
    const int32_t *offs, int32_t *keys_out, int32_t *vals_out)
{
    constexpr int kWaves = kRadixThreads / 64;
    __shared__ int32_t run[256];           // keys of each digit placed so far
    __shared__ int32_t wcnt[kWaves][256];  // this step's count per wave and digit
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    run[tid] = offs[(int64_t)tid * ntiles + blockIdx.x];
    for (int k = 0; k < kWaves; ++k) wcnt[k][tid] = 0;
    __syncthreads();
    const int64_t base = (int64_t)blockIdx.x * kTile;
    const uint64_t below = (1ull << lane) - 1ull;
    for (int j = 0; j < kRadixSteps; ++j) {
        const int64_t i = base + j * kRadixThreads + tid;
        const bool valid = i < n;
        const int32_t key = valid ? keys[i] : 0;
        const int d = valid ? rdigit(key, shift) : 0;
        // lanes of this wave holding the same digit
        uint64_t peers = __ballot(valid);
#pragma unroll
        for (int b = 0; b < 8; ++b) {
            const uint64_t bal = __ballot(valid && ((d >> b) & 1));
            peers &= ((d >> b) & 1) ? bal : ~bal;
        }
        const int rank = __popcll(peers & below);
        if (valid && rank == 0) wcnt[wv][d] = __popcll(peers);
        __syncthreads();
        if (valid) {
            int before = run[d] + rank;
            for (int k = 0; k < wv; ++k) before += wcnt[k][d];
            keys_out[before] = key;
            vals_out[before] = vals[i];
        }
        __syncthreads();
        int add = 0;
        for (int k = 0; k < kWaves; ++k) {
            add += wcnt[k][tid];
            wcnt[k][tid] = 0;
        }
        run[tid] += add;
        __syncthreads();
    }
}

__global__ void k_iota(int32_t *a, int32_t n)
{
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) a[i] = i;
}

__global__ void k_gather_pieces(const int32_t *order, const int32_t *npieces, int32_t T,
                                int32_t *np_sorted)
{
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < T) np_sorted[i] = npieces[order[i]];
}

// Window order[i] starts at item pos[i].
__global__ void k_place_items(const int32_t *order, const int32_t *pos, const int32_t *nb,
                              const int32_t *blk_off, const int32_t *npieces,
                              const int32_t *slot_base, const int32_t *split_idx, int32_t T,
                              int32_t piece, WorkItem *items, int32_t *merges,
                              int32_t *split_item)
{
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= T) return;
    const int w = order[i], p = pos[i];
    const int n = nb[w], b0 = blk_off[w];
    if (n <= piece) {
        items[p] = WorkItem{w, b0, b0 + n, -1};
    } else {
        const int s = split_idx[w];
        merges[3 * s + 0] = w;
        merges[3 * s + 1] = slot_base[w];
        merges[3 * s + 2] = npieces[w];
        split_item[s] = p;
    }
}

inline unsigned blocks_for(int64_t n, int threads)
{
    return (unsigned)(n > 0 ? (n + threads - 1) / threads : 1);
}

}  // namespace

int64_t worklist_count_ints(int32_t T)
{
    const int64_t ntiles = (T + kTile - 1) / kTile;
    return 256 * (ntiles > 0 ? ntiles : 1) + 1;
}

hipError_t launch_worklist(const int32_t *key, const int32_t *nb, const int32_t *blk_off,
                           const int32_t *npieces, const int32_t *slot_base,
                           const int32_t *split_idx, int32_t T, int32_t piece,
                           const WorkListScratch &ws, WorkItem *items, int32_t *merges,
                           int32_t *split_item, int32_t *n_items_out, hipStream_t s)
{
    if (T == 0) return hipSuccess;
    const int32_t ntiles = (T + kTile - 1) / kTile;
    const int32_t cells = 256 * ntiles;
    hipError_t e;
    // keys ping-pong between ws.keys_a / ws.keys_b, windows between
    // ws.order_in / ws.order; the first pass reads the caller's keys
    k_iota<<<blocks_for(T, 256), 256, 0, s>>>(ws.order_in, T);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    const int32_t *kin = key;
    const int32_t *vin = ws.order_in;
    int32_t *kout = ws.keys_a, *vout = ws.order;
    int passes = 0;
    for (int shift = 0; shift == 0 || (shift < 31 && (piece >> shift) != 0); shift += 8) {
        k_digit_count<<<ntiles, kRadixThreads, 0, s>>>(kin, T, shift, ntiles, ws.counts);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        e = launch_scan(ws.counts, ws.counts, cells, ws.scan_tmp, nullptr, s);
        if (e != hipSuccess) return e;
        k_digit_scatter<<<ntiles, kRadixThreads, 0, s>>>(kin, vin, T, shift, ntiles,
                                                          ws.counts, kout, vout);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        ++passes;
        // the next pass reads this one's output
        kin = kout;
        vin = vout;
        kout = kout == ws.keys_a ? ws.keys_b : ws.keys_a;
        vout = vout == ws.order ? ws.order_in : ws.order;
    }
    const int32_t *order = vin;  // windows, largest key first
    k_gather_pieces<<<blocks_for(T, 256), 256, 0, s>>>(order, npieces, T, ws.pos);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    e = launch_scan(ws.pos, ws.pos, T, ws.scan_tmp, n_items_out, s);
    if (e != hipSuccess) return e;
    k_place_items<<<blocks_for(T, 256), 256, 0, s>>>(order, ws.pos, nb, blk_off, npieces,
                                                     slot_base, split_idx, T, piece, items,
                                                     merges, split_item);
    (void)passes;
    return hipGetLastError();
}

}  // namespace f3s
