// Stable least-significant-digit radix sort of (key, value) pairs of int32,
// keys in [0, max_key], ascending or descending, with 8-bit digits (one pass
// per 8 bits of max_key): per tile of kTile keys a digit histogram, one scan
// over (digit, tile), then a stable scatter in which each tile ranks its keys
// (in order, 256 at a time, equal digits by wavefront ballots) into digit
// order in LDS and writes them out run by run.
#include "f3s_internal.h"

namespace f3s {
namespace {

constexpr int kRadixThreads = 256;
constexpr int kRadixSteps = 16;
constexpr int kTile = kRadixThreads * kRadixSteps;  // keys per tile

__device__ __forceinline__ int rdigit(int32_t key, int shift, bool descending)
{
    const int x = (key >> shift) & 255;
    return descending ? 255 - x : x;
}

// counts[d * ntiles + tile] = keys of tile `tile` whose digit is d.
__global__ __launch_bounds__(kRadixThreads) void k_digit_count(const int32_t *keys,
                                                               int32_t n, int shift,
                                                               bool descending,
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
        if (i < n) atomicAdd(&h[rdigit(keys[i], shift, descending)], 1);
    }
    __syncthreads();
    counts[(int64_t)tid * ntiles + blockIdx.x] = h[tid];
}

// Stable scatter of one tile.  The tile's keys are first placed in LDS in
// digit order: taken in index order, 256 per step, a key's rank among equal
// digits comes from ballots (within its wavefront) and the counts of the
// earlier wavefronts of the step.  Then the tile is written out in that
// order, so each digit's run of keys goes to consecutive addresses.
__global__ __launch_bounds__(kRadixThreads) void k_digit_scatter(
    const int32_t *keys, const int32_t *vals, int32_t n, int shift, bool descending,
    int32_t ntiles, const int32_t *offs, int32_t *keys_out, int32_t *vals_out)
{
    constexpr int kWaves = kRadixThreads / 64;
    __shared__ int32_t s_key[kTile], s_val[kTile];  // the tile in digit order
    __shared__ int32_t start[256];                  // first slot of each digit
    __shared__ int32_t run[256];                    // next free slot of each digit
    __shared__ int32_t wcnt[kWaves][256];           // this step's count per wave, digit
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int64_t base = (int64_t)blockIdx.x * kTile;
    const int tn = (int)min((int64_t)kTile, (int64_t)n - base);
    run[tid] = 0;
    for (int k = 0; k < kWaves; ++k) wcnt[k][tid] = 0;
    __syncthreads();
    for (int j = 0; j < kRadixSteps; ++j) {
        const int64_t i = base + j * kRadixThreads + tid;
        if (i < n) atomicAdd(&run[rdigit(keys[i], shift, descending)], 1);
    }
    __syncthreads();
    // exclusive scan of the tile's digit counts
    const int cnt = run[tid];
    start[tid] = cnt;
    __syncthreads();
    for (int off = 1; off < 256; off <<= 1) {
        const int t = tid >= off ? start[tid - off] : 0;
        __syncthreads();
        start[tid] += t;
        __syncthreads();
    }
    const int excl = start[tid] - cnt;
    __syncthreads();
    start[tid] = excl;
    run[tid] = excl;
    __syncthreads();
    const uint64_t below = (1ull << lane) - 1ull;
    for (int j = 0; j < kRadixSteps; ++j) {
        const int64_t i = base + j * kRadixThreads + tid;
        const bool valid = i < n;
        const int32_t key = valid ? keys[i] : 0;
        const int d = valid ? rdigit(key, shift, descending) : 0;
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
            int slot = run[d] + rank;
            for (int k = 0; k < wv; ++k) slot += wcnt[k][d];
            s_key[slot] = key;
            s_val[slot] = vals[i];
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
    for (int q = tid; q < tn; q += kRadixThreads) {
        const int32_t key = s_key[q];
        const int d = rdigit(key, shift, descending);
        const int64_t g = offs[(int64_t)d * ntiles + blockIdx.x] + (q - start[d]);
        keys_out[g] = key;
        vals_out[g] = s_val[q];
    }
}

}  // namespace

int64_t radix_count_ints(int32_t n)
{
    const int64_t ntiles = (n + kTile - 1) / kTile;
    return 256 * (ntiles > 0 ? ntiles : 1) + 1;
}

hipError_t launch_radix_pairs(const int32_t *keys, const int32_t *vals, int32_t n,
                              int32_t max_key, bool descending, const RadixScratch &rs,
                              const int32_t **keys_out, const int32_t **vals_out,
                              hipStream_t s)
{
    const int32_t *kin = keys, *vin = vals;
    if (n > 0) {
        const int32_t ntiles = (n + kTile - 1) / kTile;
        const int32_t cells = 256 * ntiles;
        int32_t *kout = rs.keys_a, *vout = rs.vals_a;
        for (int shift = 0; shift == 0 || (shift < 31 && (max_key >> shift) != 0);
             shift += 8) {
            k_digit_count<<<ntiles, kRadixThreads, 0, s>>>(kin, n, shift, descending, ntiles,
                                                            rs.counts);
            hipError_t e = hipGetLastError();
            if (e != hipSuccess) return e;
            e = launch_scan(rs.counts, rs.counts, cells, rs.scan_tmp, nullptr, s);
            if (e != hipSuccess) return e;
            k_digit_scatter<<<ntiles, kRadixThreads, 0, s>>>(kin, vin, n, shift, descending,
                                                              ntiles, rs.counts, kout, vout);
            if ((e = hipGetLastError()) != hipSuccess) return e;
            kin = kout;
            vin = vout;
            kout = kout == rs.keys_a ? rs.keys_b : rs.keys_a;
            vout = vout == rs.vals_a ? rs.vals_b : rs.vals_a;
        }
    }
    *keys_out = kin;
    *vals_out = vin;
    return hipSuccess;
}

}  // namespace f3s
