// Stable least-significant-digit radix sort of (key, value) pairs of int32,
// keys in [0, max_key], ascending or descending, with 8-bit digits (one pass
// per 8 bits of max_key): per tile of kTile keys a digit histogram, one scan
// over (digit, tile), then a stable scatter in which each tile ranks its keys
// (each wavefront its quarter, in order, equal digits by ballots) into digit
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
    const int64_t base = (int64_t)blockIdx.x * kTile + tid;
    int32_t key[kRadixSteps];
#pragma unroll
    for (int j = 0; j < kRadixSteps; ++j) {
        const int64_t i = base + j * kRadixThreads;
        key[j] = i < n ? keys[i] : 0;
    }
    h[tid] = 0;
    __syncthreads();
#pragma unroll
    for (int j = 0; j < kRadixSteps; ++j)
        if (base + j * kRadixThreads < n) atomicAdd(&h[rdigit(key[j], shift, descending)], 1);
    __syncthreads();
    counts[(int64_t)tid * ntiles + blockIdx.x] = h[tid];
}

// Stable scatter of one tile.  Wavefront w holds elements [1024 w,
// 1024 (w + 1)) of the tile in registers (lane l has elements 64 j + l) and
// ranks them in order without barriers: per 64 keys, a key's rank among
// equal digits comes from ballots, added to the wave's running count of that
// digit in LDS.  One scan over the digits then gives each wave the first
// slot of each digit, the tile is placed in LDS in digit order and written
// out run by run, so each digit's keys go to consecutive addresses.
__global__ __launch_bounds__(kRadixThreads) void k_digit_scatter(
    const int32_t *keys, const int32_t *vals, int32_t n, int shift, bool descending,
    int32_t ntiles, const int32_t *offs, int32_t *keys_out, int32_t *vals_out)
{
    constexpr int kWaves = kRadixThreads / 64;
    constexpr int kPerWave = kTile / kWaves;
    __shared__ int32_t s_key[kTile], s_val[kTile];  // the tile in digit order
    __shared__ int32_t wave_digit[kWaves][256];     // count, then first slot, per wave and digit
    __shared__ int32_t start[256];                  // first slot of each digit
    __shared__ int32_t wave_sum[kWaves];
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int64_t base = (int64_t)blockIdx.x * kTile;
    const int tn = (int)min((int64_t)kTile, (int64_t)n - base);
    const int q0 = wv * kPerWave + lane;
    int32_t key[kRadixSteps], val[kRadixSteps], rank[kRadixSteps];
#pragma unroll
    for (int j = 0; j < kRadixSteps; ++j) {
        const int q = q0 + 64 * j;
        key[j] = q < tn ? keys[base + q] : 0;
        val[j] = q < tn ? (vals ? vals[base + q] : (int32_t)(base + q)) : 0;
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) wave_digit[wv][lane + 64 * k] = 0;
    const uint64_t below = (1ull << lane) - 1ull;
#pragma unroll
    for (int j = 0; j < kRadixSteps; ++j) {
        const bool valid = q0 + 64 * j < tn;
        const int d = rdigit(key[j], shift, descending);
        uint64_t peers = __ballot(valid);
#pragma unroll
        for (int b = 0; b < 8; ++b) {
            const uint64_t bal = __ballot(valid && ((d >> b) & 1));
            peers &= ((d >> b) & 1) ? bal : ~bal;
        }
        const int r = __popcll(peers & below);
        // a wave's LDS accesses take effect in program order, so every lane
        // reads the count before the digit's first lane updates it
        const int prior = valid ? wave_digit[wv][d] : 0;
        rank[j] = prior + r;
        if (valid && r == 0) wave_digit[wv][d] = prior + __popcll(peers);
    }
    __syncthreads();
    // thread t: digit t's count over the tile, its first slot, each wave's
    int c[kWaves], tot = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
        c[w] = wave_digit[w][tid];
        tot += c[w];
    }
    const int incl = wave_inclusive_sum(tot, lane);
    if (lane == 63) wave_sum[wv] = incl;
    __syncthreads();
    int first = incl - tot;
    for (int w = 0; w < wv; ++w) first += wave_sum[w];
    start[tid] = first;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
        wave_digit[w][tid] = first;
        first += c[w];
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < kRadixSteps; ++j) {
        if (q0 + 64 * j < tn) {
            const int slot = wave_digit[wv][rdigit(key[j], shift, descending)] + rank[j];
            s_key[slot] = key[j];
            s_val[slot] = val[j];
        }
    }
    __syncthreads();
    for (int q = tid; q < tn; q += kRadixThreads) {
        const int32_t k = s_key[q];
        const int d = rdigit(k, shift, descending);
        const int64_t g = offs[(int64_t)d * ntiles + blockIdx.x] + (q - start[d]);
        keys_out[g] = k;
        vals_out[g] = s_val[q];
    }
}

}  // namespace

int radix_passes(int32_t max_key)
{
    int passes = 1;
    for (int shift = 8; shift < 31 && (max_key >> shift) != 0; shift += 8) ++passes;
    return passes;
}

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
        const int passes = radix_passes(max_key);
        for (int shift = 0; shift < 8 * passes; shift += 8) {
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
