// Plan construction on the GPU: CSR -> Binary Sparse Block layout
// (Section 3.1) and the heavy-first work list (Section 3.2).
//
//  1. row_ptr validation
//  2. per row window: sorted distinct columns and the window's 256-bit block
//     bitmaps, staged at offsets fixed by the CSR (one wavefront per window
//     with a register bitonic sort; larger windows a workgroup LDS sort;
//     heavier windows a column bitmap in LDS with popcount ranks, walked in
//     chunks of 2^17 columns)
//  3. blocks per window (ceil(u/16)) and their exclusive prefix (tro)
//  4. padded column lists (sptd) and bitmaps copied to their final blocks
//  5. work list keys: block count per window (the stable sort, largest
//     first, is worklist.hip's), windows above `piece` blocks split into
//     pieces of whole block pairs
//
// Every kernel is deterministic: integer atomics only commute (bitwise OR,
// counters whose final value is all that is read), and every position in
// the output is owned by exactly one thread.
#include <limits.h>

#include "f3s_internal.h"

// Dynamic LDS of k_heavy_lds (declared at global scope: this file is also
// built as relocatable device code, where a block-scope declaration inside
// the anonymous namespace would name an undefined internal variable).
extern __shared__ uint32_t f3s_heavy_lds_dyn[];

namespace f3s {
namespace {

constexpr int kSortCap = 4096;     // entries a window may have for LDS sort
// Staging offset (in 32-bit words) of window w's bitmaps, whose CSR entries
// start at beg.  A window with n entries has at most ceil(n/16) blocks, 8n/16
// + 8 words at most, and the next window's offset lies at least n/2 + 8
// words further on, so the regions never overlap; all of them fit in
// nnz/2 + 8T + 8 words.
__device__ __forceinline__ int64_t mask_stage(int32_t beg, int32_t w)
{
    return (int64_t)(beg >> 1) + 8 * (int64_t)w;
}

// Orders the LDS accesses of one wavefront (the wave's LDS operations run in
// issue order, so only the compiler has to be kept from moving them).
__device__ __forceinline__ void wave_lds_order()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ int wave_excl_scan(int v, int lane, int *total)
{
    int incl = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int t = __shfl_up(incl, o);
        if (lane >= o) incl += t;
    }
    *total = __shfl(incl, 63);
    return incl - v;
}

// Compare-exchange of x with the x of lane ^ lj (lj a power of two below
// 64): the smaller of the two if take_min, else the larger.  The partner's
// value comes from cross-lane moves that stay in the vector ALU: DPP quad
// permutations (lj = 1, 2) and row rotations (lj = 4, 8; rotation by n
// within 16 lanes delivers lane i - n, probed on the GPU), and the gfx950
// permlane swaps (lj = 16, 32), which give each lane the pair of its own and
// its partner's value in some order; min and max do not depend on it.  lj
// is a constant once the sorting network is unrolled.
__device__ __forceinline__ int xchg_lanes(int x, int lj, int lane, bool take_min)
{
    int a = x, b;
    switch (lj) {
    case 1: b = __builtin_amdgcn_mov_dpp(x, 0xB1, 0xF, 0xF, false); break;  // [1,0,3,2]
    case 2: b = __builtin_amdgcn_mov_dpp(x, 0x4E, 0xF, 0xF, false); break;  // [2,3,0,1]
    case 4: {
        const int from_below = __builtin_amdgcn_mov_dpp(x, 0x124, 0xF, 0xF, false);  // i - 4
        const int from_above = __builtin_amdgcn_mov_dpp(x, 0x12C, 0xF, 0xF, false);  // i + 4
        b = (lane & 4) ? from_below : from_above;
        break;
    }
    case 8: b = __builtin_amdgcn_mov_dpp(x, 0x128, 0xF, 0xF, false); break;  // i +- 8
    case 16: {
        const auto r = __builtin_amdgcn_permlane16_swap(x, x, false, false);
        a = (int)r[0];
        b = (int)r[1];
        break;
    }
    default: {
        const auto r = __builtin_amdgcn_permlane32_swap(x, x, false, false);
        a = (int)r[0];
        b = (int)r[1];
        break;
    }
    }
    return take_min ? min(a, b) : max(a, b);
}

// Bitonic sorting network, ascending, over the 64*E keys of one wavefront:
// key t = E*lane + i sits in x[i] of lane `lane`.  Compare distances below E
// stay inside a lane, larger ones pair lanes lane and lane ^ (j/E).
template <int E>
__device__ __forceinline__ void wave_bitonic(int (&x)[E], int lane)
{
#pragma unroll
    for (int k = 2; k <= 64 * E; k <<= 1) {
#pragma unroll
        for (int j = k >> 1; j > 0; j >>= 1) {
            if (j >= E) {
                const bool lower = (lane & (j / E)) == 0;
#pragma unroll
                for (int i = 0; i < E; ++i) {
                    const bool up = ((E * lane + i) & k) == 0;
                    x[i] = xchg_lanes(x[i], j / E, lane, lower == up);
                }
            } else {
#pragma unroll
                for (int i = 0; i < E; ++i) {
                    if (i & j) continue;
                    const bool up = ((E * lane + i) & k) == 0;
                    const int a = x[i], b = x[i | j];
                    x[i] = up ? min(a, b) : max(a, b);
                    x[i | j] = up ? max(a, b) : min(a, b);
                }
            }
        }
    }
}

// Entries a window may have for the one-wave path over all windows (8 keys
// per lane); windows up to kWaveCap16 entries get a second one-wave pass with
// 16 keys per lane, launched over the larger windows only (its registers
// would cut the occupancy of the first pass threefold).
constexpr int kWaveCap = 512;
constexpr int kWaveCap16 = 1024;

// Window of n <= 64*E entries starting at CSR offset beg; lanes 0..nr of rp
// hold the window's row starts (INT_MAX above).  Writes the sorted distinct
// columns to tmp_cols[beg..), the block bitmaps to their staging region, u[w]
// and the number of set bits to bits[w].
template <int E>
__device__ void window_wave(const int32_t *col_idx, int32_t N, int32_t w, int32_t beg,
                            int32_t n, int32_t rp, int lane, int32_t *s_cols,
                            uint32_t *s_mask, int32_t *tmp_cols, uint32_t *tmp_mask,
                            int32_t *u, int32_t *bits_out, int32_t *err)
{
    int x[E];
#pragma unroll
    for (int i = 0; i < E; ++i) {
        const int e = 64 * i + lane;  // coalesced loads; a sort input's order is free
        int v = INT_MAX;
        if (e < n) {
            v = col_idx[beg + e];
            if (v < 0 || v >= N) {
                atomicOr(err, 1);
                v = INT_MAX;
            }
        }
        x[i] = v;
    }
    wave_bitonic<E>(x, lane);

    // distinct keys in sorted order, compacted by a wave prefix sum
    const int before = __shfl_up(x[E - 1], 1);
    uint32_t first = 0;
#pragma unroll
    for (int i = 0; i < E; ++i) {
        const int prev = i ? x[i - 1] : before;
        if (x[i] != INT_MAX && ((lane == 0 && i == 0) || x[i] != prev)) first |= 1u << i;
    }
    int total;
    int off = wave_excl_scan(__popc(first), lane, &total);
#pragma unroll
    for (int i = 0; i < E; ++i)
        if (first & (1u << i)) {
            tmp_cols[beg + off] = x[i];
            s_cols[off] = x[i];
            ++off;
        }
    const int nbw = (total + kBlockCols - 1) / kBlockCols;
    for (int k = lane; k < kMaskWords * nbw; k += 64) s_mask[k] = 0;
    wave_lds_order();

    // one bit per entry: row from the row starts, compacted column by binary
    // search in the distinct list
    int starts[kWindowRows - 1];  // wave-uniform: scalar registers
#pragma unroll
    for (int r = 1; r < kWindowRows; ++r) starts[r - 1] = __builtin_amdgcn_readlane(rp, r);
#pragma unroll
    for (int i = 0; i < E; ++i) {
        const int e = 64 * i + lane;
        if (e >= n) continue;
        const int c = col_idx[beg + e];  // again (cache-resident) to spare registers
        if (c < 0 || c >= N) continue;
        int row = 0;
#pragma unroll
        for (int r = 1; r < kWindowRows; ++r) row += beg + e >= starts[r - 1];
        // position of c in the distinct list (it is there): a fixed-step,
        // branch-free search, so the E searches of a lane interleave
        int lo = 0;
#pragma unroll
        for (int step = 32 * E; step > 0; step >>= 1)
            if (lo + step <= total && s_cols[lo + step - 1] < c) lo += step;
        if (lo >= total) continue;  // every valid column is in the list
        const int cc = lo % kBlockCols;
        const int bit = 4 * (row + 16 * (cc / 4)) + (cc % 4);
        atomicOr(&s_mask[kMaskWords * (lo / kBlockCols) + bit / 32], 1u << (bit % 32));
    }
    wave_lds_order();
    uint32_t *gm = tmp_mask + mask_stage(beg, w);
    int bits = 0;
    for (int k = lane; k < kMaskWords * nbw; k += 64) {
        const uint32_t m = s_mask[k];
        gm[k] = m;
        bits += __popc(m);
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) bits += __shfl_xor(bits, o);
    if (lane == 0) {
        u[w] = total;
        bits_out[w] = bits;
    }
}

// Loads a window's row starts into lanes 0..nr of the wave (INT_MAX above).
__device__ __forceinline__ int32_t window_row_starts(const int32_t *row_ptr, int32_t N,
                                                     const int32_t *win_row, int32_t w,
                                                     int lane, int32_t *beg, int32_t *n)
{
    int32_t r0, nr;
    window_rows(win_row, N, w, &r0, &nr);
    const int32_t rp = lane <= nr ? row_ptr[r0 + lane] : INT_MAX;
    *beg = __shfl(rp, 0);
    *n = __shfl(rp, nr) - *beg;
    return rp;
}

// One wavefront (one workgroup) per window.  Windows with more than kWaveCap
// entries are flagged in is_big (up to kSortCap entries) or is_heavy for the
// later passes.  (No counter shared by all windows: atomics on one address
// serialise, tens of ns each.)
__global__ __launch_bounds__(64) void k_window_wave(
    const int32_t *row_ptr, const int32_t *col_idx, int32_t N, const int32_t *win_row,
    int32_t *tmp_cols, uint32_t *tmp_mask, int32_t *u, int32_t *is_big, int32_t *is_heavy,
    int32_t *bits_out, int32_t *err)
{
    __shared__ int32_t s_cols[kWaveCap];
    __shared__ uint32_t s_mask[kWaveCap / kBlockCols * kMaskWords];
    const int lane = threadIdx.x;
    const int w = blockIdx.x;
    // k_check_row_ptr ran before on the same stream: a malformed row_ptr
    // stops every wave here, before any column is read (is_big stays valid
    // for the scan that follows)
    if (*(volatile int32_t *)err) {
        if (lane == 0) is_big[w] = is_heavy[w] = 0;
        return;
    }
    int32_t beg, n;
    const int32_t rp = window_row_starts(row_ptr, N, win_row, w, lane, &beg, &n);
    if (lane == 0) {
        is_big[w] = n > kWaveCap && n <= kSortCap;
        is_heavy[w] = n > kSortCap;
    }
    if (n > kWaveCap) return;
    if (n <= 64)
        window_wave<1>(col_idx, N, w, beg, n, rp, lane, s_cols, s_mask, tmp_cols,
                       tmp_mask, u, bits_out, err);
    else if (n <= 128)
        window_wave<2>(col_idx, N, w, beg, n, rp, lane, s_cols, s_mask, tmp_cols,
                       tmp_mask, u, bits_out, err);
    else if (n <= 256)
        window_wave<4>(col_idx, N, w, beg, n, rp, lane, s_cols, s_mask, tmp_cols,
                       tmp_mask, u, bits_out, err);
    else
        window_wave<8>(col_idx, N, w, beg, n, rp, lane, s_cols, s_mask, tmp_cols,
                       tmp_mask, u, bits_out, err);
}

// The windows of `big` with kWaveCap < n <= kWaveCap16 entries, one wavefront
// each with 16 keys per lane; the others are left to k_window_sort.
__global__ __launch_bounds__(64) void k_window_wave16(
    const int32_t *row_ptr, const int32_t *col_idx, int32_t N, const int32_t *win_row,
    const int32_t *big, int32_t *tmp_cols, uint32_t *tmp_mask, int32_t *u,
    int32_t *bits_out, int32_t *err)
{
    __shared__ int32_t s_cols[kWaveCap16];
    __shared__ uint32_t s_mask[kWaveCap16 / kBlockCols * kMaskWords];
    const int lane = threadIdx.x;
    const int w = big[blockIdx.x];
    int32_t beg, n;
    const int32_t rp = window_row_starts(row_ptr, N, win_row, w, lane, &beg, &n);
    if (n <= kWaveCap || n > kWaveCap16) return;
    window_wave<16>(col_idx, N, w, beg, n, rp, lane, s_cols, s_mask, tmp_cols, tmp_mask,
                    u, bits_out, err);
}

__global__ void k_check_row_ptr(const int32_t *row_ptr, int32_t N, int32_t nnz,
                                int32_t *err)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i > N) return;
    const int32_t a = row_ptr[i];
    bool bad = a < 0 || a > nnz;
    if (i == 0) bad |= a != 0;
    if (i < N) bad |= row_ptr[i + 1] < a;
    if (bad) atomicOr(err, 1);
}

// Windows of the list `big` with more than kWaveCap16 entries (at most
// kSortCap), one workgroup each: bitonic sort of kSortCap keys (the window's
// columns padded with INT_MAX), 4 per thread in registers -- key t = 4 tid +
// i -- so compare distances 1 and 2 stay in a thread, 4 .. 128 pair lanes of
// a wavefront (xchg_lanes) and only the 10 steps of distance 256 and more go
// through LDS (double-buffered: one barrier each); then compaction into
// tmp_cols and u, and the block bitmaps assembled in LDS and stored to the
// staging area, their set bits to bits[w].
constexpr int kSortThreads = 1024;
constexpr int kSortPer = kSortCap / kSortThreads;  // keys per thread

// Exclusive scan of one int per thread over a workgroup of kSortThreads.
__device__ int block_excl_scan_sort(int v, int *lds, int *total)
{
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    int wt;
    const int x = wave_excl_scan(v, lane, &wt);
    if (lane == 0) lds[wv] = wt;
    __syncthreads();
    int before = 0, all = 0;
    for (int k = 0; k < kSortThreads / 64; ++k) {
        const int c = lds[k];
        before += k < wv ? c : 0;
        all += c;
    }
    *total = all;
    __syncthreads();
    return before + x;
}

__global__ __launch_bounds__(kSortThreads) void k_window_sort(
    const int32_t *row_ptr, const int32_t *col_idx, int32_t N, const int32_t *win_row,
    const int32_t *big, int32_t *tmp_cols, uint32_t *tmp_mask, int32_t *u,
    int32_t *bits_out, int32_t *err)
{
    static_assert(kSortPer == 4, "the register network assumes 4 keys per thread");
    __shared__ int32_t xbuf[2][kSortCap];  // cross-wave exchanges, then the distinct list
    __shared__ int scan[kSortThreads / 64];
    __shared__ int32_t edge[kSortThreads / 64];
    __shared__ uint32_t s_mask[kSortCap / kBlockCols * kMaskWords];
    __shared__ int32_t s_rp[kWindowRows + 1];
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int w = big[blockIdx.x];
    int32_t r0, nr;
    window_rows(win_row, N, w, &r0, &nr);
    const int beg = row_ptr[r0];
    const int n = row_ptr[r0 + nr] - beg;
    if (n <= kWaveCap16 || n > kSortCap) return;  // k_window_wave16 / heavy paths
    if (tid <= nr) s_rp[tid] = row_ptr[r0 + tid];
    int x[kSortPer];
#pragma unroll
    for (int i = 0; i < kSortPer; ++i) {
        const int t = kSortPer * tid + i;
        int v = INT_MAX;
        if (t < n) {
            v = col_idx[beg + t];
            if (v < 0 || v >= N) {
                atomicOr(err, 1);
                v = INT_MAX;
            }
        }
        x[i] = v;
    }
    // bitonic network, ascending
    int buf = 0;
#pragma unroll
    for (int k = 2; k <= kSortCap; k <<= 1) {
#pragma unroll
        for (int j = k >> 1; j > 0; j >>= 1) {
            if (j >= 64 * kSortPer) {
#pragma unroll
                for (int i = 0; i < kSortPer; ++i) xbuf[buf][kSortPer * tid + i] = x[i];
                __syncthreads();
#pragma unroll
                for (int i = 0; i < kSortPer; ++i) {
                    const int t = kSortPer * tid + i;
                    const int p = xbuf[buf][t ^ j];
                    const bool take_min = ((t & j) == 0) == ((t & k) == 0);
                    x[i] = take_min ? min(x[i], p) : max(x[i], p);
                }
                buf ^= 1;
            } else if (j >= kSortPer) {
                const int lj = j / kSortPer;
                const bool lower = (lane & lj) == 0;
#pragma unroll
                for (int i = 0; i < kSortPer; ++i) {
                    const bool up = ((kSortPer * tid + i) & k) == 0;
                    x[i] = xchg_lanes(x[i], lj, lane, lower == up);
                }
            } else {
#pragma unroll
                for (int i = 0; i < kSortPer; ++i) {
                    if (i & j) continue;
                    const bool up = ((kSortPer * tid + i) & k) == 0;
                    const int a = x[i], b = x[i | j];
                    x[i] = up ? min(a, b) : max(a, b);
                    x[i | j] = up ? max(a, b) : min(a, b);
                }
            }
        }
    }
    // distinct values: key t is new if it differs from key t - 1 (the last
    // key of the previous thread: a lane move, or across waves through LDS)
    if (lane == 63) edge[wv] = x[kSortPer - 1];
    __syncthreads();
    int prev = __shfl_up(x[kSortPer - 1], 1);
    if (lane == 0) prev = wv ? edge[wv - 1] : INT_MIN;
    uint32_t first = 0;
#pragma unroll
    for (int i = 0; i < kSortPer; ++i) {
        const int pv = i ? x[i - 1] : prev;
        if (x[i] != INT_MAX && x[i] != pv) first |= 1u << i;
    }
    int total;
    int off = block_excl_scan_sort(__popc(first), scan, &total);
    // the distinct list goes to xbuf[buf], whose last reads were separated from
    // these writes by the scan's barriers
    int32_t *list = xbuf[buf];
#pragma unroll
    for (int i = 0; i < kSortPer; ++i)
        if (first & (1u << i)) {
            tmp_cols[beg + off] = x[i];
            list[off] = x[i];
            ++off;
        }
    const int nbw = (total + kBlockCols - 1) / kBlockCols;
    for (int k = tid; k < kMaskWords * nbw; k += kSortThreads) s_mask[k] = 0;
    __syncthreads();
    // one bit per entry: row among the row starts, compacted column by binary
    // search in the distinct list
    for (int e = tid; e < n; e += kSortThreads) {
        const int c = col_idx[beg + e];
        if (c < 0 || c >= N) continue;
        int row = 0;
        for (int r = 1; r < nr; ++r) row += beg + e >= s_rp[r];
        int a = 0, b = total;
        while (a < b) {
            const int mid = (a + b) >> 1;
            if (list[mid] < c) a = mid + 1;
            else b = mid;
        }
        if (a >= total) continue;  // every valid column is in the list
        const int cc = a % kBlockCols;
        const int bit = 4 * (row + 16 * (cc / 4)) + (cc % 4);
        atomicOr(&s_mask[kMaskWords * (a / kBlockCols) + bit / 32], 1u << (bit % 32));
    }
    __syncthreads();
    uint32_t *gm = tmp_mask + mask_stage(beg, w);
    int cnt = 0;
    for (int k = tid; k < kMaskWords * nbw; k += kSortThreads) {
        const uint32_t m = s_mask[k];
        gm[k] = m;
        cnt += __popc(m);
    }
    int nbits;
    (void)block_excl_scan_sort(cnt, scan, &nbits);
    if (tid == 0) {
        u[w] = total;
        bits_out[w] = nbits;
    }
}

// Heavy windows (more than kSortCap entries), one workgroup each.  The column
// range is walked in chunks of kChunkCols: a chunk's columns are marked in a
// bitmap in LDS and a prefix popcount over its words ranks them, so every
// entry's compacted column is (distinct columns of earlier chunks) + rank +
// popcount of the lower bits of its word; no search.  A first walk counts the
// distinct columns (for the size of the block bitmaps), the second writes
// them in order to tmp_cols and sets the entries' bits, in LDS when the
// bitmaps fit (mask_words: what the LDS budget leaves after the chunk
// bitmap and ranks), else with atomics on the staging area.  On
// graphs of up to kChunkCols nodes the first walk's bitmap is reused.
constexpr int kHeavyThreads = 1024;
constexpr int kChunkCols = 1 << 17;       // 16 KB bitmap + 16 KB ranks
// LDS of one workgroup: two of them (2 x 1024 threads) still fit a CU.
constexpr int kHeavyLdsBytes = 76 * 1024;

__global__ __launch_bounds__(kHeavyThreads) void k_heavy_lds(
    const int32_t *row_ptr, const int32_t *col_idx, int32_t N, const int32_t *win_row,
    const int32_t *heavy, int32_t *tmp_cols, uint32_t *tmp_mask, int32_t *u,
    int32_t *bits_out, int32_t *err, int32_t mask_words)
{
    uint32_t *lds = f3s_heavy_lds_dyn;  // [cw] bitmap, [cw] ranks, [mask_words]
    __shared__ int32_t s_rp[kWindowRows + 1];
    __shared__ int scan[kHeavyThreads / 64];
    const int tid = threadIdx.x;
    const int cw = (min(N, kChunkCols) + 31) / 32;  // bitmap words of one chunk
    uint32_t *bm = lds;
    int32_t *rank = (int32_t *)(lds + cw);
    uint32_t *sm = lds + 2 * cw;
    const int w = heavy[blockIdx.x];
    int32_t r0, nr;
    window_rows(win_row, N, w, &r0, &nr);
    if (tid <= nr) s_rp[tid] = row_ptr[r0 + tid];
    __syncthreads();
    const int beg = s_rp[0], n = s_rp[nr] - beg;
    const int nchunk = (N + kChunkCols - 1) / kChunkCols;
    // A thread ORs the bits of its successive entries that land in the same
    // word in a register, with one atomic per change of word (a window's
    // entries often repeat a few words: banded rows, sorted rows), and
    // follows its row incrementally.  With one column chunk each thread takes
    // a contiguous run of entries (most repeats); with several, whose walks
    // re-read the entries once per chunk, entries are strided over the
    // threads so the loads stay coalesced (measured: contiguous runs cost 23%
    // there).
    const int per = (n + kHeavyThreads - 1) / kHeavyThreads;
    const int e0 = nchunk == 1 ? min(tid * per, n) : tid;
    const int e1 = nchunk == 1 ? min(e0 + per, n) : n;
    const int es = nchunk == 1 ? 1 : kHeavyThreads;
    // marks the columns of chunk q in bm (zeroed first)
    auto mark = [&](int q, bool report) {
        for (int k = tid; k < cw; k += kHeavyThreads) bm[k] = 0;
        __syncthreads();
        const int c0 = q * kChunkCols;
        int cur = -1;
        uint32_t acc = 0;
        for (int e = e0; e < e1; e += es) {
            const int c = col_idx[beg + e];
            if (c < 0 || c >= N) {
                if (report) atomicOr(err, 1);
                continue;
            }
            if (c < c0 || c - c0 >= kChunkCols) continue;
            const int wd = (c - c0) >> 5;
            if (wd != cur) {
                if (acc) atomicOr(&bm[cur], acc);
                cur = wd;
                acc = 0;
            }
            acc |= 1u << (c & 31);
        }
        if (acc) atomicOr(&bm[cur], acc);
        __syncthreads();
    };
    const int ch = (cw + kHeavyThreads - 1) / kHeavyThreads;
    const int lo = min(tid * ch, cw), hi = min(lo + ch, cw);
    // walk 1: distinct columns
    int total = 0, first_off = 0;  // first_off: this thread's rank offset (one chunk)
    for (int q = 0; q < nchunk; ++q) {
        mark(q, q == 0);
        int cnt = 0;
        for (int k = lo; k < hi; ++k) cnt += __popc(bm[k]);
        int t;
        first_off = block_excl_scan_sort(cnt, scan, &t);
        total += t;
    }
    const int nbw = (total + kBlockCols - 1) / kBlockCols;
    const bool in_lds = kMaskWords * nbw <= mask_words;
    uint32_t *gm = tmp_mask + mask_stage(beg, w);
    uint32_t *dst = in_lds ? sm : gm;
    for (int k = tid; k < kMaskWords * nbw; k += kHeavyThreads) dst[k] = 0;
    __threadfence_block();  // global staging: only this workgroup's atomics (at the L2)
    __syncthreads();
    // walk 2: ranks, distinct columns in order, the entries' bits
    int base = 0;
    for (int q = 0; q < nchunk; ++q) {
        const int c0 = q * kChunkCols;
        int t, off;
        if (nchunk == 1) {  // walk 1's bitmap and offsets still hold
            t = total;
            off = first_off;
        } else {
            mark(q, false);
            int cnt = 0;
            for (int k = lo; k < hi; ++k) cnt += __popc(bm[k]);
            off = base + block_excl_scan_sort(cnt, scan, &t);
        }
        for (int k = lo; k < hi; ++k) {
            rank[k] = off;
            uint32_t x = bm[k];
            while (x) {
                tmp_cols[beg + off++] = c0 + 32 * k + __ffs(x) - 1;
                x &= x - 1;
            }
        }
        __syncthreads();
        int row = 0, cur = -1;
        uint32_t acc = 0;
        for (int e = e0; e < e1; e += es) {
            while (row + 1 < nr && beg + e >= s_rp[row + 1]) ++row;
            const int c = col_idx[beg + e];
            if (c < c0 || c >= N || c - c0 >= kChunkCols) continue;
            const int cl = c - c0;
            const uint32_t below = bm[cl >> 5] & ((1u << (cl & 31)) - 1u);
            const int a = rank[cl >> 5] + __popc(below);
            const int cc = a % kBlockCols;
            const int bit = 4 * (row + 16 * (cc / 4)) + (cc % 4);
            const int wd = kMaskWords * (a / kBlockCols) + bit / 32;
            if (wd != cur) {
                if (acc) atomicOr(&dst[cur], acc);
                cur = wd;
                acc = 0;
            }
            acc |= 1u << (bit % 32);
        }
        if (acc) atomicOr(&dst[cur], acc);
        base += t;
        __syncthreads();
    }
    __threadfence_block();
    __syncthreads();
    int nb_bits = 0;
    for (int k = tid; k < kMaskWords * nbw; k += kHeavyThreads) {
        uint32_t m;
        if (in_lds) {
            m = sm[k];
            gm[k] = m;
        } else {
            m = __hip_atomic_load(&gm[k], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        nb_bits += __popc(m);
    }
    int all_bits;
    (void)block_excl_scan_sort(nb_bits, scan, &all_bits);
    if (tid == 0) {
        u[w] = total;
        bits_out[w] = all_bits;
    }
}


// Per window: blocks nb = ceil(u/16); over all windows: sum of u (distinct
// columns), sum of bits (distinct entries), sum of nb (blocks) and the
// largest nb.  Grid-stride, then a workgroup reduction and one atomic per
// statistic and workgroup.
constexpr int kStatThreads = 256;
constexpr int kStatBlocks = 64;

__global__ __launch_bounds__(kStatThreads) void k_window_stats(
    const int32_t *u, const int32_t *bits, int32_t T, int32_t *nb,
    unsigned long long *sum_u, unsigned long long *sum_bits, int32_t *sum_nb,
    int32_t *max_nb)
{
    __shared__ unsigned long long part[3][kStatThreads / 64];
    __shared__ int32_t pmax[kStatThreads / 64];
    unsigned long long su = 0, sb = 0, sn = 0;
    int32_t mx = 0;
    for (int64_t w = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; w < T;
         w += (int64_t)gridDim.x * blockDim.x) {
        const int32_t uw = u[w];
        const int32_t b = (uw + kBlockCols - 1) / kBlockCols;
        nb[w] = b;
        su += (unsigned long long)uw;
        sb += (unsigned long long)bits[w];
        sn += (unsigned long long)b;
        mx = max(mx, b);
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        su += __shfl_xor(su, o);
        sb += __shfl_xor(sb, o);
        sn += __shfl_xor(sn, o);
        mx = max(mx, __shfl_xor(mx, o));
    }
    const int wv = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) {
        part[0][wv] = su;
        part[1][wv] = sb;
        part[2][wv] = sn;
        pmax[wv] = mx;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int k = 1; k < kStatThreads / 64; ++k) {
            su += part[0][k];
            sb += part[1][k];
            sn += part[2][k];
            mx = max(mx, pmax[k]);
        }
        if (su) atomicAdd(sum_u, su);
        if (sb) atomicAdd(sum_bits, sb);
        if (sn) atomicAdd(sum_nb, (int32_t)sn);
        if (mx) atomicMax(max_nb, mx);
    }
}

constexpr int kScanThreads = 1024;
constexpr int kScanItems = 4;
constexpr int kScanTile = kScanThreads * kScanItems;
// Up to this many elements one workgroup scans them in one launch, 16 per
// thread (a second launch costs more than the longer tile).
constexpr int kScanOneLaunch = kScanThreads * 16;
// Up to this many elements the tile totals fit one workgroup's threads.
constexpr int64_t kScanTwoPass = (int64_t)kScanTile * kScanThreads;

__device__ __forceinline__ int scan_element(const ScanArray &a, int64_t i)
{
    return a.gather ? a.in[a.gather[i]] : a.in[i];
}

// tile_sums[tile] = sum of the tile's elements.  blockIdx.y selects one of
// two independent arrays.
__global__ __launch_bounds__(kScanThreads) void k_scan_reduce(ScanArray a0, ScanArray a1,
                                                              int32_t n)
{
    const ScanArray a = blockIdx.y ? a1 : a0;
    __shared__ int32_t wave_sum[kScanThreads / 64];
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int64_t first = ((int64_t)blockIdx.x * kScanThreads + tid) * kScanItems;
    int own = 0;
#pragma unroll
    for (int j = 0; j < kScanItems; ++j) own += first + j < n ? scan_element(a, first + j) : 0;
    const int incl = wave_inclusive_sum(own, lane);
    if (lane == 63) wave_sum[wv] = incl;
    __syncthreads();
    if (tid == 0) {
        int t = 0;
        for (int k = 0; k < kScanThreads / 64; ++k) t += wave_sum[k];
        a.tile_sums[blockIdx.x] = t;
    }
}

enum ScanCarry { kCarryNone, kCarrySumBefore, kCarryScanned };

// Exclusive scan of one tile of kScanThreads * K ints per workgroup, in
// place or not: thread t owns K consecutive elements, so one wavefront sum
// and one barrier cover the tile.  The carry into the tile is 0 (a single
// tile), the sum of the totals of the tiles before it (at most kScanThreads
// of them), or the tile's entry of the already scanned totals.  The last
// tile writes out[n] = total (and *total).  Nonzero elements are listed when
// a list is given.  blockIdx.y selects one of two independent arrays.
template <int K, ScanCarry C>
__global__ __launch_bounds__(kScanThreads) void k_scan(ScanArray a0, ScanArray a1, int32_t n)
{
    const ScanArray a = blockIdx.y ? a1 : a0;
    __shared__ int32_t wave_sum[kScanThreads / 64], wave_carry[kScanThreads / 64];
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int64_t first = ((int64_t)blockIdx.x * kScanThreads + tid) * K;
    int v[K];
#pragma unroll
    for (int j = 0; j < K; ++j) v[j] = first + j < n ? scan_element(a, first + j) : 0;
    int carry_part = 0;
    if (C == kCarrySumBefore && tid < (int)blockIdx.x) carry_part = a.tile_sums[tid];
    int own = 0;
#pragma unroll
    for (int j = 0; j < K; ++j) own += v[j];
    const int incl = wave_inclusive_sum(own, lane);
    if (lane == 63) wave_sum[wv] = incl;
    if (C == kCarrySumBefore) {
        const int c = wave_inclusive_sum(carry_part, lane);
        if (lane == 63) wave_carry[wv] = c;
    }
    __syncthreads();
    int before = 0, total = 0, carry = 0;
#pragma unroll
    for (int k = 0; k < kScanThreads / 64; ++k) {
        const int t = wave_sum[k];
        before += k < wv ? t : 0;
        total += t;
        if (C == kCarrySumBefore) carry += wave_carry[k];
    }
    if (C == kCarryScanned) carry = a.tile_sums[blockIdx.x];
    int run = carry + before + incl - own;
#pragma unroll
    for (int j = 0; j < K; ++j) {
        if (first + j < n) {
            a.out[first + j] = run;
            if (a.list && v[j] && run < n) a.list[run] = (int32_t)(first + j);
        }
        run += v[j];
    }
    if (tid == 0 && blockIdx.x == gridDim.x - 1) {
        a.out[n] = carry + total;
        if (a.total) *a.total = carry + total;
    }
}


// Padded column lists (sptd, -1 past the window's distinct columns) and the
// block bitmaps copied from the staging areas to the window's blocks; one
// workgroup per window (a hub window has thousands of blocks).
__global__ __launch_bounds__(256) void k_fill_windows(
    const int32_t *row_ptr, const int32_t *win_row, const int32_t *tmp_cols,
    const uint32_t *tmp_mask, const int32_t *u, const int32_t *blk_off, int32_t *cols,
    uint32_t *mask)
{
    const int w = blockIdx.x;
    const int32_t beg = row_ptr[win_row ? win_row[w] : w * kWindowRows];
    const int uw = u[w];
    const int64_t ob = blk_off[w];
    const int nbw = blk_off[w + 1] - blk_off[w];
    const int32_t *src = tmp_cols + beg;
    const uint32_t *msrc = tmp_mask + mask_stage(beg, w);
    int32_t *dst = cols + kBlockCols * ob;
    uint32_t *mdst = mask + kMaskWords * ob;
    for (int k = threadIdx.x; k < kBlockCols * nbw; k += 256) dst[k] = k < uw ? src[k] : -1;
    for (int k = threadIdx.x; k < kMaskWords * nbw; k += 256) mdst[k] = msrc[k];
}

// Work-list piece size (even): about n_blocks / slots blocks (slots = 8 per
// CU), so the work list has of the order of 8 items per CU, at least 16
// blocks (smaller pieces help the forward on tiny graphs a little but add
// merge launches to the backward); never above the largest window (a larger
// value splits nothing and only widens the bucket histogram of the work-list
// sort).  forced >= 2 overrides the estimate.
__device__ int32_t plan_piece(int64_t n_blocks, int32_t max_blocks, int32_t forced,
                              int32_t slots)
{
    const int64_t cap = ((int64_t)(max_blocks > 2 ? max_blocks : 2) + 1) & ~1LL;
    int64_t piece;
    if (forced >= 2) {
        piece = forced & ~1;
    } else {
        piece = (n_blocks + slots - 1) / slots;
        if (piece < 16) piece = 16;
        piece = (piece + 1) & ~1LL;
    }
    return (int32_t)(piece < cap ? piece : cap);
}

__global__ void k_bin_keys(const int32_t *nb, int32_t T, const int32_t *n_blocks,
                           const int32_t *max_blocks, int32_t forced, int32_t slots,
                           bool reorder, int32_t *piece_out, int32_t *npieces,
                           int32_t *key, int32_t *split_pieces, int32_t *split_one)
{
    const int w = blockIdx.x * blockDim.x + threadIdx.x;
    const int32_t piece = plan_piece(*n_blocks, *max_blocks, forced, slots);
    if (w == 0) *piece_out = piece;
    if (w >= T) return;
    const int n = nb[w];
    const bool split = n > piece;
    const int np = split ? (n + piece - 1) / piece : 1;
    npieces[w] = np;
    key[w] = reorder ? (split ? piece : n) : 0;
    split_pieces[w] = split ? np : 0;
    split_one[w] = split ? 1 : 0;
}

// Work items of the pieces of split window s (one wavefront per split
// window): piece k of np covers the block pairs [floor(k*pairs/np),
// floor((k+1)*pairs/np)) of the window, pairs = ceil(nb/2).
__global__ __launch_bounds__(256) void k_split_items(const int32_t *merges,
                                                     const int32_t *split_item,
                                                     const int32_t *blk_off,
                                                     int32_t n_split, WorkItem *items)
{
    const int s = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (s >= n_split) return;
    const int w = merges[3 * s], slot = merges[3 * s + 1], np = merges[3 * s + 2];
    const int pos = split_item[s];
    const int b0 = blk_off[w], n = blk_off[w + 1] - b0;
    const int64_t pairs = (n + 1) / 2;
    for (int k = threadIdx.x & 63; k < np; k += 64) {
        const int a = (int)((k * pairs) / np);
        const int b = (int)(((k + 1) * pairs) / np);
        items[pos + k] = WorkItem{w, b0 + 2 * a, b0 + min(n, 2 * b), slot + k};
    }
}

// Integrity check of a finished plan: every work item lies inside its window's
// block range, every block's first slot is a real column and every slot is a
// column or -1, every merge record points at existing partial slots.  Any
// violation sets err (nothing that the fused kernel reads can then be out of
// bounds).
__global__ void k_validate_plan(const int32_t *blk_off, int32_t T, const int32_t *cols,
                                int64_t n_blocks, const WorkItem *items, int32_t n_items,
                                const int32_t *merges, int32_t n_split,
                                int32_t n_pieces, int32_t N, int32_t *err)
{
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    bool bad = false;
    if (t < n_items) {
        const WorkItem it = items[t];
        bad |= it.window < 0 || it.window >= T;
        if (!bad)
            bad |= it.blk_begin < blk_off[it.window] || it.blk_end < it.blk_begin ||
                   it.blk_end > blk_off[it.window + 1];
        bad |= it.slot < -1 || it.slot >= n_pieces;
    }
    if (t < n_blocks) {
        const int32_t *c = cols + kBlockCols * t;
        bad |= c[0] < 0 || c[0] >= N;
        for (int k = 1; k < kBlockCols; ++k) bad |= c[k] < -1 || c[k] >= N;
    }
    if (t < n_split) {
        const int w = merges[3 * t], first = merges[3 * t + 1], np = merges[3 * t + 2];
        bad |= w < 0 || w >= T || first < 0 || np < 1 || first + np > n_pieces;
    }
    if (bad) atomicOr(err, 1);
}

inline unsigned grid_for(int64_t n, int threads)
{
    int64_t g = (n + threads - 1) / threads;
    return (unsigned)(g < 1 ? 1 : g);
}

}  // namespace

hipError_t launch_check_row_ptr(const int32_t *row_ptr, int32_t N, int32_t nnz,
                                int32_t *err, hipStream_t s)
{
    k_check_row_ptr<<<grid_for((int64_t)N + 1, 256), 256, 0, s>>>(row_ptr, N, nnz, err);
    return hipGetLastError();
}

int64_t mask_stage_words(int64_t nnz, int32_t T) { return (nnz >> 1) + 8ll * T + 8; }

hipError_t launch_window_wave(const int32_t *row_ptr, const int32_t *col_idx, int32_t N,
                              const int32_t *win_row, int32_t T, int32_t *tmp_cols,
                              uint32_t *tmp_mask, int32_t *u, int32_t *is_big,
                              int32_t *is_heavy, int32_t *bits, int32_t *err, hipStream_t s)
{
    if (T == 0) return hipSuccess;
    k_window_wave<<<T, 64, 0, s>>>(row_ptr, col_idx, N, win_row, tmp_cols, tmp_mask, u,
                                   is_big, is_heavy, bits, err);
    return hipGetLastError();
}

hipError_t launch_window_sort(const int32_t *row_ptr, const int32_t *col_idx,
                              int32_t N, const int32_t *win_row, const int32_t *big,
                              int32_t n_big, int32_t *tmp_cols, uint32_t *tmp_mask,
                              int32_t *u, int32_t *bits, int32_t *err, hipStream_t s)
{
    if (n_big == 0) return hipSuccess;
    k_window_wave16<<<n_big, 64, 0, s>>>(row_ptr, col_idx, N, win_row, big, tmp_cols,
                                         tmp_mask, u, bits, err);
    k_window_sort<<<n_big, kSortThreads, 0, s>>>(row_ptr, col_idx, N, win_row, big,
                                                 tmp_cols, tmp_mask, u, bits, err);
    return hipGetLastError();
}

hipError_t launch_heavy_lds(const int32_t *row_ptr, const int32_t *col_idx, int32_t N,
                            const int32_t *win_row, const int32_t *heavy, int32_t n_heavy,
                            int32_t *tmp_cols, uint32_t *tmp_mask, int32_t *u,
                            int32_t *bits, int32_t *err, hipStream_t s)
{
    if (n_heavy == 0) return hipSuccess;
    const int cw = (min(N, kChunkCols) + 31) / 32;
    const int mask_words = (kHeavyLdsBytes / 4 - 2 * cw) & ~(kMaskWords - 1);
    const size_t lds = (size_t)(2 * cw + mask_words) * 4;
    k_heavy_lds<<<n_heavy, kHeavyThreads, lds, s>>>(row_ptr, col_idx, N, win_row, heavy,
                                                     tmp_cols, tmp_mask, u, bits, err,
                                                     mask_words);
    return hipGetLastError();
}

hipError_t launch_window_stats(const int32_t *u, const int32_t *bits, int32_t T,
                               int32_t *nb, unsigned long long *sum_u,
                               unsigned long long *sum_bits, int32_t *sum_nb,
                               int32_t *max_nb, hipStream_t s)
{
    if (T == 0) return hipSuccess;
    const unsigned g = grid_for(T, kStatThreads);
    k_window_stats<<<g < kStatBlocks ? g : kStatBlocks, kStatThreads, 0, s>>>(
        u, bits, T, nb, sum_u, sum_bits, sum_nb, max_nb);
    return hipGetLastError();
}

// Up to kScanOneLaunch elements: one launch of one workgroup.  Up to
// kScanTwoPass: the tile totals, then every tile scanned with the sum of the
// totals before it (two launches).  Above: the tile totals, their own scan,
// then the tiles.
int64_t scan_tmp_ints(int64_t n)
{
    const int64_t ntiles = (n + kScanTile - 1) / kScanTile;
    if (n <= kScanTile) return 1;
    if (n <= kScanTwoPass) return 2 * ntiles;
    return ntiles + 1 + scan_tmp_ints(ntiles);
}

hipError_t launch_scan_pair(ScanArray a0, ScanArray a1, int arrays, int32_t n,
                            hipStream_t s)
{
    const int32_t ntiles = (int32_t)((n + kScanTile - 1) / kScanTile);
    if (n <= kScanThreads) {
        k_scan<1, kCarryNone><<<dim3(1, arrays), kScanThreads, 0, s>>>(a0, a1, n);
    } else if (n <= kScanTile) {
        k_scan<kScanItems, kCarryNone><<<dim3(1, arrays), kScanThreads, 0, s>>>(a0, a1, n);
    } else if (n <= kScanOneLaunch) {
        k_scan<kScanOneLaunch / kScanThreads, kCarryNone>
            <<<dim3(1, arrays), kScanThreads, 0, s>>>(a0, a1, n);
    } else {
        k_scan_reduce<<<dim3(ntiles, arrays), kScanThreads, 0, s>>>(a0, a1, n);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        k_scan<kScanItems, kCarrySumBefore>
            <<<dim3(ntiles, arrays), kScanThreads, 0, s>>>(a0, a1, n);
    }
    return hipGetLastError();
}

hipError_t launch_scan(ScanArray a, int32_t n, int32_t *tmp, hipStream_t s)
{
    a.tile_sums = tmp;
    if (n <= kScanTwoPass) return launch_scan_pair(a, a, 1, n, s);
    const int32_t ntiles = (int32_t)((n + kScanTile - 1) / kScanTile);
    k_scan_reduce<<<ntiles, kScanThreads, 0, s>>>(a, a, n);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    e = launch_scan(tmp, tmp, ntiles, tmp + ntiles + 1, nullptr, s);
    if (e != hipSuccess) return e;
    k_scan<kScanItems, kCarryScanned><<<ntiles, kScanThreads, 0, s>>>(a, a, n);
    return hipGetLastError();
}

hipError_t launch_scan(const int32_t *in, int32_t *out, int32_t n, int32_t *tmp,
                       int32_t *total_out, hipStream_t s)
{
    ScanArray a;
    a.in = in;
    a.out = out;
    a.total = total_out;
    return launch_scan(a, n, tmp, s);
}

hipError_t launch_scan2(ScanArray a0, ScanArray a1, int32_t n, int32_t *tmp, hipStream_t s)
{
    if (n <= kScanTwoPass) {
        a0.tile_sums = tmp;
        a1.tile_sums = tmp + (n + kScanTile - 1) / kScanTile;
        return launch_scan_pair(a0, a1, 2, n, s);
    }
    hipError_t e = launch_scan(a0, n, tmp, s);
    return e != hipSuccess ? e : launch_scan(a1, n, tmp, s);
}

hipError_t launch_fill_windows(const int32_t *row_ptr, const int32_t *win_row, int32_t T,
                               const int32_t *tmp_cols, const uint32_t *tmp_mask,
                               const int32_t *u, const int32_t *blk_off, int32_t *cols,
                               uint32_t *mask, hipStream_t s)
{
    if (T == 0) return hipSuccess;
    k_fill_windows<<<T, 256, 0, s>>>(row_ptr, win_row, tmp_cols, tmp_mask, u, blk_off, cols,
                                     mask);
    return hipGetLastError();
}

hipError_t launch_bin_keys(const int32_t *nb, int32_t T, const int32_t *n_blocks,
                           const int32_t *max_blocks, int32_t forced, int32_t slots,
                           bool reorder, int32_t *piece_out, int32_t *npieces,
                           int32_t *key, int32_t *split_pieces, int32_t *split_one,
                           hipStream_t s)
{
    k_bin_keys<<<grid_for(T, 256), 256, 0, s>>>(nb, T, n_blocks, max_blocks, forced, slots,
                                                reorder, piece_out, npieces, key,
                                                split_pieces, split_one);
    return hipGetLastError();
}

hipError_t launch_split_items(const int32_t *merges, const int32_t *split_item,
                              const int32_t *blk_off, int32_t n_split, WorkItem *items,
                              hipStream_t s)
{
    if (n_split == 0) return hipSuccess;
    k_split_items<<<grid_for(n_split, 4), 256, 0, s>>>(merges, split_item, blk_off, n_split,
                                                      items);
    return hipGetLastError();
}

hipError_t launch_validate_plan(const f3s_plan_s &p, int32_t *err, hipStream_t s)
{
    int64_t n = p.n_items;
    if (p.n_blocks > n) n = p.n_blocks;
    if (p.n_split > n) n = p.n_split;
    if (n == 0) return hipSuccess;
    k_validate_plan<<<grid_for(n, 256), 256, 0, s>>>(p.blk_off, p.T, p.cols, p.n_blocks,
                                                    p.items, p.n_items, p.merges,
                                                    p.n_split, p.n_pieces, p.N, err);
    return hipGetLastError();
}


}  // namespace f3s
