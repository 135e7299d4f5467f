// Plan construction on the GPU: CSR -> Binary Sparse Block layout
// (Section 3.1) and the heavy-first work list (Section 3.2).
//
//  1. row_ptr validation
//  2. per row window: sorted distinct columns (LDS bitonic sort; windows too
//     large for LDS use an N-bit column bitmap and popcount compaction)
//  3. blocks per window (ceil(u/16)) and their exclusive prefix (tro)
//  4. padded column lists (sptd) and one 256-bit bitmap per 16x16 block,
//     built in LDS per window
//  5. work list: windows stably sorted by block count, largest first, with
//     windows above `piece` blocks split into pieces of whole block pairs
//
// Every kernel is deterministic: integer atomics only commute (bitwise OR,
// counters whose final value is all that is read), and every position in
// the output is owned by exactly one thread.
#include <limits.h>

#include "f3s_internal.h"

namespace f3s {
namespace {

constexpr int kSortCap = 4096;     // entries a window may have for LDS sort
constexpr int kPlanThreads = 256;

// Exclusive scan of one int per thread over a 256-thread block.
__device__ int block_exclusive_scan256(int v, int *lds, int *total)
{
    const int tid = threadIdx.x;
    lds[tid] = v;
    __syncthreads();
    for (int off = 1; off < kPlanThreads; off <<= 1) {
        int t = tid >= off ? lds[tid - off] : 0;
        __syncthreads();
        lds[tid] += t;
        __syncthreads();
    }
    const int incl = lds[tid];
    *total = lds[kPlanThreads - 1];
    __syncthreads();
    return incl - v;
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

__global__ __launch_bounds__(kPlanThreads) void k_window_sort(
    const int32_t *row_ptr, const int32_t *col_idx, int32_t N, int32_t *tmp_cols,
    int32_t *u, int32_t *heavy, int32_t *n_heavy, int32_t *err)
{
    __shared__ int32_t keys[kSortCap];
    __shared__ int scan[kPlanThreads];
    // k_check_row_ptr ran before on the same stream: a malformed row_ptr
    // stops every block here, before any column is read
    if (*(volatile int32_t *)err) return;
    const int tid = threadIdx.x;
    const int w = blockIdx.x;
    const int r0 = w * kWindowRows;
    const int r1 = min(r0 + kWindowRows, N);
    const int beg = row_ptr[r0];
    const int n = row_ptr[r1] - beg;
    if (n > kSortCap) {
        if (tid == 0) {
            heavy[atomicAdd(n_heavy, 1)] = w;
            u[w] = 0;
        }
        return;
    }
    int p2 = 1;
    while (p2 < n) p2 <<= 1;
    for (int t = tid; t < p2; t += kPlanThreads) {
        int v = INT_MAX;
        if (t < n) {
            v = col_idx[beg + t];
            if (v < 0 || v >= N) {
                atomicOr(err, 1);
                v = INT_MAX;
            }
        }
        keys[t] = v;
    }
    __syncthreads();
    // bitonic sort, ascending
    for (int k = 2; k <= p2; k <<= 1) {
        for (int j = k >> 1; j > 0; j >>= 1) {
            for (int t = tid; t < p2; t += kPlanThreads) {
                const int x = t ^ j;
                if (x > t) {
                    const int a = keys[t], b = keys[x];
                    const bool up = (t & k) == 0;
                    if ((a > b) == up) {
                        keys[t] = b;
                        keys[x] = a;
                    }
                }
            }
            __syncthreads();
        }
    }
    // distinct values, written in order at the window's CSR offset
    const int ch = (p2 + kPlanThreads - 1) / kPlanThreads;
    const int lo = min(tid * ch, n), hi = min(lo + ch, n);
    int cnt = 0;
    for (int k = lo; k < hi; ++k)
        cnt += keys[k] != INT_MAX && (k == 0 || keys[k] != keys[k - 1]);
    int total;
    int off = block_exclusive_scan256(cnt, scan, &total);
    for (int k = lo; k < hi; ++k)
        if (keys[k] != INT_MAX && (k == 0 || keys[k] != keys[k - 1]))
            tmp_cols[beg + off++] = keys[k];
    if (tid == 0) u[w] = total;
}

__global__ __launch_bounds__(kPlanThreads) void k_heavy_compact(
    const int32_t *row_ptr, const int32_t *col_idx, int32_t N,
    const int32_t *heavy, uint32_t *bitmap, int32_t words, int32_t *tmp_cols,
    int32_t *u, int32_t *err)
{
    __shared__ int scan[kPlanThreads];
    const int tid = threadIdx.x;
    const int w = heavy[blockIdx.x];
    uint32_t *bm = bitmap + (int64_t)blockIdx.x * words;
    const int r0 = w * kWindowRows;
    const int r1 = min(r0 + kWindowRows, N);
    const int beg = row_ptr[r0], end = row_ptr[r1];
    for (int e = beg + tid; e < end; e += kPlanThreads) {
        const int c = col_idx[e];
        if (c < 0 || c >= N) {
            atomicOr(err, 1);
            continue;
        }
        atomicOr(&bm[c >> 5], 1u << (c & 31));
    }
    // the atomics and the loads below are issued by this workgroup alone and
    // performed at the L2: workgroup-scope ordering is enough (a device-scope
    // fence would write back the whole L2 for every block)
    __threadfence_block();
    __syncthreads();
    const int ch = (words + kPlanThreads - 1) / kPlanThreads;
    const int lo = min(tid * ch, words), hi = min(lo + ch, words);
    int cnt = 0;
    for (int k = lo; k < hi; ++k)
        cnt += __popc(__hip_atomic_load(&bm[k], __ATOMIC_RELAXED,
                                        __HIP_MEMORY_SCOPE_AGENT));
    int total;
    int off = block_exclusive_scan256(cnt, scan, &total);
    for (int k = lo; k < hi; ++k) {
        uint32_t x = __hip_atomic_load(&bm[k], __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
        while (x) {
            const int b = __ffs(x) - 1;
            tmp_cols[beg + off++] = 32 * k + b;
            x &= x - 1;
        }
    }
    if (tid == 0) u[w] = total;
}

__global__ void k_blocks_per_window(const int32_t *u, int32_t T, int32_t *nb)
{
    const int w = blockIdx.x * blockDim.x + threadIdx.x;
    if (w < T) nb[w] = (u[w] + kBlockCols - 1) / kBlockCols;
}

constexpr int kScanThreads = 1024;
constexpr int kScanItems = 4;
constexpr int kScanTile = kScanThreads * kScanItems;

// Exclusive scan of one tile of kScanTile ints per workgroup, in place or
// not; the tile's total goes to tile_sums[tile] (when given).  With one
// workgroup and n > kScanTile it walks the tiles in order with a carry
// (used for the short array of tile totals), and writes out[n] = total.
__global__ __launch_bounds__(kScanThreads) void k_scan(const int32_t *in, int32_t *out,
                                                       int32_t n, int32_t *tile_sums,
                                                       int32_t *total_out)
{
    __shared__ int32_t sh[kScanThreads];
    const int tid = threadIdx.x;
    const bool whole = gridDim.x == 1;
    int carry = 0;
    const int64_t first = whole ? 0 : (int64_t)blockIdx.x * kScanTile;
    const int64_t last = whole ? n : min((int64_t)n, first + kScanTile);
    for (int64_t base = first; base < last; base += kScanTile) {
        int v[kScanItems];
        int s = 0;
        for (int j = 0; j < kScanItems; ++j) {
            const int64_t idx = base + (int64_t)tid * kScanItems + j;
            v[j] = idx < last ? in[idx] : 0;
            s += v[j];
        }
        sh[tid] = s;
        __syncthreads();
        for (int off = 1; off < kScanThreads; off <<= 1) {
            int t = tid >= off ? sh[tid - off] : 0;
            __syncthreads();
            sh[tid] += t;
            __syncthreads();
        }
        int run = carry + sh[tid] - s;
        const int tile_total = sh[kScanThreads - 1];
        __syncthreads();
        for (int j = 0; j < kScanItems; ++j) {
            const int64_t idx = base + (int64_t)tid * kScanItems + j;
            if (idx < last) out[idx] = run;
            run += v[j];
        }
        carry += tile_total;
    }
    if (tid == 0) {
        if (whole) {
            out[n] = carry;
            if (total_out) *total_out = carry;
        } else {
            tile_sums[blockIdx.x] = carry;
        }
    }
}

// Adds the scanned tile offsets to every tile after the first and writes
// the total.
__global__ __launch_bounds__(256) void k_scan_add(int32_t *out, int32_t n,
                                                  const int32_t *tile_offs, int32_t ntiles,
                                                  int32_t *total_out)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) {
        const int64_t tile = i / kScanTile;
        if (tile > 0) out[i] += tile_offs[tile];
    }
    if (i == 0) {
        out[n] = tile_offs[ntiles];
        if (total_out) *total_out = tile_offs[ntiles];
    }
}

// Column lists (sptd, padded with -1) and block bitmaps of one window per
// workgroup.  The window's sorted distinct columns and its bitmaps are held
// in LDS: each CSR entry finds its row among the 16 row starts and its
// compacted column by binary search, sets its bit with an LDS atomic OR, and
// the block arrays are written out once, coalesced.  The set bits are
// counted on the way out (distinct (row, col) pairs of A).  A window with
// more distinct columns than the LDS holds (from the heavy path) works on
// its own global bitmaps instead, zeroed first.
__global__ __launch_bounds__(kPlanThreads) void k_fill_windows(
    const int32_t *row_ptr, const int32_t *col_idx, int32_t N,
    const int32_t *tmp_cols, const int32_t *u, const int32_t *blk_off,
    int32_t *cols, uint32_t *mask, unsigned long long *nnz_out)
{
    __shared__ int32_t s_uc[kSortCap];
    __shared__ uint32_t s_mask[kSortCap / kBlockCols * kMaskWords];
    __shared__ int32_t s_rp[kWindowRows + 1];
    __shared__ unsigned long long s_cnt;
    const int tid = threadIdx.x;
    const int w = blockIdx.x;
    const int r0 = w * kWindowRows;
    const int nr = min(r0 + kWindowRows, N) - r0;
    if (tid <= nr) s_rp[tid] = row_ptr[r0 + tid];
    if (tid == 0) s_cnt = 0;
    const int32_t *uc = tmp_cols + row_ptr[r0];
    const int uw = u[w];
    const int ob = blk_off[w];
    const int nbw = blk_off[w + 1] - ob;
    const bool in_lds = uw <= kSortCap;
    uint32_t *gmask = mask + (int64_t)kMaskWords * ob;
    for (int k = tid; k < kMaskWords * nbw; k += kPlanThreads) {
        if (in_lds) s_mask[k] = 0;
        else gmask[k] = 0;
    }
    if (in_lds)
        for (int k = tid; k < uw; k += kPlanThreads) s_uc[k] = uc[k];
    __threadfence_block();
    __syncthreads();
    const int beg = s_rp[0], n = s_rp[nr] - beg;
    for (int e = tid; e < n; e += kPlanThreads) {
        // row of entry e: the last row start <= beg + e
        int rlo = 0, rhi = nr;
        while (rhi - rlo > 1) {
            const int mid = (rlo + rhi) >> 1;
            if (s_rp[mid] <= beg + e) rlo = mid;
            else rhi = mid;
        }
        const int c = col_idx[beg + e];
        int lo = 0, hi = uw;
        while (lo < hi) {
            const int mid = (lo + hi) >> 1;
            if ((in_lds ? s_uc[mid] : uc[mid]) < c) lo = mid + 1;
            else hi = mid;
        }
        if (lo >= uw || (in_lds ? s_uc[lo] : uc[lo]) != c) continue;  // unreachable on valid CSR
        const int cc = lo % kBlockCols;
        const int bit = 4 * (rlo + 16 * (cc / 4)) + (cc % 4);
        const int word = kMaskWords * (lo / kBlockCols) + bit / 32;
        if (in_lds) atomicOr(&s_mask[word], 1u << (bit % 32));
        else atomicOr(&gmask[word], 1u << (bit % 32));
    }
    __threadfence_block();  // as in k_heavy_compact: one workgroup, L2 atomics
    __syncthreads();
    for (int k = tid; k < kBlockCols * nbw; k += kPlanThreads)
        cols[(int64_t)kBlockCols * ob + k] = k < uw ? (in_lds ? s_uc[k] : uc[k]) : -1;
    unsigned long long cnt = 0;
    for (int k = tid; k < kMaskWords * nbw; k += kPlanThreads) {
        uint32_t m;
        if (in_lds) {
            m = s_mask[k];
            gmask[k] = m;
        } else {
            m = __hip_atomic_load(&gmask[k], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        cnt += __popc(m);
    }
    if (cnt) atomicAdd(&s_cnt, cnt);
    __syncthreads();
    if (tid == 0 && s_cnt) atomicAdd(nnz_out, s_cnt);
}

__global__ void k_sum_i32(const int32_t *in, int32_t n, unsigned long long *out)
{
    unsigned long long acc = 0;
    for (int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; k < n;
         k += (int64_t)gridDim.x * blockDim.x)
        acc += (unsigned long long)in[k];
    if (acc) atomicAdd(out, acc);
}

__global__ void k_max_i32(const int32_t *in, int32_t n, int32_t *out)
{
    int32_t acc = 0;
    for (int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; k < n;
         k += (int64_t)gridDim.x * blockDim.x)
        acc = max(acc, in[k]);
    atomicMax(out, acc);
}

__global__ void k_bin_keys(const int32_t *nb, int32_t T, int32_t piece, bool reorder,
                           int32_t *npieces, int32_t *key, int32_t *split_pieces,
                           int32_t *split_one)
{
    const int w = blockIdx.x * blockDim.x + threadIdx.x;
    if (w >= T) return;
    const int n = nb[w];
    const bool split = n > piece;
    const int np = split ? (n + piece - 1) / piece : 1;
    npieces[w] = np;
    key[w] = reorder ? (split ? piece : n) : 0;
    split_pieces[w] = split ? np : 0;
    split_one[w] = split ? 1 : 0;
}

// One thread per chunk of windows; hist is [piece + 1][nchunks], row b holds
// the items of key (piece - b), so a flat scan orders keys largest first,
// then chunks, then windows inside a chunk: a stable descending sort.
__global__ void k_bin_hist(const int32_t *npieces, const int32_t *key, int32_t T,
                           int32_t piece, int32_t chunk, int32_t nchunks,
                           int32_t *hist)
{
    const int c = blockIdx.x * blockDim.x + threadIdx.x;
    if (c >= nchunks) return;
    const int w1 = min(T, (c + 1) * chunk);
    for (int w = c * chunk; w < w1; ++w)
        hist[(int64_t)(piece - key[w]) * nchunks + c] += npieces[w];
}

__global__ void k_bin_scatter(const int32_t *nb, const int32_t *blk_off,
                              const int32_t *npieces, const int32_t *key,
                              const int32_t *slot_base, const int32_t *split_idx,
                              int32_t T, int32_t piece, int32_t chunk,
                              int32_t nchunks, int32_t *offs, WorkItem *items,
                              int32_t *merges)
{
    const int c = blockIdx.x * blockDim.x + threadIdx.x;
    if (c >= nchunks) return;
    const int w1 = min(T, (c + 1) * chunk);
    for (int w = c * chunk; w < w1; ++w) {
        int32_t *cell = offs + (int64_t)(piece - key[w]) * nchunks + c;
        const int pos = *cell;
        const int n = nb[w], b0 = blk_off[w], np = npieces[w];
        if (n <= piece) {
            items[pos] = WorkItem{w, b0, b0 + n, -1};
        } else {
            const int64_t pairs = (n + 1) / 2;
            for (int k = 0; k < np; ++k) {
                const int a = (int)((k * pairs) / np);
                const int b = (int)(((k + 1) * pairs) / np);
                items[pos + k] = WorkItem{w, b0 + 2 * a, b0 + min(n, 2 * b),
                                          slot_base[w] + k};
            }
            const int s = split_idx[w];
            merges[3 * s + 0] = w;
            merges[3 * s + 1] = slot_base[w];
            merges[3 * s + 2] = np;
        }
        *cell = pos + np;
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

// Entries of the pattern read back from a plan (every set bitmap bit is a
// distinct (row, col) of A), one workgroup per window.  Without `out`, counts
// the entries of each column; with it, scatters the row of each entry to
// position cursor[col]++ of the transposed CSR (order inside a transposed row
// is arbitrary: a plan built from it sorts its columns anyway).
__global__ __launch_bounds__(256) void k_transpose_entries(const int32_t *blk_off,
                                                           const int32_t *cols,
                                                           const uint32_t *mask,
                                                           int32_t *cursor, int32_t *out)
{
    const int w = blockIdx.x;
    const int64_t w0 = (int64_t)blk_off[w] * kMaskWords, w1 = (int64_t)blk_off[w + 1] * kMaskWords;
    for (int64_t t = w0 + threadIdx.x; t < w1; t += blockDim.x) {
        const int64_t blk = t / kMaskWords;
        const int word = (int)(t % kMaskWords);
        uint32_t x = mask[t];
        while (x) {
            const int k = 32 * word + __ffs(x) - 1;
            x &= x - 1;
            const int r = (k >> 2) & 15;           // window row
            const int c = 4 * (k >> 6) + (k & 3);  // block column
            const int col = cols[kBlockCols * blk + c];
            const int pos = atomicAdd(&cursor[col], 1);
            if (out) out[pos] = w * kWindowRows + r;
        }
    }
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

hipError_t launch_window_sort(const int32_t *row_ptr, const int32_t *col_idx,
                              int32_t N, int32_t T, int32_t *tmp_cols,
                              int32_t *u, int32_t *heavy, int32_t *n_heavy,
                              int32_t *err, hipStream_t s)
{
    if (T == 0) return hipSuccess;
    k_window_sort<<<T, kPlanThreads, 0, s>>>(row_ptr, col_idx, N, tmp_cols, u,
                                             heavy, n_heavy, err);
    return hipGetLastError();
}

hipError_t launch_heavy_compact(const int32_t *row_ptr, const int32_t *col_idx,
                                int32_t N, const int32_t *heavy, int32_t count,
                                uint32_t *bitmap, int32_t words,
                                int32_t *tmp_cols, int32_t *u, int32_t *err,
                                hipStream_t s)
{
    if (count == 0) return hipSuccess;
    k_heavy_compact<<<count, kPlanThreads, 0, s>>>(row_ptr, col_idx, N, heavy,
                                                   bitmap, words, tmp_cols, u, err);
    return hipGetLastError();
}

hipError_t launch_blocks_per_window(const int32_t *u, int32_t T, int32_t *nb,
                                    hipStream_t s)
{
    if (T == 0) return hipSuccess;
    k_blocks_per_window<<<grid_for(T, 256), 256, 0, s>>>(u, T, nb);
    return hipGetLastError();
}

int64_t scan_tmp_ints(int64_t n)
{
    return n <= kScanTile ? 1 : (n + kScanTile - 1) / kScanTile + 1;
}

hipError_t launch_scan(const int32_t *in, int32_t *out, int32_t n, int32_t *tmp,
                       int32_t *total_out, hipStream_t s)
{
    if (n <= kScanTile) {
        k_scan<<<1, kScanThreads, 0, s>>>(in, out, n, nullptr, total_out);
        return hipGetLastError();
    }
    const int32_t ntiles = (int32_t)((n + kScanTile - 1) / kScanTile);
    k_scan<<<ntiles, kScanThreads, 0, s>>>(in, out, n, tmp, nullptr);
    k_scan<<<1, kScanThreads, 0, s>>>(tmp, tmp, ntiles, nullptr, nullptr);
    k_scan_add<<<grid_for(n, 256), 256, 0, s>>>(out, n, tmp, ntiles, total_out);
    return hipGetLastError();
}

hipError_t launch_fill_windows(const int32_t *row_ptr, const int32_t *col_idx,
                               int32_t N, int32_t T, const int32_t *tmp_cols,
                               const int32_t *u, const int32_t *blk_off,
                               int32_t *cols, uint32_t *mask,
                               unsigned long long *nnz_out, hipStream_t s)
{
    if (T == 0) return hipSuccess;
    k_fill_windows<<<T, kPlanThreads, 0, s>>>(row_ptr, col_idx, N, tmp_cols, u,
                                              blk_off, cols, mask, nnz_out);
    return hipGetLastError();
}

hipError_t launch_sum_i32(const int32_t *in, int32_t n, unsigned long long *out,
                          hipStream_t s)
{
    if (n == 0) return hipSuccess;
    const unsigned g = grid_for(n, 256);
    k_sum_i32<<<g < 4096 ? g : 4096, 256, 0, s>>>(in, n, out);
    return hipGetLastError();
}

hipError_t launch_max_i32(const int32_t *in, int32_t n, int32_t *out,
                          hipStream_t s)
{
    if (n == 0) return hipSuccess;
    const unsigned g = grid_for(n, 256);
    k_max_i32<<<g < 4096 ? g : 4096, 256, 0, s>>>(in, n, out);
    return hipGetLastError();
}

hipError_t launch_bin_keys(const int32_t *nb, int32_t T, int32_t piece, bool reorder,
                           int32_t *npieces, int32_t *key, int32_t *split_pieces,
                           int32_t *split_one, hipStream_t s)
{
    if (T == 0) return hipSuccess;
    k_bin_keys<<<grid_for(T, 256), 256, 0, s>>>(nb, T, piece, reorder, npieces, key,
                                               split_pieces, split_one);
    return hipGetLastError();
}

hipError_t launch_bin_hist(const int32_t *npieces, const int32_t *key, int32_t T,
                           int32_t piece, int32_t chunk, int32_t nchunks,
                           int32_t *hist, hipStream_t s)
{
    if (nchunks == 0) return hipSuccess;
    k_bin_hist<<<grid_for(nchunks, 64), 64, 0, s>>>(npieces, key, T, piece, chunk,
                                                   nchunks, hist);
    return hipGetLastError();
}

hipError_t launch_bin_scatter(const int32_t *nb, const int32_t *blk_off,
                              const int32_t *npieces, const int32_t *key,
                              const int32_t *slot_base, const int32_t *split_idx,
                              int32_t T, int32_t piece, int32_t chunk,
                              int32_t nchunks, int32_t *offs, WorkItem *items,
                              int32_t *merges, hipStream_t s)
{
    if (nchunks == 0) return hipSuccess;
    k_bin_scatter<<<grid_for(nchunks, 64), 64, 0, s>>>(
        nb, blk_off, npieces, key, slot_base, split_idx, T, piece, chunk, nchunks,
        offs, items, merges);
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

hipError_t launch_transpose_entries(const f3s_plan_s &p, int32_t *cursor, int32_t *out,
                                   hipStream_t s)
{
    if (p.T == 0) return hipSuccess;
    k_transpose_entries<<<p.T, 256, 0, s>>>(p.blk_off, p.cols, p.mask, cursor, out);
    return hipGetLastError();
}

}  // namespace f3s
