// CSR of the transposed pattern A^T from a plan of A, on the GPU, without
// atomics: the plan's block bitmaps are decoded into (column, row) pairs,
// the pairs are radix-sorted by column (radix.hip, stable), and the row
// pointers of A^T follow from the sorted columns by binary search.  A^T's
// rows come out in increasing column order (the sort is stable and the
// pairs are decoded window by window, row-ascending within a column), so
// comparing every row of A, read from the plan in the same order, with the
// same row of A^T decides exactly whether A^T = A.  The pattern a plan holds
// is A with duplicates merged (Section 3.1's bitmaps), so A^T has one entry
// per set bit.
#include "f3s_internal.h"

namespace f3s {
namespace {

__device__ __forceinline__ int wave_excl_scan_t(int v, int lane, int *total)
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

// Set bits of each window's bitmaps; one wavefront per window.
__global__ __launch_bounds__(256) void k_window_bits(const int32_t *blk_off,
                                                     const uint32_t *mask, int32_t T,
                                                     int32_t *cnt)
{
    const int lane = threadIdx.x & 63;
    const int w = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (w >= T) return;
    const int64_t k0 = (int64_t)kMaskWords * blk_off[w];
    const int64_t k1 = (int64_t)kMaskWords * blk_off[w + 1];
    int c = 0;
    for (int64_t k = k0 + lane; k < k1; k += 64) c += __popc(mask[k]);
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) c += __shfl_xor(c, o);
    if (lane == 0) cnt[w] = c;
}

// (column, row) of every set bit of window w, written from off[w] on in bit
// order; one wavefront per window.
__global__ __launch_bounds__(256) void k_window_pairs(const int32_t *blk_off,
                                                      const int32_t *cols,
                                                      const uint32_t *mask,
                                                      const int32_t *win_row, int32_t T,
                                                      const int32_t *off, int32_t *keys,
                                                      int32_t *rows)
{
    const int lane = threadIdx.x & 63;
    const int w = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (w >= T) return;
    // first row of the window (16-row windows, or those of a plan aligned to
    // the graphs of a batch)
    const int r0 = win_row ? win_row[w] : w * kWindowRows;
    const int64_t k0 = (int64_t)kMaskWords * blk_off[w];
    const int64_t k1 = (int64_t)kMaskWords * blk_off[w + 1];
    int64_t base = off[w];
    for (int64_t kb = k0; kb < k1; kb += 64) {
        const int64_t k = kb + lane;
        uint32_t m = k < k1 ? mask[k] : 0u;
        int total;
        int64_t pos = base + wave_excl_scan_t(__popc(m), lane, &total);
        const int64_t blk = k / kMaskWords;
        const int word = (int)(k % kMaskWords);
        while (m) {
            const int bit = 32 * word + __ffs(m) - 1;
            m &= m - 1;
            const int r = (bit >> 2) & 15;             // window row
            const int c = 4 * (bit >> 6) + (bit & 3);  // block column
            keys[pos] = cols[kBlockCols * blk + c];
            rows[pos] = r0 + r;
            ++pos;
        }
        base += total;
    }
}

// rp[c] = number of sorted keys below c, for c = 0 .. N.
__global__ void k_rows_from_sorted(const int32_t *keys, int32_t n, int32_t N, int32_t *rp)
{
    const int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (c > N) return;
    int lo = 0, hi = n;
    while (lo < hi) {
        const int mid = (int)(((int64_t)lo + hi) >> 1);
        if ((int64_t)keys[mid] < c) lo = mid + 1;
        else hi = mid;
    }
    rp[c] = lo;
}

// win[b] = the window of block b; one wavefront per window.
__global__ __launch_bounds__(256) void k_block_window(const int32_t *blk_off, int32_t T,
                                                      int32_t *win)
{
    const int w = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (w >= T) return;
    for (int b = blk_off[w] + (threadIdx.x & 63); b < blk_off[w + 1]; b += 64) win[b] = w;
}

// Position of column c among the distinct columns of window v (cols padded
// with -1 after the last one), or -1.
__device__ int find_col(const int32_t *blk_off, const int32_t *cols, int v, int c)
{
    const int32_t *list = cols + (int64_t)kBlockCols * blk_off[v];
    int lo = 0, hi = kBlockCols * (blk_off[v + 1] - blk_off[v]);
    while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        const int x = list[mid];
        if (x >= 0 && x < c) lo = mid + 1;
        else hi = mid;
    }
    return lo < kBlockCols * (blk_off[v + 1] - blk_off[v]) && list[lo] == c ? lo : -1;
}

// Sets *asym when some entry (r, c) of the plan's pattern has no entry (c, r),
// straight from the plan (no transposed CSR needed): for every set bit, the
// row r is looked up among the distinct columns of row c's window and the
// bit of (c, r) tested.  One thread per bitmap word over
// all blocks (a hub window's entries spread over many waves); stops early
// once an asymmetry is known.
__global__ __launch_bounds__(256) void k_check_symmetric(const int32_t *blk_off,
                                                         const int32_t *cols,
                                                         const uint32_t *mask,
                                                         const int32_t *win, int64_t words,
                                                         int32_t *asym)
{
    const int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (k >= words || *(volatile int32_t *)asym) return;
    uint32_t m = mask[k];
    if (!m) return;
    const int64_t blk = k / kMaskWords;
    const int word = (int)(k % kMaskWords);
    const int w = win[blk];
    while (m) {
        const int bit = 32 * word + __ffs(m) - 1;
        m &= m - 1;
        const int r = w * kWindowRows + ((bit >> 2) & 15);
        const int c = cols[kBlockCols * blk + 4 * (bit >> 6) + (bit & 3)];
        const int v = c / kWindowRows;
        const int a = find_col(blk_off, cols, v, r);
        bool bad = a < 0;
        if (!bad) {
            const int cc = a % kBlockCols;
            const int b2 = 4 * (c % kWindowRows + 16 * (cc / 4)) + (cc % 4);
            const int64_t blk2 = blk_off[v] + a / kBlockCols;
            bad = ((mask[kMaskWords * blk2 + b2 / 32] >> (b2 % 32)) & 1u) == 0;
        }
        if (bad) {
            atomicOr(asym, 1);
            return;
        }
    }
}


// Row r's 16 bits (block columns 0..15) of one block's bitmap words: the
// four bits of block columns 4q .. 4q+3 are bits 4 (r % 8) .. +3 of word
// 2q + r / 8.
__device__ __forceinline__ uint32_t row_bits(const uint32_t (&mw)[kMaskWords], int r)
{
    uint32_t m = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) m |= ((mw[2 * q + (r >> 3)] >> (4 * (r & 7))) & 15u) << (4 * q);
    return m;
}

// Inclusive sum over the 64 lanes with DPP row shifts (within rows of 16
// lanes, out-of-row sources read 0) and the three row totals by readlane.
__device__ __forceinline__ int wave_sum_dpp(int x, int lane)
{
    x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xF, 0xF, true);  // row_shr:1
    x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xF, 0xF, true);  // row_shr:2
    x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xF, 0xF, true);  // row_shr:4
    x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xF, 0xF, true);  // row_shr:8
    const int r0 = __builtin_amdgcn_readlane(x, 15), r1 = __builtin_amdgcn_readlane(x, 31);
    const int r2 = __builtin_amdgcn_readlane(x, 47);
    const int row = lane >> 4;
    return x + (row >= 1 ? r0 : 0) + (row >= 2 ? r1 : 0) + (row >= 3 ? r2 : 0);
}

// The symmetry decision on A^T's CSR (rpt, cit; rows in increasing column
// order), in two passes.  Row r of A, read from the plan, is in increasing
// column order too: blocks in order, and within a block the compacted
// columns, which are sorted.  So the k-th entry of row r in A must be entry
// k of row r in A^T, and the row lengths must agree.  (A walk of each row by
// one thread, without the prefix array, measured 2.5x slower: a chain of
// dependent loads per row.)
//
// Pass 1, one wavefront per window, 64 blocks per step (lane = block): for
// each of the 16 rows, a wave prefix of the row's entry counts per block
// gives pre[16 b + r] = entries of row r in the window's blocks before b;
// the row totals are checked against A^T's row lengths.
__global__ __launch_bounds__(256) void k_row_prefix(const int32_t *blk_off,
                                                    const uint32_t *mask, int32_t T, int32_t N,
                                                    const int32_t *rpt, int32_t *pre,
                                                    int32_t *asym)
{
    const int lane = threadIdx.x & 63;
    const int w = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (w >= T) return;
    // a known asymmetry ends the wave early: one lane's read decides for all
    // (the lane moves below need the whole wave)
    if (__builtin_amdgcn_readfirstlane(*(volatile int32_t *)asym)) return;
    const int b0 = blk_off[w], b1 = blk_off[w + 1];
    int base[kWindowRows];  // wave-uniform: entries of each row so far
#pragma unroll
    for (int r = 0; r < kWindowRows; ++r) base[r] = 0;
    for (int bg = b0; bg < b1; bg += 64) {  // wave-uniform trip count
        const int b = bg + lane;
        uint32_t mw[kMaskWords];
#pragma unroll
        for (int k = 0; k < kMaskWords; ++k)
            mw[k] = b < b1 ? mask[(int64_t)kMaskWords * b + k] : 0u;
#pragma unroll
        for (int r = 0; r < kWindowRows; ++r) {
            const int cnt = __popc(row_bits(mw, r));
            const int incl = wave_sum_dpp(cnt, lane);
            if (b < b1) pre[(int64_t)kWindowRows * b + r] = base[r] + incl - cnt;
            base[r] += __builtin_amdgcn_readlane(incl, 63);
        }
    }
    const int row = w * kWindowRows + lane;
    bool bad = false;
#pragma unroll
    for (int r = 0; r < kWindowRows; ++r)
        if (lane == r) bad = row < N ? rpt[row + 1] - rpt[row] != base[r] : base[r] != 0;
    if (bad) atomicOr(asym, 1);
}

// Pass 2, one thread per (block, row): entry k of row r in block b (the
// block's set bits of row r, in column order) must be entry pre + k of A^T's
// row; all loads of a thread are issued before its comparisons.
__global__ __launch_bounds__(256) void k_compare_blocks(const int32_t *cols,
                                                        const uint32_t *mask,
                                                        const int32_t *win, int64_t n_blocks,
                                                        int32_t N, const int32_t *rpt,
                                                        const int32_t *cit, const int32_t *pre,
                                                        int32_t *asym)
{
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= kWindowRows * n_blocks || *(volatile int32_t *)asym) return;
    const int64_t b = t / kWindowRows;
    const int r = (int)(t % kWindowRows);
    const uint32_t *mwp = mask + kMaskWords * b + (r >> 3);
    uint32_t m = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) m |= ((mwp[2 * q] >> (4 * (r & 7))) & 15u) << (4 * q);
    if (!m) return;
    const int row = win[b] * kWindowRows + r;
    if (row >= N) {  // rows past N have no entries in a valid plan
        atomicOr(asym, 1);
        return;
    }
    const int start = rpt[row], len = rpt[row + 1] - start, k0 = pre[t];
    typedef int32_t i4 __attribute__((ext_vector_type(4)));
    const i4 *cp = reinterpret_cast<const i4 *>(cols + kBlockCols * b);
    int32_t c[kBlockCols];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const i4 v = cp[q];
        c[4 * q + 0] = v[0];
        c[4 * q + 1] = v[1];
        c[4 * q + 2] = v[2];
        c[4 * q + 3] = v[3];
    }
    int32_t got[kBlockCols];
#pragma unroll
    for (int s = 0; s < kBlockCols; ++s) {
        const int k = k0 + __popc(m & ((1u << s) - 1u));
        got[s] = ((m >> s) & 1u) && k < len ? cit[start + k] : -1;
    }
    bool bad = false;
#pragma unroll
    for (int s = 0; s < kBlockCols; ++s) bad |= ((m >> s) & 1u) && got[s] != c[s];
    if (bad) atomicOr(asym, 1);
}

}  // namespace

hipError_t launch_check_symmetric(const f3s_plan_s &p, int32_t *win, int32_t *asym,
                                  hipStream_t s)
{
    if (p.T == 0 || p.n_blocks == 0) return hipSuccess;
    k_block_window<<<(p.T + 3) / 4, 256, 0, s>>>(p.blk_off, p.T, win);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int64_t words = (int64_t)kMaskWords * p.n_blocks;
    k_check_symmetric<<<(unsigned)((words + 255) / 256), 256, 0, s>>>(p.blk_off, p.cols,
                                                                      p.mask, win, words,
                                                                      asym);
    return hipGetLastError();
}

hipError_t launch_compare_rows(const f3s_plan_s &p, const int32_t *rpt, const int32_t *cit,
                               int32_t *win, int32_t *pre, int32_t *asym, hipStream_t s)
{
    if (p.T == 0) return hipSuccess;
    k_row_prefix<<<(p.T + 3) / 4, 256, 0, s>>>(p.blk_off, p.mask, p.T, p.N, rpt, pre, asym);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || p.n_blocks == 0) return e;
    k_block_window<<<(p.T + 3) / 4, 256, 0, s>>>(p.blk_off, p.T, win);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    const int64_t threads = (int64_t)kWindowRows * p.n_blocks;
    k_compare_blocks<<<(unsigned)((threads + 255) / 256), 256, 0, s>>>(p.cols, p.mask, win,
                                                                       p.n_blocks, p.N, rpt,
                                                                       cit, pre, asym);
    return hipGetLastError();
}

// Scratch of launch_transpose_csr: the decoded pairs (which serve as the
// radix sort's second buffer pair), the first buffer pair, per-window counts
// and offsets, digit counts and the scans' workspace.
size_t transpose_scratch_bytes(const f3s_plan_s &p)
{
    const int64_t n = p.nnz > 0 ? p.nnz : 1;
    const int64_t rc = radix_count_ints((int32_t)n);
    int64_t scan = p.T > n ? p.T : n;
    if (rc > scan) scan = rc;
    auto r = [](int64_t ints) { return (size_t)((4 * ints + 255) & ~255ll); };
    return 4 * r(n) + 2 * r((int64_t)p.T + 1) + r(rc) + r(scan_tmp_ints(scan));
}

hipError_t launch_transpose_csr(const f3s_plan_s &p, void *scratch, size_t scratch_bytes,
                                int32_t *rp, int32_t *ci, hipStream_t s)
{
    const int32_t n = (int32_t)p.nnz;
    const int32_t T = p.T;
    const int64_t nn = n > 0 ? n : 1;
    const int64_t rc = radix_count_ints((int32_t)nn);
    int64_t scan = T > nn ? T : nn;
    if (rc > scan) scan = rc;
    char *at = static_cast<char *>(scratch);
    auto take = [&](int64_t ints) {
        int32_t *q = reinterpret_cast<int32_t *>(at);
        at += (4 * ints + 255) & ~255ll;
        return q;
    };
    RadixScratch rs;
    int32_t *keys_in = take(nn), *rows_in = take(nn);
    rs.keys_a = take(nn);
    rs.vals_a = take(nn);
    rs.keys_b = keys_in;  // free once the first pass has read them
    rs.vals_b = rows_in;
    // the last pass writes the rows straight into ci: passes alternate
    // between the buffer pairs a and b, starting with a
    if (n > 0) (radix_passes(p.N - 1) % 2 ? rs.vals_a : rs.vals_b) = ci;
    int32_t *cnt = take((int64_t)T + 1), *off = take((int64_t)T + 1);
    rs.counts = take(rc);
    rs.scan_tmp = take(scan_tmp_ints(scan));
    if ((size_t)(at - static_cast<char *>(scratch)) > scratch_bytes) return hipErrorInvalidValue;
    hipError_t e;
    if (T > 0) {
        k_window_bits<<<(T + 3) / 4, 256, 0, s>>>(p.blk_off, p.mask, T, cnt);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        e = launch_scan(cnt, off, T, rs.scan_tmp, nullptr, s);
        if (e != hipSuccess) return e;
        k_window_pairs<<<(T + 3) / 4, 256, 0, s>>>(p.blk_off, p.cols, p.mask, p.win_row, T,
                                                   off, keys_in, rows_in);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    const int32_t *sorted_cols = keys_in, *sorted_rows = rows_in;
    if (n > 0) {
        e = launch_radix_pairs(keys_in, rows_in, n, p.N - 1, false, rs, &sorted_cols,
                               &sorted_rows, s);
        if (e != hipSuccess) return e;
        if (sorted_rows != ci) return hipErrorUnknown;  // the pass count above is wrong
    }
    k_rows_from_sorted<<<(unsigned)(((int64_t)p.N + 1 + 255) / 256), 256, 0, s>>>(
        sorted_cols, n, p.N, rp);
    return hipGetLastError();
}

}  // namespace f3s
