// Internal declarations shared by the f3s HIP sources (not installed).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stdlib.h>

#include "f3s.h"

namespace f3s {

constexpr int kWindowRows = 16;   // r: rows per row window (Section 3.1)
constexpr int kBlockCols = 16;    // c: compacted columns per block
constexpr int kMaskWords = 8;     // 256-bit bitmap per 16x16 block
constexpr int kMaxD = 256;        // largest supported feature dimension

// Storage type of Q, K, V in the forward kernels.
constexpr int kInF16 = 0;
constexpr int kInBF16 = 1;
constexpr int kInFP8 = 2;     // OCP e4m3 (finite values up to 448)

// One unit of work for the fused kernel: a whole row window or one piece of
// a split window.  Blocks are absolute indices into the plan's block arrays.
struct WorkItem {
    int32_t window;
    int32_t blk_begin;
    int32_t blk_end;
    int32_t slot;  // partial-result slot of a piece, -1 for a whole window
};
static_assert(sizeof(WorkItem) == 16, "WorkItem must be 16 bytes");

}  // namespace f3s

struct f3s_plan_s {
    int device = 0;
    int32_t N = 0;
    int32_t T = 0;               // row windows
    int64_t nnz_csr = 0;
    int64_t nnz = 0;             // distinct (row, col) pairs
    int64_t n_unique = 0;
    int64_t n_blocks = 0;
    int32_t max_blocks = 0;
    int32_t piece = 0;
    int32_t n_items = 0;
    int32_t n_split = 0;
    int32_t n_pieces = 0;
    int32_t flags = 0;           // bit 0: work list in window order; bit 1: narrow gathers;
                                 // bit 2: windows aligned to the graphs of a batch;
                                 // bit 3: split-row forward (ablation)
    uint64_t id = 0;             // process-unique plan id
    uint64_t transpose_of = 0;   // id of the plan this one transposes (0: none)
    void *store = nullptr;       // one allocation: blk_off, cols, mask, items, merges
    void *part_store = nullptr;  // one allocation: part_o, part_ml
    int64_t part_bytes = 0;
    int32_t *blk_off = nullptr;  // [T + 1]
    int32_t *cols = nullptr;     // [16 * n_blocks]
    uint32_t *mask = nullptr;    // [8 * n_blocks]
    f3s::WorkItem *items = nullptr;  // [n_items]
    int32_t *merges = nullptr;   // [3 * n_split]
    int32_t *win_row = nullptr;  // [T + 1] first row of each window, then N (plans whose
                                 // windows follow the graphs of a batch; null: window w
                                 // is rows 16 w .. 16 w + 15)
    // Partial results of split windows for one launch group of nh heads
    // (nh * d <= kMaxD): slot (piece, head) = piece * nh + head.
    float *part_o = nullptr;     // [n_pieces * 16 * part_row]
    int32_t part_row = f3s::kMaxD;  // floats per piece row of part_o (transposed plans:
                                 // 2 * kMaxD, for the dK and dV partials)
    float *part_ml = nullptr;    // [n_pieces * (kMaxD/32) * 32]: 16 maxima, 16 sums
    int64_t device_bytes = 0;
    int64_t bsb_bytes = 0;
    double build_ms = 0.0;
};

namespace f3s {

// ---- plan kernels (plan_kernels.hip) ------------------------------------
// Workgroup order flags of the fused kernels: heads outermost (one pass over
// the work list per head), and consecutive ranges of the order per XCD.
constexpr uint32_t kOrderHead = 1u;
constexpr uint32_t kOrderXcd = 2u;
// Plans whose windows are nearly uniform: at least 2048 windows, the largest
// holding at most twice the mean block count.  Their work list keeps window
// order (heavy-first sorting has nothing to balance), and launches of 1, 2,
// 4 or 8 heads give each XCD a consecutive range of it.
inline bool uniform_windows(int64_t windows, int64_t blocks, int64_t max_blocks)
{
    return windows >= 2048 && max_blocks * windows <= 2 * blocks;
}
// Whether a launch of nh > 1 heads over plan p, whose K and V (all heads)
// hold kv_bytes, runs head by head instead of window-major (item * nh +
// head).  Window-major order shares a window's column lists and bitmaps
// among its heads, and with nh = 2, 4 or 8 round-robin dispatch still leaves
// each XCD one head (b mod 8 fixes b mod nh).  Head by head wins
// - when K and V exceed the 256 MB Infinity Cache: each head's gathers then
//   stream like a single head's;
// - when nh does not divide 8: window-major order then gives every XCD the
//   rows of every head (hub-heavy Chung-Lu graph, 3 heads: 97.1 -> 88.7 us
//   forward, 245.7 -> 226.7 us backward);
// - on nearly uniform plans, whose XCD ranges then hold one head's rows at a
//   time (3, 4 and 8 heads: 5-28% faster on the molecule batch and the
//   sequence workload; equal with 2).
// Window-major stays for skewed plans with 2, 4 or 8 heads (hub-heavy graph,
// 4 heads: 108.6 against 113.8 us head by head).  F3S_HEAD_MAJOR_BYTES=
// <bytes>, when set, replaces all three tests with kv_bytes > bytes (read at
// launch).
inline bool head_major_order(const f3s_plan_s &p, int32_t nh, uint64_t kv_bytes)
{
    if (nh <= 1) return false;
    const char *e = getenv("F3S_HEAD_MAJOR_BYTES");
    if (e && *e) return kv_bytes > (uint64_t)strtoull(e, nullptr, 10);
    return kv_bytes > ((uint64_t)256 << 20) || 8 % nh != 0 ||
           uniform_windows(p.n_items, p.n_blocks, p.max_blocks);
}
// Whether a launch of `heads` heads over plan p gives each XCD consecutive
// ranges of the work list (see workgroup_position): for nearly uniform plans
// (no XCD's range is then much heavier than another's), window-major with
// 1, 2, 4 or 8 heads, head-major with any.  With its window-order work list
// the molecule batch ran 18.8 -> 15.6 us forward and 52.8 -> 45.0 us
// backward with one head, 33.7 -> 26.4 us forward with two.  On skewed plans
// the ranges would give the heaviest items to one XCD (1.7x slower on the
// million-node graph).  Window-major ranges over all heads of a window would
// give every XCD the rows of every head, where round-robin order with 2, 4
// or 8 heads leaves each XCD one head (b mod 8 fixes b mod heads): that
// measured 45% slower with four heads of the sequence workload, so other
// head counts keep round-robin there.  F3S_XCD_CHUNKS=0 or 1 forces the
// choice where the ranges apply (read at launch).
inline bool xcd_chunks(const f3s_plan_s &p, int32_t heads, bool head_major = false)
{
    if (heads < 1 || (!head_major && 8 % heads != 0)) return false;
    const char *e = getenv("F3S_XCD_CHUNKS");
    if (e && *e) return atoi(e) != 0;
    return uniform_windows(p.n_items, p.n_blocks, p.max_blocks);
}
// Waves sharing one work item (forward and backward): 4 when a launch would
// have fewer waves than the GPU has SIMDs (items x heads < 1024) and the
// items average at least 4 blocks; else 2 when twice the waves still fit
// the GPU at once (`resident`: the kernel's waves per SIMD x 1024 SIMDs) and
// the items average at least 8 blocks (two pairs per wave); else 1.  More
// waves than fit at once would run as a second round, whose tail and the
// extra per-wave Q loads and combination cost more than the parallelism
// gains (4 waves measured 18% slower on the 2048-window sequence workload).
// F3S_WAVES_PER_ITEM=1, 2 or 4 forces it (read at launch).
inline int waves_per_item(int64_t n_blocks, int64_t n_items, int32_t heads, int64_t resident)
{
    const char *e = getenv("F3S_WAVES_PER_ITEM");
    if (e && *e) {
        const int v = atoi(e);
        return v == 4 ? 4 : v == 2 ? 2 : 1;
    }
    if (n_items <= 0) return 1;
    const int64_t waves = n_items * heads;
    if (waves < 1024 && n_blocks >= 4 * n_items) return 4;
    if (2 * waves <= resident && n_blocks >= 8 * n_items) return 2;
    return 1;
}
// First row and row count of window w: rows 16 w .. 16 w + 15 (the last
// window clipped at N), or those given by win_row (device code).
__device__ __forceinline__ void window_rows(const int32_t *win_row, int32_t N, int32_t w,
                                           int32_t *r0, int32_t *nr)
{
    if (win_row) {
        *r0 = win_row[w];
        *nr = win_row[w + 1] - *r0;
    } else {
        *r0 = w * kWindowRows;
        *nr = min(kWindowRows, N - *r0);
    }
}
// Inclusive sum over the lanes of a wavefront (device code).
__device__ __forceinline__ int wave_inclusive_sum(int x, int lane)
{
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const int t = __shfl_up(x, off, 64);
        if (lane >= off) x += t;
    }
    return x;
}

hipError_t launch_check_row_ptr(const int32_t *row_ptr, int32_t N, int32_t nnz,
                                int32_t *err, hipStream_t s);
// Staging area of the window bitmaps, in 32-bit words, for nnz CSR entries.
int64_t mask_stage_words(int64_t nnz, int32_t T);
// Per window of at most 512 entries (one wavefront each): sorted distinct
// columns into tmp_cols at the window's CSR offset, their count into u, the
// block bitmaps into the staging area, their set bits into bits.  Larger
// windows get is_big = 1 (up to 4096 entries) or is_heavy = 1.
// win_row: the windows' first rows (null: 16-row windows); also below.
hipError_t launch_window_wave(const int32_t *row_ptr, const int32_t *col_idx, int32_t N,
                              const int32_t *win_row, int32_t T, int32_t *tmp_cols,
                              uint32_t *tmp_mask, int32_t *u, int32_t *is_big,
                              int32_t *is_heavy, int32_t *bits, int32_t *err, hipStream_t s);
// The windows big[0 .. n_big): sorted distinct columns, u, bitmaps and bits
// as above (one wavefront with 16 keys per lane up to 1024 entries, else an
// LDS sort).
hipError_t launch_window_sort(const int32_t *row_ptr, const int32_t *col_idx,
                              int32_t N, const int32_t *win_row, const int32_t *big,
                              int32_t n_big, int32_t *tmp_cols, uint32_t *tmp_mask,
                              int32_t *u, int32_t *bits, int32_t *err, hipStream_t s);
// Heavy windows (more than 4096 entries): columns, u, bitmaps and bits as
// above, one workgroup per window (column bitmap in LDS, walked in chunks).
hipError_t launch_heavy_lds(const int32_t *row_ptr, const int32_t *col_idx, int32_t N,
                            const int32_t *win_row, const int32_t *heavy, int32_t n_heavy,
                            int32_t *tmp_cols, uint32_t *tmp_mask, int32_t *u,
                            int32_t *bits, int32_t *err, hipStream_t s);
// nb[w] = ceil(u[w] / 16) and the sums of u, bits and nb and the largest nb
// (added / max-ed into the four outputs, zeroed by the caller).
hipError_t launch_window_stats(const int32_t *u, const int32_t *bits, int32_t T,
                               int32_t *nb, unsigned long long *sum_u,
                               unsigned long long *sum_bits, int32_t *sum_nb,
                               int32_t *max_nb, hipStream_t s);
// Exclusive scan of n int32 into out[0..n], out[n] = total (in == out ok).
// Element i is in[i], or in[gather[i]] when gather is given.  With list
// given, every nonzero element i is also listed: list[out[i]] = i (flag
// compaction).  total (may be null) also receives the total.
struct ScanArray {
    const int32_t *in = nullptr;
    const int32_t *gather = nullptr;
    int32_t *out = nullptr;
    int32_t *total = nullptr;
    int32_t *list = nullptr;
    int32_t *tile_sums = nullptr;  // set by the launcher (from tmp)
};
// tmp: scan_tmp_ints(n) ints of workspace.
int64_t scan_tmp_ints(int64_t n);
hipError_t launch_scan(ScanArray a, int32_t n, int32_t *tmp, hipStream_t s);
hipError_t launch_scan(const int32_t *in, int32_t *out, int32_t n, int32_t *tmp,
                       int32_t *total_out, hipStream_t s);
// Two independent scans of n ints each (one launch when n is small).
hipError_t launch_scan2(ScanArray a0, ScanArray a1, int32_t n, int32_t *tmp, hipStream_t s);
// Padded column lists and block bitmaps of the plan from the staging areas.
hipError_t launch_fill_windows(const int32_t *row_ptr, const int32_t *win_row, int32_t T,
                               const int32_t *tmp_cols, const uint32_t *tmp_mask,
                               const int32_t *u, const int32_t *blk_off, int32_t *cols,
                               uint32_t *mask, hipStream_t s);
// Work list: the piece size (from the block count and largest window on the
// device, see plan_piece; forced >= 2 overrides it; slots = 8 per CU) into
// *piece_out, then per window piece count, bucket key, split flags.
// reorder == false gives every window the same key (window order kept).
hipError_t launch_bin_keys(const int32_t *nb, int32_t T, const int32_t *n_blocks,
                           const int32_t *max_blocks, int32_t forced, int32_t slots,
                           bool reorder, int32_t *piece_out, int32_t *npieces,
                           int32_t *key, int32_t *split_pieces, int32_t *split_one,
                           hipStream_t s);
// Pieces of the split windows: items[split_item[s] + k] for piece k of
// split window s (merges[3s..3s+2] = window, first slot, pieces).
hipError_t launch_split_items(const int32_t *merges, const int32_t *split_item,
                              const int32_t *blk_off, int32_t n_split, WorkItem *items,
                              hipStream_t s);

// ---- radix sort (radix.hip) -------------------------------------------------
// Stable sort of n (key, value) int32 pairs, keys in [0, max_key], ascending
// or descending; vals == nullptr stands for the values 0 .. n-1 (the sort
// then yields the sorting permutation).  The inputs are not written; the
// results end up in one of the two scratch pairs (*keys_out, *vals_out say
// which).
struct RadixScratch {
    int32_t *keys_a, *vals_a, *keys_b, *vals_b;  // [n] each
    int32_t *counts;                              // radix_count_ints(n)
    int32_t *scan_tmp;                            // scan_tmp_ints(max(n, radix_count_ints(n)))
};
int64_t radix_count_ints(int32_t n);
// Digit passes of a sort with keys up to max_key (the results of an odd
// count end up in keys_a / vals_a, of an even count in keys_b / vals_b).
int radix_passes(int32_t max_key);
hipError_t launch_radix_pairs(const int32_t *keys, const int32_t *vals, int32_t n,
                              int32_t max_key, bool descending, const RadixScratch &rs,
                              const int32_t **keys_out, const int32_t **vals_out,
                              hipStream_t s);

// ---- work list (worklist.hip) ----------------------------------------------
struct WorkListScratch {
    int32_t *pos;        // [T + 1] first item of each window in sorted order
    RadixScratch radix;  // for n = T
};
// Heavy-first work list from the keys of launch_bin_keys: whole windows as
// items, split windows as merge records plus split_item (their pieces:
// launch_split_items); the item count goes to *n_items_out.  window_order:
// the list keeps window order (what the stable sort gives when every key
// is equal), so key is not read and no sort is launched.
hipError_t launch_worklist(const int32_t *key, const int32_t *nb, const int32_t *blk_off,
                           const int32_t *npieces, const int32_t *slot_base,
                           const int32_t *split_idx, int32_t T, int32_t piece,
                           bool window_order, const WorkListScratch &ws, WorkItem *items,
                           int32_t *merges, int32_t *split_item, int32_t *n_items_out,
                           hipStream_t s);

// ---- transposed pattern (transpose.hip) ----------------------------------
// CSR of A^T (rp[N+1], ci[nnz], each row in increasing column order) from a
// plan's bitmaps; scratch of transpose_scratch_bytes(p) bytes.
size_t transpose_scratch_bytes(const f3s_plan_s &p);
hipError_t launch_transpose_csr(const f3s_plan_s &p, void *scratch, size_t scratch_bytes,
                                int32_t *rp, int32_t *ci, hipStream_t s);
// Sets *asym (zeroed by the caller) unless the plan's pattern is symmetric,
// from the plan alone (binary searches in the windows' column lists; cheap
// on small patterns); win: scratch of n_blocks ints.
hipError_t launch_check_symmetric(const f3s_plan_s &p, int32_t *win, int32_t *asym,
                                  hipStream_t s);
// The same decision given the CSR of A^T (every row of A compared with the
// same row of A^T, position by position; cheaper on large patterns once A^T
// is sorted anyway).  win: n_blocks ints, pre: 16 * n_blocks ints of scratch.
hipError_t launch_compare_rows(const f3s_plan_s &p, const int32_t *rpt, const int32_t *cit,
                               int32_t *win, int32_t *pre, int32_t *asym, hipStream_t s);

// Sets *err when a finished plan is internally inconsistent.
hipError_t launch_validate_plan(const f3s_plan_s &p, int32_t *err, hipStream_t s);

// ---- fused operator (fused3s.hip) ---------------------------------------
// H heads of size d; Q, K, V, O rows hold the heads back to back (stride H*d).
// lse (may be null): [N, H] natural-log log-sum-exp of each row's scores.
// in_type: kInF16, kInBF16 or kInFP8; out_f16: O is fp16 instead of fp32.
hipError_t launch_fused(const f3s_plan_s &p, const void *Q, const void *K,
                        const void *V, int in_type, void *O, bool out_f16, float *lse,
                        int32_t H, int32_t d, float scale_log2, hipStream_t s);
hipError_t launch_fused_bf16(const f3s_plan_s &p, const void *Q, const void *K,
                             const void *V, void *O, bool out_f16, float *lse, int32_t H,
                             int32_t d, float scale_log2, hipStream_t s);
// Measurement instance of the one-head fp16 -> fp32 forward: the same result
// in O, plus a 32-byte record per workgroup in trace (start and end times on
// the constant clock, hardware ids of the compute unit, workgroup index).
hipError_t launch_fused_trace(const f3s_plan_s &p, const void *Q, const void *K,
                              const void *V, void *O, int32_t d, float sl2, uint32_t *trace,
                              hipStream_t s);
// Ablation: fp16 -> fp32 forward with 4-byte K/V gathers (plan flag bit 1).
hipError_t launch_fused_narrow(const f3s_plan_s &p, const void *Q, const void *K,
                               const void *V, void *O, float *lse, int32_t H, int32_t d,
                               float scale_log2, hipStream_t s);
// Ablation: fp16 -> fp32 forward with the split-row partition of a window
// among its waves (plan flag bit 3; d a multiple of 64, 32-bit addressing).
hipError_t launch_fused_split_row(const f3s_plan_s &p, const void *Q, const void *K,
                                  const void *V, float *O, float *lse, int32_t H, int32_t d,
                                  float scale_log2, hipStream_t s);
hipError_t launch_fused_fp8(const f3s_plan_s &p, const void *Q, const void *K,
                            const void *V, void *O, bool out_f16, float *lse, int32_t H,
                            int32_t d, float scale_log2, hipStream_t s);

// Records s as this thread's last error (f3s_last_error) and returns it.
f3s_status_t record_error(f3s_status_t s);

// Gradients (backward_kernel.h; fp16 inputs: backward.hip, bf16 inputs:
// backward_bf16.hip).  pt is the plan of the transposed pattern; row_stats:
// [N, H, 2] (base-2 lse, delta) written by the dQ pass.
hipError_t launch_backward(const f3s_plan_s &p, const f3s_plan_s &pt, const void *Q,
                           const void *K, const void *V, const float *O, const void *G,
                           const float *lse, float *row_stats, float *dQ, float *dK, float *dV,
                           int32_t H, int32_t d, float scale, hipStream_t s);
hipError_t launch_backward_bf16(const f3s_plan_s &p, const f3s_plan_s &pt, const void *Q,
                                const void *K, const void *V, const float *O, const void *G,
                                const float *lse, float *row_stats, float *dQ, float *dK,
                                float *dV, int32_t H, int32_t d, float scale, hipStream_t s);

}  // namespace f3s
