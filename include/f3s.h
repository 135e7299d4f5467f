/*
 * f3s.h -- fused sparse attention (3S) on AMD MI355X (gfx950).
 *
 * The operator (Fused3S, Section 2.1, Eq. 1, with the masked reading of the
 * element-wise product and the max-stabilised online softmax of Section 3.5):
 *
 *     O = softmax_rows( mask_A( scale * Q K^T ) ) V
 *
 * A is a binary N x N pattern given as CSR.  For row i only the columns j
 * with A[i][j] != 0 enter the softmax; a row without any such column gives
 * O[i,:] = 0.  Precisions follow Table 5: Q, K, V fp16, scores and softmax
 * fp32, the normalised scores cast to fp16 for the second product, O fp32.
 *
 * Two calls:
 *   f3s_plan  builds, on the GPU, the Binary Sparse Block layout of
 *             Section 3.1 (16-row windows, all-zero columns removed, 16x16
 *             blocks with one 256-bit bitmap each) and the heavy-first work
 *             list of Section 3.2 (with heavy windows split into pieces).
 *   f3s_run   evaluates the operator with the fused kernel of Algorithm 1
 *             (score block, mask, online softmax, fp16 probabilities, value
 *             product, final normalisation; scores never reach HBM).
 *
 * Threading: calls are thread-safe except that one plan must not be used by
 * two f3s_run calls that overlap in time (they share the plan's partial-result
 * scratch).  Different plans may run concurrently.
 */
#ifndef F3S_H
#define F3S_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    F3S_OK = 0,
    F3S_ERR_INVALID_VALUE = 1, /* null/misaligned pointer, bad size, aliasing   */
    F3S_ERR_INVALID_CSR = 2,   /* row_ptr[0] != 0, decreasing, column not in [0,N) */
    F3S_ERR_UNSUPPORTED = 3,   /* d not a multiple of 32 in [32, 256]           */
    F3S_ERR_OUT_OF_MEMORY = 4, /* a device allocation failed (environment
                                  F3S_ALLOC_LIMIT_BYTES=<n> makes every
                                  allocation above n bytes fail this way)      */
    F3S_ERR_HIP = 5,           /* any other HIP runtime error                   */
    F3S_ERR_TOO_LARGE = 6,     /* the call needs more than a fixed capacity of
                                  the library (f3s_backward_noalloc)            */
    /* not statuses: they give the type the whole int32 range, so any int a
       caller passes (f3s_status_string) is a valid value of the type */
    F3S_STATUS_MIN_ = -2147483647 - 1,
    F3S_STATUS_MAX_ = 2147483647
} f3s_status_t;

typedef struct f3s_plan_s *f3s_plan_t;

typedef struct {
    int32_t N;             /* rows (= columns) of A                              */
    int32_t n_windows;     /* T_r = ceil(N / 16) (Algorithm 1), or the windows
                              of f3s_plan_segments                              */
    int64_t nnz_csr;       /* entries in the CSR, repeats included               */
    int64_t nnz;           /* distinct (row, column) pairs: the non-zeros of A   */
    int64_t n_unique;      /* sum over windows of distinct columns (bc, Table 3) */
    int64_t n_blocks;      /* 16x16 blocks (b, Table 3)                          */
    int32_t max_blocks;    /* largest block count of one window                  */
    int32_t piece_blocks;  /* windows with more blocks are split into pieces     */
    int32_t n_items;       /* work items (windows or pieces) in the work list    */
    int32_t n_split;       /* windows that were split                            */
    int32_t n_pieces;      /* pieces in total (partial-result slots)             */
    int32_t flags;         /* bit 0: work list in window order (forced, or
                              chosen for nearly uniform windows; see f3s_plan);
                              bit 1: narrow K/V gathers (ablation);
                              bit 2: windows aligned to the graphs of a batch
                              (f3s_plan_segments);
                              bit 3: split-row forward (ablation)                */
    int64_t bsb_bytes;     /* window offsets + column lists + bitmaps            */
    int64_t device_bytes;  /* everything the plan holds on the device            */
    double build_ms;       /* wall time of f3s_plan                              */
} f3s_plan_info_t;

/*
 * Build a plan from a CSR pattern that lives in DEVICE memory.
 * Environment (read at plan time; for ablations):
 *   F3S_PIECE_BLOCKS=<even n>  piece size of split windows (capped at the
 *                              largest window)
 *   F3S_NO_REORDER=1           work list in window order instead of
 *                              decreasing block count (Section 3.2);
 *                              =0 always sorts.  Unset, plans of nearly
 *                              uniform windows (at least 2048, the largest
 *                              at most twice the mean block count) keep
 *                              window order, which lets the forward and
 *                              backward give each XCD runs of
 *                              neighbouring windows; all others are sorted
 *   F3S_NARROW_GATHER=1        the fp16 -> fp32 forward gathers K and V rows
 *                              in 4-byte words instead of 16-byte chunks (the
 *                              access granularity without the register
 *                              remapping of Section 3.4); other type pairs
 *                              then return F3S_ERR_UNSUPPORTED
 *   F3S_SPLIT_ROW=1            the fp16 -> fp32 forward partitions each
 *                              window among 2 or 4 waves by feature slices
 *                              (split-row score product summed through LDS
 *                              once per block pair, split-column value
 *                              product; Section 3.3) instead of by block
 *                              pairs; d must be a multiple of 64 and Q/K/V
 *                              below 4 GiB, and other type pairs, other d
 *                              or F3S_NARROW_GATHER=1 together with it
 *                              return F3S_ERR_UNSUPPORTED
 *   row_ptr  int32[N+1], row_ptr[0] == 0, non-decreasing
 *   col_idx  int32[row_ptr[N]], every entry in [0, N); order inside a row is
 *            free and repeated entries count once (A is binary, Section 3.1)
 *   N        >= 0; N == 0 gives a valid empty plan
 * The plan copies what it needs: the caller may free the CSR on return.
 * Synchronous on the current device's null stream.  Returns NULL on error;
 * f3s_last_error() then tells why (F3S_ERR_INVALID_CSR for a malformed
 * pattern, nothing is leaked).
 */
f3s_plan_t f3s_plan(const int32_t *row_ptr, const int32_t *col_idx, int32_t N);

/*
 * Device bytes of scratch a build of f3s_plan_ws needs for a pattern of N
 * rows and nnz CSR entries: 6 bytes per entry plus about 110 per row
 * window (0 for negative sizes).  Host-only; calls no HIP function.
 */
size_t f3s_plan_workspace_bytes(int32_t N, int64_t nnz);

/*
 * f3s_plan with the build's scratch lent by the caller instead of allocated
 * and freed by the library (a caching allocator can then serve repeated
 * builds): workspace is device memory of at least
 * f3s_plan_workspace_bytes(N, row_ptr[N]) bytes, 256-byte aligned.  The
 * plan keeps no reference to it; the build is synchronous, so the caller
 * may reuse or free it on return.  The plan's own arrays are still
 * allocated by the library.  A workspace that is null, misaligned or too
 * small gives F3S_ERR_INVALID_VALUE.  Otherwise as f3s_plan.
 */
f3s_plan_t f3s_plan_ws(const int32_t *row_ptr, const int32_t *col_idx, int32_t N,
                       void *workspace, size_t workspace_bytes);

/*
 * f3s_plan for a batch of graphs stored as one block-diagonal pattern, with
 * row windows aligned to the graphs (the use of component boundaries that
 * Section 4.2 leaves to future work).  Graph g holds the consecutive rows
 * seg_ptr[g] .. seg_ptr[g+1] - 1.  Walking from row 0, a window is the next
 * 16 rows of the current graph while more than 16 of them remain; otherwise
 * it is the rest of that graph together with every whole graph after it
 * that still fits into 16 rows (empty graphs always fit).  A window thus
 * holds 1 to 16 rows and never part of a graph together with rows of
 * another, except that a long graph's last rows may share a window with
 * whole small graphs.  The block layout, bitmaps (rows counted from the
 * window's first row) and work list are those of f3s_plan over these
 * windows.
 *   seg_ptr  HOST int32[n_segs + 1]: seg_ptr[0] == 0, non-decreasing,
 *            seg_ptr[n_segs] == N (else F3S_ERR_INVALID_VALUE); the caller
 *            keeps ownership
 *   n_segs   >= 0 graphs
 * The segments only choose the windows: the operator's result is the same
 * for any segmentation, also when edges cross segments.  Such a plan serves
 * every forward and backward call; f3s_plan_transpose gives it a plan of A^T
 * with 16-row windows (built from the rows of A^T, never a copy).  Otherwise
 * as f3s_plan.
 */
f3s_plan_t f3s_plan_segments(const int32_t *row_ptr, const int32_t *col_idx, int32_t N,
                             const int32_t *seg_ptr, int32_t n_segs);

/*
 * O = softmax_rows(mask_A(scale * Q K^T)) V  (Algorithm 1, Section 3).
 *   Q, K, V  device, fp16, N x d row-major, contiguous, 16-byte aligned; they
 *            may alias each other (Q = K = V as in AGNN, Section 2.1)
 *   O        device, fp32, N x d row-major, 16-byte aligned, must not overlap
 *            Q, K or V; every row is overwritten (empty rows with 0)
 *   d        multiple of 32, 32 <= d <= 256
 *   scale    finite; multiplies the fp32 dot products
 *   stream   HIP stream of the device the plan was built on (else
 *            F3S_ERR_INVALID_VALUE); the call is asynchronous on it,
 *            allocates nothing and copies nothing between host and device
 * Inputs must be finite.  Returns F3S_OK or an error code (no launch happens
 * on an argument error).
 */
f3s_status_t f3s_run(f3s_plan_t plan, const void *Q, const void *K, const void *V,
                     void *O, int32_t d, float scale, hipStream_t stream);

/*
 * Multi-head form: n_heads independent operators that share one pattern A
 * (the attention layer of a Graph Transformer, Section 2.1 Eq. 4, has one
 * per head).  Q, K, V are fp16 [N, n_heads, d] row-major (row i holds head h
 * at elements (i*n_heads + h)*d ...), O is fp32 [N, n_heads, d]; head h of O
 * is the single-head operator applied to head h of Q, K, V.  Same pointer,
 * alignment, d, scale and stream rules as f3s_run; n_heads >= 1 and
 * n_items * n_heads < 2^31.  f3s_run is f3s_run_mh with n_heads = 1.
 * All heads run in one launch: head by head when K and V (all heads)
 * exceed the 256 MB Infinity Cache, when n_heads does not divide 8, or when
 * the plan's windows are nearly uniform (then each XCD takes consecutive
 * ranges of one head's work list at a time), window-major otherwise
 * (environment F3S_HEAD_MAJOR_BYTES=<bytes> replaces these tests with a K/V
 * size threshold; results are identical either way).  When a launch would have fewer waves than the GPU has SIMDs
 * (work items x heads < 1024) four waves share each work item, and two when
 * twice the waves still fit the GPU at once; they combine their partial
 * softmax states (environment F3S_WAVES_PER_ITEM=1, 2 or 4 forces the
 * count; the rounding of the combination differs).
 */
f3s_status_t f3s_run_mh(f3s_plan_t plan, const void *Q, const void *K, const void *V,
                        void *O, int32_t n_heads, int32_t d, float scale,
                        hipStream_t stream);

/*
 * Forward with the per-row log-sum-exp kept for a later backward call.
 *   lse  device fp32 [N, n_heads] (4-byte aligned) or NULL: for row i, head h,
 *        lse = log(sum_j exp(scale * Q_i . K_j)) over the row's columns
 *        (natural log; -inf for an empty row)
 * Everything else as f3s_run_mh (which is f3s_forward with lse = NULL).
 */
f3s_status_t f3s_forward(f3s_plan_t plan, const void *Q, const void *K, const void *V,
                         void *O, float *lse, int32_t n_heads, int32_t d, float scale,
                         hipStream_t stream);

/* Element types of the typed forward. */
typedef enum {
    F3S_DTYPE_F16 = 0,   /* IEEE 754 binary16 */
    F3S_DTYPE_BF16 = 1,  /* bfloat16: the upper 16 bits of an IEEE binary32 */
    F3S_DTYPE_F32 = 2,   /* IEEE 754 binary32 */
    F3S_DTYPE_FP8_E4M3 = 3,  /* OCP 8-bit float e4m3 (bias 7, finite to 448, no inf) */
    /* not types: the whole int32 range is a valid value (others are rejected
       with F3S_ERR_UNSUPPORTED) */
    F3S_DTYPE_MIN_ = -2147483647 - 1,
    F3S_DTYPE_MAX_ = 2147483647
} f3s_dtype_t;

/*
 * Forward with a choice of storage types (the precision variants beside
 * Table 5's scheme).
 *   in_dtype   type of Q, K, V: F3S_DTYPE_F16 (Table 5), F3S_DTYPE_BF16 or
 *              F3S_DTYPE_FP8_E4M3 (the 8-bit inputs the paper's future work
 *              names).  With bf16 inputs the scores use the bf16 matrix
 *              product and the probabilities enter the value product as two
 *              bf16 terms (about 16 significant bits), so the error stays
 *              within the fp16 scheme's bound.  fp8 inputs are widened to
 *              fp16 exactly as they are loaded and then follow the fp16
 *              scheme; any per-tensor dequantisation factor of Q and K folds
 *              into `scale`, and one of V multiplies O afterwards.
 *   out_dtype  type of O: F3S_DTYPE_F32 (Table 5) or F3S_DTYPE_F16 (the
 *              normalised fp32 result rounded to nearest even).
 * Other types give F3S_ERR_UNSUPPORTED.  Layouts, alignment, d, scale, lse
 * and stream rules as f3s_forward, with element sizes taken from the types.
 * f3s_forward is this call with (F3S_DTYPE_F16, F3S_DTYPE_F32).
 */
f3s_status_t f3s_forward_typed(f3s_plan_t plan, const void *Q, const void *K, const void *V,
                               f3s_dtype_t in_dtype, void *O, f3s_dtype_t out_dtype,
                               float *lse, int32_t n_heads, int32_t d, float scale,
                               hipStream_t stream);

/*
 * Plan of the transposed pattern A^T, built on the GPU from `plan` alone
 * (its bitmaps list A's entries).  Needed by f3s_backward: the gradients of
 * K and V are sums over the rows that attend to a key, i.e. over the rows of
 * A^T, so each window of A^T owns its keys' gradients (no atomics).  An
 * exact symmetry check first: if A^T = A the result is a copy of the plan.
 * The check runs on the plan for patterns below 8 M entries and on the
 * sorted rows of A^T above (environment F3S_SYMMETRY_SORT_FIRST=<entries>
 * moves that threshold; 0 always sorts first).  A plan of f3s_plan_segments
 * skips the check: its A^T always gets its own plan of 16-row windows.
 * Synchronous; NULL on error (f3s_last_error).  Destroy with f3s_destroy.
 */
f3s_plan_t f3s_plan_transpose(f3s_plan_t plan);

/*
 * Device bytes of scratch f3s_plan_transpose_ws needs for `plan` (0 for a
 * null plan).  Host-only.
 */
size_t f3s_plan_transpose_workspace_bytes(f3s_plan_t plan);

/*
 * f3s_plan_transpose with its scratch lent by the caller (device memory of
 * at least f3s_plan_transpose_workspace_bytes(plan) bytes, 256-byte
 * aligned; no reference kept, reusable on return).  The new plan's own
 * arrays are still allocated by the library.  A null, misaligned or short
 * workspace gives F3S_ERR_INVALID_VALUE.
 */
f3s_plan_t f3s_plan_transpose_ws(f3s_plan_t plan, void *workspace, size_t workspace_bytes);

/*
 * Gradients of L with respect to Q, K, V given G = dL/dO (the backward pass
 * the paper leaves to future work).  With P the forward probabilities:
 *   delta_i = G_i . O_i,  dS_ij = P_ij (G_i . V_j - delta_i)  on the pattern,
 *   dQ = scale dS K,  dK = scale dS^T Q,  dV = P^T G.
 *   plan, plan_t  a plan and f3s_plan_transpose(plan)
 *   Q, K, V, dO   device fp16 [N, n_heads, d] (the forward's inputs, and G)
 *   O, lse        device fp32: the forward's output [N, n_heads, d] and
 *                 log-sum-exp [N, n_heads] from f3s_forward
 *   row_stats     device fp32 [N, n_heads, 2], written: per row and head the
 *                 base-2 log-sum-exp (lse * log2 e) and delta_i = G_i . O_i;
 *                 8-byte aligned.  The dK/dV pass gathers this one 8-byte
 *                 record for every row attending to a key.
 *   dQ, dK, dV    device fp32 [N, n_heads, d], every element written
 *   d             multiple of 32, 32 <= d <= 256 (as the forward)
 * P and dS enter the products as fp16 (round to nearest even).  Outputs must
 * not overlap each other or any input; 16-byte aligned (lse: 4, row_stats: 8).
 * Asynchronous on `stream` (of the device both plans were built on, else
 * F3S_ERR_INVALID_VALUE), no allocation.  Deterministic (no atomics).
 */
f3s_status_t f3s_backward(f3s_plan_t plan, f3s_plan_t plan_t, const void *Q,
                          const void *K, const void *V, const float *O, const void *dO,
                          const float *lse, float *row_stats, float *dQ, float *dK,
                          float *dV, int32_t n_heads, int32_t d, float scale,
                          hipStream_t stream);

/*
 * f3s_backward with a choice of input type: in_dtype F3S_DTYPE_F16 (as
 * f3s_backward) or F3S_DTYPE_BF16, the type of Q, K, V and dO (O, lse and
 * the outputs stay fp32).  With bf16 inputs the score and dP products use
 * the bf16 matrix product, and P and dS enter the gradient products as two
 * bf16 terms each (about 16 significant bits), so the error stays within
 * the fp16 scheme's bound.  Other types give F3S_ERR_UNSUPPORTED.  Layouts,
 * alignment, d, heads and stream rules as f3s_backward.  O and lse come
 * from f3s_forward_typed with the same inputs and an fp32 O.
 */
f3s_status_t f3s_backward_typed(f3s_plan_t plan, f3s_plan_t plan_t, const void *Q,
                                const void *K, const void *V, f3s_dtype_t in_dtype,
                                const float *O, const void *dO, const float *lse,
                                float *row_stats, float *dQ, float *dK, float *dV,
                                int32_t n_heads, int32_t d, float scale, hipStream_t stream);

/*
 * f3s_backward_typed for callers that cannot allocate device memory (code
 * under HIP graph capture, serving loops, harnesses that forbid hipMalloc):
 * the per-row (base-2 lse, delta) records that f3s_backward_typed keeps in
 * the caller's row_stats buffer live instead in a fixed array of the
 * library, 16 MiB per device, holding f3s_backward_noalloc_max_records()
 * = 2^21 (row, head) records; the array is looked up on the first call on
 * a device (make one call before capturing a graph) and held until the
 * process ends.  The call allocates nothing and never frees.
 *   N * n_heads above 2^21 gives F3S_ERR_TOO_LARGE (nothing launched).
 *   Every other argument, and the result, as f3s_backward_typed.
 * All calls on one device share that device's array: two calls that
 * overlap in time on one device (two streams, two threads) race and give
 * wrong gradients; calls on one stream are ordered and safe.  The array's
 * contents are written by each call before they are read (nothing has to
 * start at zero).
 */
f3s_status_t f3s_backward_noalloc(f3s_plan_t plan, f3s_plan_t plan_t, const void *Q,
                                  const void *K, const void *V, f3s_dtype_t in_dtype,
                                  const float *O, const void *dO, const float *lse,
                                  float *dQ, float *dK, float *dV, int32_t n_heads,
                                  int32_t d, float scale, hipStream_t stream);

/* Capacity of f3s_backward_noalloc's array in (row, head) records.  Host-only. */
int64_t f3s_backward_noalloc_max_records(void);

/* Release a plan and all its device memory.  NULL is a no-op. */
void f3s_destroy(f3s_plan_t plan);

/* Sizes and statistics of a plan (host struct filled on return). */
f3s_status_t f3s_plan_info(f3s_plan_t plan, f3s_plan_info_t *out);

/*
 * Copy the plan's layout to HOST buffers (for inspection and tests).  Any
 * pointer may be NULL to skip that array.  Sizes come from f3s_plan_info:
 *   blk_off  int32[n_windows + 1]  first block of each window (the tro array)
 *   cols     int32[16 * n_blocks]  original column of each compacted block
 *                                  column (the sptd gather list), -1 = padding
 *   mask     uint32[8 * n_blocks]  bitmap of each block: the non-zero at
 *                                  window row r, block column c is bit
 *                                  k = 4*(r + 16*(c/4)) + c%4, i.e. bit k%32 of
 *                                  word k/32
 *   items    int32[4 * n_items]    work list in launch order: window, first
 *                                  block, end block, partial slot (-1 = none)
 *   merges   int32[3 * n_split]    split windows: window, first slot, pieces
 * Synchronous.
 */
f3s_status_t f3s_plan_export(f3s_plan_t plan, int32_t *blk_off, int32_t *cols,
                             uint32_t *mask, int32_t *items, int32_t *merges);

/*
 * The first row of every window of the plan followed by N (int32[n_windows
 * + 1], HOST buffer): 16 w for the windows of f3s_plan, the windows chosen
 * by f3s_plan_segments for its plans.  Synchronous.
 */
f3s_status_t f3s_plan_window_rows(f3s_plan_t plan, int32_t *win_row);

/* Status of the last failing call on this thread (F3S_OK if none). */
f3s_status_t f3s_last_error(void);

/* Static, human-readable name of a status code. */
const char *f3s_status_string(f3s_status_t status);

#ifdef __cplusplus
}
#endif

#endif /* F3S_H */
