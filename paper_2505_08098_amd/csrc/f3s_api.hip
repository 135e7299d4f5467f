// C ABI of the f3s library: argument checks, plan orchestration, dispatch.
#include <math.h>
#include <stdlib.h>
#include <string.h>

#include <atomic>
#include <chrono>
#include <new>
#include <vector>

#include "f3s_internal.h"
#include "f3s_probe.h"

namespace {

thread_local f3s_status_t g_last_error = F3S_OK;
std::atomic<uint64_t> g_next_plan_id{1};

f3s_status_t fail(f3s_status_t s)
{
    g_last_error = s;
    return s;
}

f3s_status_t from_hip(hipError_t e)
{
    if (e == hipSuccess) return F3S_OK;
    return e == hipErrorOutOfMemory ? F3S_ERR_OUT_OF_MEMORY : F3S_ERR_HIP;
}

// Largest single device allocation the library makes: F3S_ALLOC_LIMIT_BYTES
// when set (a larger request then fails as if the device were out of
// memory, so tests can drive every out-of-memory path from the host),
// otherwise unlimited.
size_t alloc_limit()
{
    const char *e = getenv("F3S_ALLOC_LIMIT_BYTES");
    return e && *e ? (size_t)strtoull(e, nullptr, 10) : ~(size_t)0;
}

// One device allocation carved into 256-byte aligned pieces (the scratch of
// one f3s_plan call, or a plan's arrays); sizing pass first (add), then one
// hipMalloc (alloc), then the pieces in the same order (take).
struct Arena {
    char *base = nullptr;
    size_t used = 0, cap = 0;
    static size_t round(size_t b) { return (b + 255) & ~(size_t)255; }
    template <typename T>
    void add(int64_t count)
    {
        cap += round((size_t)(count > 0 ? count : 1) * sizeof(T));
    }
    hipError_t alloc()
    {
        const size_t n = cap ? cap : 256;
        if (n > alloc_limit()) return hipErrorOutOfMemory;
        return hipMalloc((void **)&base, n);
    }
    template <typename T>
    T *take(int64_t count)
    {
        T *p = reinterpret_cast<T *>(base + used);
        used += round((size_t)(count > 0 ? count : 1) * sizeof(T));
        return p;
    }
};

// Scratch arena freed on every exit path of a plan build (unless the caller
// lent the memory).
struct ScratchArena : Arena {
    bool owned = true;
    ~ScratchArena()
    {
        if (base && owned) (void)hipFree(base);
    }
};

void free_plan_arrays(f3s_plan_s *p)
{
    if (p->store) (void)hipFree(p->store);
    if (p->part_store) (void)hipFree(p->part_store);
    p->store = p->part_store = nullptr;
    p->blk_off = nullptr;
    p->cols = nullptr;
    p->mask = nullptr;
    p->items = nullptr;
    p->merges = nullptr;
    p->win_row = nullptr;
    p->part_o = nullptr;
    p->part_ml = nullptr;
}

// Partial-result buffers of split windows: part_row floats per piece row
// for O (kMaxD for a plan, 2 * kMaxD for a transposed plan, which holds the
// dK and dV partials), and the (m, l) records.  Replaces any previous ones.
hipError_t alloc_parts(f3s_plan_s *p, int32_t part_row)
{
    if (p->part_store) {
        (void)hipFree(p->part_store);
        p->device_bytes -= (int64_t)p->part_bytes;
        p->part_store = nullptr;
        p->part_o = p->part_ml = nullptr;
        p->part_bytes = 0;
    }
    p->part_row = part_row;
    if (p->n_pieces == 0) return hipSuccess;
    Arena a;
    a.add<float>((int64_t)p->n_pieces * f3s::kWindowRows * part_row);
    // one (m, l) record of 16 + 16 floats per piece and head of a launch
    // group; a group holds at most kMaxD / 32 heads (nh * d <= kMaxD)
    a.add<float>((int64_t)p->n_pieces * 32 * (f3s::kMaxD / 32));
    hipError_t e = a.alloc();
    if (e != hipSuccess) return e;
    p->part_store = a.base;
    p->part_bytes = (int64_t)a.cap;
    p->device_bytes += (int64_t)a.cap;
    p->part_o = a.take<float>((int64_t)p->n_pieces * f3s::kWindowRows * part_row);
    p->part_ml = a.take<float>((int64_t)p->n_pieces * 32 * (f3s::kMaxD / 32));
    return hipSuccess;
}

// The plan's arrays in one allocation, laid out from its counts (T, blocks,
// items, split windows): blk_off, cols, mask, items, merges, and the window
// rows of a plan aligned to the graphs of a batch.  Returns the allocation's
// size in *bytes.
hipError_t alloc_store(f3s_plan_s *p, size_t *bytes)
{
    using namespace f3s;
    const int64_t B = p->n_blocks;
    Arena a;
    a.add<int32_t>((int64_t)p->T + 1);
    a.add<int32_t>((int64_t)kBlockCols * B);
    a.add<uint32_t>((int64_t)kMaskWords * B);
    a.add<WorkItem>(p->n_items);
    a.add<int32_t>(3ll * p->n_split);
    if (p->flags & 4) a.add<int32_t>((int64_t)p->T + 1);
    hipError_t e = a.alloc();
    if (e != hipSuccess) return e;
    p->store = a.base;
    p->device_bytes += (int64_t)a.cap;
    p->blk_off = a.take<int32_t>((int64_t)p->T + 1);
    p->cols = a.take<int32_t>((int64_t)kBlockCols * B);
    p->mask = a.take<uint32_t>((int64_t)kMaskWords * B);
    p->items = a.take<WorkItem>(p->n_items);
    p->merges = a.take<int32_t>(3ll * p->n_split);
    p->win_row = (p->flags & 4) ? a.take<int32_t>((int64_t)p->T + 1) : nullptr;
    if (bytes) *bytes = a.cap;
    return hipSuccess;
}

int env_int(const char *name, int dflt)
{
    const char *v = getenv(name);
    if (!v || !*v) return dflt;
    return atoi(v);
}

#define HIP_TRY(expr)                                          \
    do {                                                       \
        hipError_t e_ = (expr);                                \
        if (e_ != hipSuccess) return from_hip(e_);             \
    } while (0)

// Work-list slots of a device: 8 per compute unit (the count is queried
// once per device; a full property query costs tens of microseconds).
int32_t plan_slots(int device)
{
    constexpr int kMaxDevices = 64;
    static std::atomic<int32_t> cached[kMaxDevices] = {};
    if (device >= 0 && device < kMaxDevices) {
        const int32_t c = cached[device].load(std::memory_order_relaxed);
        if (c > 0) return c;
    }
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device) !=
            hipSuccess ||
        cus <= 0)
        cus = 256;
    if (device >= 0 && device < kMaxDevices) cached[device].store(8 * cus);
    return 8 * cus;
}

// Device-side statistics of a plan build, read back with one copy each
// time the host needs them.
struct BuildStats {
    unsigned long long n_unique;  // sum of distinct columns over windows
    unsigned long long nnz;       // set bits of all bitmaps
    int32_t err;                  // malformed CSR
    int32_t n_big;                // windows too large for one wavefront
    int32_t n_heavy;              // windows too large for the LDS sort
    int32_t max_blocks;
    int32_t n_blocks;
    int32_t piece;
    int32_t n_pieces;
    int32_t n_split;
    int32_t n_items;              // item count from the work-list scan
    int32_t invalid;              // plan integrity check
};

// Pointers into the plan build's scratch.
struct BuildScratch {
    BuildStats *st;
    int32_t *tmp_cols;   // sorted distinct columns per window, at its CSR offset
    uint32_t *tmp_mask;  // block bitmaps per window, staged
    int32_t *u, *big, *is_big, *heavy, *is_heavy, *bits, *nb, *npieces, *key, *split_item;
    int32_t *big_pos, *heavy_pos, *split_pieces, *split_one, *scan_tmp;
    int32_t *win_row;    // the windows' first rows (null: 16-row windows)
    f3s::WorkListScratch wl;  // the work-list sort
};

template <typename U>
U *carve(Arena &a, bool take, int64_t n)
{
    if (take) return a.take<U>(n);
    a.add<U>(n);
    return nullptr;
}

// Row windows of an N-row pattern (64-bit sum: N may be up to 2^31 - 1).
int32_t num_windows(int32_t N)
{
    return (int32_t)(((int64_t)N + f3s::kWindowRows - 1) / f3s::kWindowRows);
}

// Lays out the build's scratch for T windows and nnz CSR entries (and the
// windows' first rows if `rows`): sizes into a (take == false) or pointers
// out of it (take == true), in one order.  O(nnz + T) bytes.
void carve_scratch(Arena &a, bool take, BuildScratch &b, int32_t T, int64_t nnz,
                   bool rows = false)
{
    using namespace f3s;
    b.st = carve<BuildStats>(a, take, 1);
    b.win_row = rows ? carve<int32_t>(a, take, (int64_t)T + 1) : nullptr;
    b.tmp_cols = carve<int32_t>(a, take, nnz);
    b.tmp_mask = carve<uint32_t>(a, take, mask_stage_words(nnz, T));
    int32_t **per_window[] = {&b.u, &b.big, &b.is_big, &b.heavy, &b.is_heavy,
                              &b.bits, &b.nb, &b.npieces, &b.key, &b.split_item};
    for (int32_t **q : per_window) *q = carve<int32_t>(a, take, T);
    int32_t **per_window1[] = {&b.big_pos, &b.heavy_pos, &b.split_pieces, &b.split_one};
    for (int32_t **q : per_window1) *q = carve<int32_t>(a, take, (int64_t)T + 1);
    const int64_t rc = radix_count_ints(T);
    b.scan_tmp = carve<int32_t>(a, take, scan_tmp_ints(T > rc ? T : rc));
    b.wl.pos = carve<int32_t>(a, take, (int64_t)T + 1);
    int32_t **radix_arrays[] = {&b.wl.radix.keys_a, &b.wl.radix.vals_a, &b.wl.radix.keys_b,
                                &b.wl.radix.vals_b};
    for (int32_t **q : radix_arrays) *q = carve<int32_t>(a, take, T);
    b.wl.radix.counts = carve<int32_t>(a, take, rc);
    b.wl.radix.scan_tmp = b.scan_tmp;
}

size_t plan_workspace_bytes(int32_t N, int64_t nnz)
{
    Arena a;
    BuildScratch b;
    const int32_t T = num_windows(N);
    carve_scratch(a, false, b, T, nnz);
    return a.cap;
}

// win_rows: the windows' first rows and N (T + 1 ints, host memory), or null
// for 16-row windows.
f3s_status_t build_plan(f3s_plan_s *p, const int32_t *row_ptr, const int32_t *col_idx,
                        int32_t part_row, void *workspace, size_t workspace_bytes,
                        const int32_t *win_rows)
{
    using namespace f3s;
    const hipStream_t s = nullptr;
    const int32_t N = p->N;
    const int32_t T = p->T;

    // ---- 1. nnz (row_ptr[0] == 0 and monotonicity are checked on the GPU)
    int32_t nnz = 0;
    HIP_TRY(hipMemcpy(&nnz, row_ptr + N, sizeof(int32_t), hipMemcpyDeviceToHost));
    if (nnz < 0) return F3S_ERR_INVALID_CSR;
    if (nnz > 0 && !col_idx) return F3S_ERR_INVALID_VALUE;
    p->nnz_csr = nnz;

    // all scratch of the build in one allocation (or the caller's workspace)
    const int32_t slots = plan_slots(p->device);
    BuildScratch b;
    ScratchArena tmp;
    carve_scratch(tmp, false, b, T, nnz, win_rows != nullptr);
    if (workspace) {
        if (workspace_bytes < tmp.cap || ((uintptr_t)workspace & 255u))
            return F3S_ERR_INVALID_VALUE;
        tmp.base = static_cast<char *>(workspace);
        tmp.owned = false;
    } else {
        HIP_TRY(tmp.alloc());
    }
    carve_scratch(tmp, true, b, T, nnz, win_rows != nullptr);
    const int32_t *wr = b.win_row;
    if (wr)
        HIP_TRY(hipMemcpy(b.win_row, win_rows, sizeof(int32_t) * ((size_t)T + 1),
                          hipMemcpyHostToDevice));
    BuildStats *st = b.st;
    int32_t *tmp_cols = b.tmp_cols;
    uint32_t *tmp_mask = b.tmp_mask;
    int32_t *u = b.u, *big = b.big, *is_big = b.is_big, *heavy = b.heavy;
    int32_t *is_heavy = b.is_heavy, *bits = b.bits, *nb = b.nb, *npieces = b.npieces;
    int32_t *key = b.key, *split_item = b.split_item, *big_pos = b.big_pos;
    int32_t *heavy_pos = b.heavy_pos, *split_pieces = b.split_pieces;
    int32_t *split_one = b.split_one, *scan_tmp = b.scan_tmp;
    BuildStats hs;
    HIP_TRY(hipMemsetAsync(st, 0, sizeof(BuildStats), s));

    // ---- 2. CSR check, distinct columns and bitmaps per window ----------
    HIP_TRY(launch_check_row_ptr(row_ptr, N, nnz, &st->err, s));
    HIP_TRY(launch_window_wave(row_ptr, col_idx, N, wr, T, tmp_cols, tmp_mask, u, is_big,
                               is_heavy, bits, &st->err, s));
    {  // the flagged windows listed in window order
        ScanArray fb, fh;
        fb.in = is_big;
        fb.out = big_pos;
        fb.total = &st->n_big;
        fb.list = big;
        fh.in = is_heavy;
        fh.out = heavy_pos;
        fh.total = &st->n_heavy;
        fh.list = heavy;
        HIP_TRY(launch_scan2(fb, fh, T, scan_tmp, s));
    }
    HIP_TRY(hipMemcpy(&hs, st, sizeof hs, hipMemcpyDeviceToHost));
    if (hs.err) return F3S_ERR_INVALID_CSR;
    HIP_TRY(launch_window_sort(row_ptr, col_idx, N, wr, big, hs.n_big, tmp_cols, tmp_mask,
                               u, bits, &st->err, s));
    HIP_TRY(launch_heavy_lds(row_ptr, col_idx, N, wr, heavy, hs.n_heavy, tmp_cols,
                             tmp_mask, u, bits, &st->err, s));

    // ---- 3. blocks per window and statistics; work-list shape: piece size,
    //         split windows, item count (one host round trip for all) -------
    HIP_TRY(launch_window_stats(u, bits, T, nb, &st->n_unique, &st->nnz, &st->n_blocks,
                                &st->max_blocks, s));
    // F3S_NO_REORDER=1 keeps window order, =0 always sorts; unset, the order
    // is chosen below once the block counts are known
    const char *order_env = getenv("F3S_NO_REORDER");
    const bool order_forced = order_env && *order_env;
    const bool reorder = !order_forced || atoi(order_env) == 0;
    p->flags = (reorder ? 0 : 1) | (env_int("F3S_NARROW_GATHER", 0) ? 2 : 0) | (wr ? 4 : 0) |
               (env_int("F3S_SPLIT_ROW", 0) ? 8 : 0);
    HIP_TRY(launch_bin_keys(nb, T, &st->n_blocks, &st->max_blocks,
                            env_int("F3S_PIECE_BLOCKS", 0), slots, reorder,
                            &st->piece, npieces, key, split_pieces, split_one, s));
    {
        ScanArray sp, so;
        sp.in = sp.out = split_pieces;
        sp.total = &st->n_pieces;
        so.in = so.out = split_one;
        so.total = &st->n_split;
        HIP_TRY(launch_scan2(sp, so, T, scan_tmp, s));
    }
    HIP_TRY(hipMemcpy(&hs, st, sizeof hs, hipMemcpyDeviceToHost));
    if (hs.err) return F3S_ERR_INVALID_CSR;
    const int32_t B = hs.n_blocks;
    p->n_blocks = B;
    p->n_unique = (int64_t)hs.n_unique;
    p->nnz = (int64_t)hs.nnz;
    p->max_blocks = hs.max_blocks;
    p->bsb_bytes = 4ll * (T + 1) + 4ll * kBlockCols * B + 4ll * kMaskWords * B;
    const int32_t piece = hs.piece;
    p->piece = piece;
    p->n_pieces = hs.n_pieces;
    p->n_split = hs.n_split;
    const int64_t n_items = (int64_t)T - p->n_split + p->n_pieces;
    if (n_items > INT32_MAX) return F3S_ERR_UNSUPPORTED;
    p->n_items = (int32_t)n_items;
    // Nearly uniform windows (the largest at most twice the mean, and many of
    // them) leave the heavy-first sort nothing to balance; window order then
    // keeps neighbouring windows -- which share K/V rows on banded and
    // block-diagonal patterns -- next to each other in the work list, which
    // the forward hands to each XCD as one consecutive range.
    if (reorder && !order_forced && uniform_windows(T, B, hs.max_blocks)) p->flags |= 1;
    const bool window_order = (p->flags & 1) != 0;

    // ---- 4. the plan's arrays: one allocation, plus the partial buffers --
    HIP_TRY(alloc_store(p, nullptr));
    HIP_TRY(alloc_parts(p, part_row));
    HIP_TRY(launch_scan(nb, p->blk_off, T, scan_tmp, nullptr, s));  // window block offsets
    if (wr)
        HIP_TRY(hipMemcpyAsync(p->win_row, wr, sizeof(int32_t) * ((size_t)T + 1),
                               hipMemcpyDeviceToDevice, s));

    // ---- 5. column lists and bitmaps into their blocks --------------------
    HIP_TRY(launch_fill_windows(row_ptr, wr, T, tmp_cols, tmp_mask, u, p->blk_off, p->cols,
                                p->mask, s));

    // ---- 6. work list: windows stably sorted by key, heavy first (or kept
    //         in window order) ----------------------------------------------
    HIP_TRY(launch_worklist(key, nb, p->blk_off, npieces, split_pieces, split_one, T, piece,
                            window_order, b.wl, p->items, p->merges, split_item,
                            &st->n_items, s));
    HIP_TRY(launch_split_items(p->merges, split_item, p->blk_off, p->n_split, p->items, s));

    // ---- 7. integrity check of the finished plan ------------------------
    HIP_TRY(launch_validate_plan(*p, &st->invalid, s));
    HIP_TRY(hipMemcpy(&hs, st, sizeof hs, hipMemcpyDeviceToHost));
    if (hs.invalid || hs.n_items != p->n_items) return F3S_ERR_HIP;
    return F3S_OK;
}

bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }

// The plan's arrays live on one device: a launch on another device's stream
// would read them from the wrong memory.
bool on_plan_device(const f3s_plan_s *p, hipStream_t stream)
{
    int dev = -1;
    const hipError_t e = stream ? hipStreamGetDevice(stream, &dev) : hipGetDevice(&dev);
    return e == hipSuccess && dev == p->device;
}

bool overlaps(const void *a, size_t na, const void *b, size_t nb)
{
    const uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
    return x < y + nb && y < x + na;
}

// A copy of plan src (same arrays, new id) whose split-window partials hold
// part_row floats per row.
f3s_plan_t clone_plan(const f3s_plan_s *src, int32_t part_row)
{
    f3s_plan_s *t = new (std::nothrow) f3s_plan_s(*src);
    if (!t) {
        fail(F3S_ERR_OUT_OF_MEMORY);
        return nullptr;
    }
    t->nnz_csr = t->nnz;  // the pattern without duplicate entries, like A^T's CSR
    t->store = t->part_store = nullptr;
    t->part_o = t->part_ml = nullptr;
    t->part_bytes = 0;
    t->device_bytes = 0;
    t->id = g_next_plan_id.fetch_add(1);
    t->transpose_of = 0;
    size_t bytes = 0;
    hipError_t e = alloc_store(t, &bytes);
    if (e == hipSuccess)
        e = hipMemcpy(t->store, src->store, bytes, hipMemcpyDeviceToDevice);
    if (e == hipSuccess) e = alloc_parts(t, part_row);
    if (e != hipSuccess) {
        free_plan_arrays(t);
        delete t;
        fail(from_hip(e));
        return nullptr;
    }
    return t;
}

// Builds a plan whose split-window partials hold part_row floats per row;
// win_rows (host, T + 1 ints) gives the windows' first rows, null the 16-row
// windows.
f3s_plan_t make_plan(const int32_t *row_ptr, const int32_t *col_idx, int32_t N,
                     int32_t part_row, void *workspace, size_t workspace_bytes,
                     const int32_t *win_rows = nullptr, int32_t T = 0)
{
    const auto t0 = std::chrono::steady_clock::now();
    if (N < 0 || (N > 0 && !row_ptr)) {
        fail(F3S_ERR_INVALID_VALUE);
        return nullptr;
    }
    f3s_plan_s *p = new (std::nothrow) f3s_plan_s();
    if (!p) {
        fail(F3S_ERR_OUT_OF_MEMORY);
        return nullptr;
    }
    p->N = N;
    p->T = win_rows ? T : num_windows(N);
    p->id = g_next_plan_id.fetch_add(1);
    f3s_status_t st = from_hip(hipGetDevice(&p->device));
    if (st == F3S_OK) {
        if (N == 0) {
            st = from_hip(alloc_store(p, nullptr));
            if (st == F3S_OK) st = from_hip(hipMemset(p->blk_off, 0, sizeof(int32_t)));
            p->piece = 16;
            p->part_row = part_row;
        } else {
            st = build_plan(p, row_ptr, col_idx, part_row, workspace, workspace_bytes,
                            win_rows);
        }
    }
    if (st != F3S_OK) {
        (void)hipDeviceSynchronize();
        (void)hipGetLastError();
        free_plan_arrays(p);
        delete p;
        fail(st);
        return nullptr;
    }
    p->build_ms = std::chrono::duration<double, std::milli>(
                      std::chrono::steady_clock::now() - t0).count();
    return p;
}

// Windows aligned to the segments (the graphs of a batch; segment g holds
// rows seg[g] .. seg[g+1] - 1): walking from row 0, a window is the next 16
// rows of the current segment while more than 16 of them remain, otherwise
// the rest of the segment together with every whole segment after it that
// still fits into 16 rows.  So no window mixes part of a graph with rows of
// another, except that a long graph's last rows may share a window with
// whole small graphs.  Returns the windows' first rows followed by N.
std::vector<int32_t> segment_windows(const int32_t *seg, int32_t n_segs)
{
    std::vector<int32_t> starts;
    const int32_t N = seg[n_segs];
    int32_t g = 0;
    for (int32_t r = 0; r < N;) {
        while (seg[g + 1] <= r) ++g;  // the segment holding row r
        starts.push_back(r);
        if (seg[g + 1] - r > f3s::kWindowRows) {
            r += f3s::kWindowRows;
            continue;
        }
        const int32_t first = r;
        r = seg[++g];
        while (g < n_segs && seg[g + 1] - first <= f3s::kWindowRows) r = seg[++g];
    }
    starts.push_back(N);
    return starts;
}

// Patterns with at least this many entries check symmetry on the sorted CSR
// of A^T (F3S_SYMMETRY_SORT_FIRST overrides the count: 0 always sorts first).
constexpr int kSortFirstEntries = 8 << 20;

// Scratch of a transposition of src: the CSR of A^T, the transposition's
// own scratch, a flag, and (with_build) the scratch of a plan build of A^T.
struct TransposeScratch {
    int32_t *rp, *ci, *asym, *win, *pre;
    void *tr, *inner;
    size_t tr_bytes, inner_bytes;
};

void carve_transpose(Arena &a, bool take, TransposeScratch &t, const f3s_plan_s *src,
                     bool with_build)
{
    t.tr_bytes = f3s::transpose_scratch_bytes(*src);
    t.inner_bytes = with_build ? plan_workspace_bytes(src->N, src->nnz) : 0;
    t.rp = carve<int32_t>(a, take, (int64_t)src->N + 1);
    t.ci = carve<int32_t>(a, take, src->nnz);
    t.asym = carve<int32_t>(a, take, 1);
    t.win = carve<int32_t>(a, take, src->n_blocks);
    t.pre = carve<int32_t>(a, take, (int64_t)f3s::kWindowRows * src->n_blocks);
    t.tr = carve<char>(a, take, (int64_t)t.tr_bytes);
    t.inner = with_build ? carve<char>(a, take, (int64_t)t.inner_bytes) : nullptr;
}

size_t transpose_workspace_bytes(const f3s_plan_s *src, bool with_build)
{
    Arena a;
    TransposeScratch t;
    carve_transpose(a, false, t, src, with_build);
    return a.cap;
}

// Plan of A^T from a plan of A: an exact symmetry check (on the plan, or for
// large patterns on the CSR of A^T); if A^T = A the plan is copied,
// otherwise the plan of A^T is built from its CSR (radix sort).  Its split-window partials hold two
// rows (dK, dV) per piece row, so a launch group still holds heads with
// nh * d <= kMaxD.
f3s_plan_t make_transpose(f3s_plan_t src, void *workspace, size_t workspace_bytes)
{
    const auto t0 = std::chrono::steady_clock::now();
    if (!src) {
        fail(F3S_ERR_INVALID_VALUE);
        return nullptr;
    }
    f3s_status_t st = F3S_OK;
    auto step = [&](hipError_t e) {
        if (st == F3S_OK && e != hipSuccess) st = from_hip(e);
    };
    int prev_device = 0;
    step(hipGetDevice(&prev_device));
    step(hipSetDevice(src->device));
    f3s_plan_t t = nullptr;
    {
        const bool lent = workspace != nullptr;
        TransposeScratch ts;
        ScratchArena tmp;
        carve_transpose(tmp, false, ts, src, lent);
        if (lent) {
            if (workspace_bytes < tmp.cap || ((uintptr_t)workspace & 255u))
                st = F3S_ERR_INVALID_VALUE;
            tmp.base = static_cast<char *>(workspace);
            tmp.owned = false;
        } else if (st == F3S_OK) {
            step(tmp.alloc());
        }
        if (st == F3S_OK) {
            carve_transpose(tmp, true, ts, src, lent);
            int32_t h = 1;
            // symmetric?  Small patterns: checked on the plan first (no sort);
            // large ones: on A^T's sorted rows, which are needed anyway if not.
            // A plan whose windows follow the graphs of a batch skips the check
            // (it assumes 16-row windows): its A^T gets a plan of 16-row
            // windows built from A^T's rows.
            const bool small = src->nnz < env_int("F3S_SYMMETRY_SORT_FIRST", kSortFirstEntries);
            bool have_csr = false;
            if (!src->win_row) {
                step(hipMemsetAsync(ts.asym, 0, sizeof(int32_t), nullptr));
                if (small) {
                    step(f3s::launch_check_symmetric(*src, ts.win, ts.asym, nullptr));
                } else {
                    step(f3s::launch_transpose_csr(*src, ts.tr, ts.tr_bytes, ts.rp, ts.ci,
                                                   nullptr));
                    step(f3s::launch_compare_rows(*src, ts.rp, ts.ci, ts.win, ts.pre,
                                                  ts.asym, nullptr));
                    have_csr = true;
                }
                step(hipMemcpy(&h, ts.asym, sizeof(int32_t), hipMemcpyDeviceToHost));
            }
            if (st == F3S_OK && h == 0) {
                t = clone_plan(src, 2 * f3s::kMaxD);
                if (!t) st = g_last_error;
            } else if (st == F3S_OK) {
                if (!have_csr)
                    step(f3s::launch_transpose_csr(*src, ts.tr, ts.tr_bytes, ts.rp, ts.ci,
                                                   nullptr));
                if (st == F3S_OK) {
                    t = make_plan(ts.rp, ts.ci, src->N, 2 * f3s::kMaxD, ts.inner,
                                  ts.inner_bytes);
                    if (!t) st = g_last_error;
                }
            }
        }
    }
    (void)hipSetDevice(prev_device);
    if (st != F3S_OK) {
        (void)hipDeviceSynchronize();
        f3s_destroy(t);
        fail(st);
        return nullptr;
    }
    t->transpose_of = src->id;
    t->build_ms = std::chrono::duration<double, std::milli>(
                      std::chrono::steady_clock::now() - t0).count();
    return t;
}

}  // namespace

namespace f3s {
f3s_status_t record_error(f3s_status_t s) { return fail(s); }
}  // namespace f3s

extern "C" {

const char *f3s_status_string(f3s_status_t status)
{
    switch (status) {
    case F3S_OK: return "F3S_OK";
    case F3S_ERR_INVALID_VALUE: return "F3S_ERR_INVALID_VALUE";
    case F3S_ERR_INVALID_CSR: return "F3S_ERR_INVALID_CSR";
    case F3S_ERR_UNSUPPORTED: return "F3S_ERR_UNSUPPORTED";
    case F3S_ERR_OUT_OF_MEMORY: return "F3S_ERR_OUT_OF_MEMORY";
    case F3S_ERR_HIP: return "F3S_ERR_HIP";
    case F3S_ERR_TOO_LARGE: return "F3S_ERR_TOO_LARGE";
    default: break;
    }
    return "F3S_ERR_UNKNOWN";
}

f3s_status_t f3s_last_error(void) { return g_last_error; }

f3s_plan_t f3s_plan(const int32_t *row_ptr, const int32_t *col_idx, int32_t N)
{
    return make_plan(row_ptr, col_idx, N, f3s::kMaxD, nullptr, 0);
}

size_t f3s_plan_workspace_bytes(int32_t N, int64_t nnz)
{
    if (N < 0 || nnz < 0) return 0;
    return plan_workspace_bytes(N, nnz);
}

f3s_plan_t f3s_plan_ws(const int32_t *row_ptr, const int32_t *col_idx, int32_t N,
                       void *workspace, size_t workspace_bytes)
{
    if (!workspace) {
        fail(F3S_ERR_INVALID_VALUE);
        return nullptr;
    }
    return make_plan(row_ptr, col_idx, N, f3s::kMaxD, workspace, workspace_bytes);
}

f3s_plan_t f3s_plan_segments(const int32_t *row_ptr, const int32_t *col_idx, int32_t N,
                             const int32_t *seg_ptr, int32_t n_segs)
{
    if (N < 0 || !seg_ptr || n_segs < 0 || seg_ptr[0] != 0 || seg_ptr[n_segs] != N) {
        fail(F3S_ERR_INVALID_VALUE);
        return nullptr;
    }
    for (int32_t g = 0; g < n_segs; ++g) {
        if (seg_ptr[g + 1] < seg_ptr[g]) {
            fail(F3S_ERR_INVALID_VALUE);
            return nullptr;
        }
    }
    std::vector<int32_t> starts;
    try {
        starts = segment_windows(seg_ptr, n_segs);
    } catch (const std::bad_alloc &) {
        fail(F3S_ERR_OUT_OF_MEMORY);
        return nullptr;
    }
    return make_plan(row_ptr, col_idx, N, f3s::kMaxD, nullptr, 0, starts.data(),
                     (int32_t)starts.size() - 1);
}

f3s_status_t f3s_plan_window_rows(f3s_plan_t p, int32_t *win_row)
{
    if (!p || !win_row) return fail(F3S_ERR_INVALID_VALUE);
    if (p->win_row) {
        const f3s_status_t st = from_hip(hipMemcpy(
            win_row, p->win_row, sizeof(int32_t) * ((size_t)p->T + 1), hipMemcpyDeviceToHost));
        return st == F3S_OK ? F3S_OK : fail(st);
    }
    for (int32_t w = 0; w < p->T; ++w) win_row[w] = w * f3s::kWindowRows;
    win_row[p->T] = p->N;
    return F3S_OK;
}

f3s_plan_t f3s_plan_transpose(f3s_plan_t src)
{
    return make_transpose(src, nullptr, 0);
}

size_t f3s_plan_transpose_workspace_bytes(f3s_plan_t src)
{
    return src ? transpose_workspace_bytes(src, true) : 0;
}

f3s_plan_t f3s_plan_transpose_ws(f3s_plan_t src, void *workspace, size_t workspace_bytes)
{
    if (!workspace) {
        fail(F3S_ERR_INVALID_VALUE);
        return nullptr;
    }
    return make_transpose(src, workspace, workspace_bytes);
}

void f3s_destroy(f3s_plan_t plan)
{
    if (!plan) return;
    free_plan_arrays(plan);
    delete plan;
}

f3s_status_t f3s_plan_info(f3s_plan_t p, f3s_plan_info_t *out)
{
    if (!p || !out) return fail(F3S_ERR_INVALID_VALUE);
    memset(out, 0, sizeof(*out));
    out->N = p->N;
    out->n_windows = p->T;
    out->nnz_csr = p->nnz_csr;
    out->nnz = p->nnz;
    out->n_unique = p->n_unique;
    out->n_blocks = p->n_blocks;
    out->max_blocks = p->max_blocks;
    out->piece_blocks = p->piece;
    out->n_items = p->n_items;
    out->n_split = p->n_split;
    out->n_pieces = p->n_pieces;
    out->flags = p->flags;
    out->bsb_bytes = p->bsb_bytes;
    out->device_bytes = p->device_bytes;
    out->build_ms = p->build_ms;
    return F3S_OK;
}

f3s_status_t f3s_plan_export(f3s_plan_t p, int32_t *blk_off, int32_t *cols,
                             uint32_t *mask, int32_t *items, int32_t *merges)
{
    if (!p) return fail(F3S_ERR_INVALID_VALUE);
    struct {
        void *dst;
        const void *src;
        size_t bytes;
    } cp[] = {
        {blk_off, p->blk_off, 4ull * (p->T + 1)},
        {cols, p->cols, 4ull * f3s::kBlockCols * p->n_blocks},
        {mask, p->mask, 4ull * f3s::kMaskWords * p->n_blocks},
        {items, p->items, sizeof(f3s::WorkItem) * p->n_items},
        {merges, p->merges, 12ull * p->n_split},
    };
    for (auto &c : cp) {
        if (!c.dst || c.bytes == 0) continue;
        f3s_status_t st = from_hip(hipMemcpy(c.dst, c.src, c.bytes, hipMemcpyDeviceToHost));
        if (st != F3S_OK) return fail(st);
    }
    return F3S_OK;
}

f3s_status_t f3s_forward_typed(f3s_plan_t p, const void *Q, const void *K, const void *V,
                               f3s_dtype_t in_dtype, void *O, f3s_dtype_t out_dtype,
                               float *lse, int32_t n_heads, int32_t d, float scale,
                               hipStream_t stream)
{
    if (!p || n_heads < 1) return fail(F3S_ERR_INVALID_VALUE);
    if (d < 32 || d > f3s::kMaxD || d % 32 != 0) return fail(F3S_ERR_UNSUPPORTED);
    if (in_dtype != F3S_DTYPE_F16 && in_dtype != F3S_DTYPE_BF16 &&
        in_dtype != F3S_DTYPE_FP8_E4M3)
        return fail(F3S_ERR_UNSUPPORTED);
    if (out_dtype != F3S_DTYPE_F32 && out_dtype != F3S_DTYPE_F16)
        return fail(F3S_ERR_UNSUPPORTED);
    // the narrow-gather ablation exists for fp16 -> fp32 only, the split-row
    // one also only for d a multiple of 64 and 32-bit addressing; not both
    if ((p->flags & 10) && (in_dtype != F3S_DTYPE_F16 || out_dtype != F3S_DTYPE_F32))
        return fail(F3S_ERR_UNSUPPORTED);
    if ((p->flags & 8) && ((p->flags & 2) || d % 64 != 0 ||
                           (uint64_t)p->N * (uint64_t)n_heads * (uint64_t)d * 2u >
                               0xFFFFFFF0ull))
        return fail(F3S_ERR_UNSUPPORTED);
    if (!isfinite(scale)) return fail(F3S_ERR_INVALID_VALUE);
    if (p->N == 0) return F3S_OK;
    if (!on_plan_device(p, stream)) return fail(F3S_ERR_INVALID_VALUE);
    if (!Q || !K || !V || !O) return fail(F3S_ERR_INVALID_VALUE);
    if (!aligned16(Q) || !aligned16(K) || !aligned16(V) || !aligned16(O))
        return fail(F3S_ERR_INVALID_VALUE);
    if ((uint64_t)p->n_items * (uint64_t)n_heads > 0x7FFFFFFFull)
        return fail(F3S_ERR_UNSUPPORTED);
    const size_t elems = (size_t)p->N * (size_t)n_heads * (size_t)d;
    const size_t in_bytes = elems * (in_dtype == F3S_DTYPE_FP8_E4M3 ? 1 : 2);
    const size_t out_bytes = elems * (out_dtype == F3S_DTYPE_F32 ? 4 : 2);
    if (overlaps(O, out_bytes, Q, in_bytes) || overlaps(O, out_bytes, K, in_bytes) ||
        overlaps(O, out_bytes, V, in_bytes))
        return fail(F3S_ERR_INVALID_VALUE);
    // base-2 softmax: 2^(x * scale * log2 e) == e^(x * scale)
    const float sl2 = (float)((double)scale * 1.4426950408889634);
    if (lse && (((uintptr_t)lse & 3u) ||
                overlaps(lse, (size_t)p->N * n_heads * 4, O, out_bytes) ||
                overlaps(lse, (size_t)p->N * n_heads * 4, Q, in_bytes) ||
                overlaps(lse, (size_t)p->N * n_heads * 4, K, in_bytes) ||
                overlaps(lse, (size_t)p->N * n_heads * 4, V, in_bytes)))
        return fail(F3S_ERR_INVALID_VALUE);
    const int in_type = in_dtype == F3S_DTYPE_BF16       ? f3s::kInBF16
                        : in_dtype == F3S_DTYPE_FP8_E4M3 ? f3s::kInFP8
                                                         : f3s::kInF16;
    f3s_status_t st = from_hip(f3s::launch_fused(*p, Q, K, V, in_type, O,
                                                 out_dtype == F3S_DTYPE_F16, lse, n_heads, d,
                                                 sl2, stream));
    return st == F3S_OK ? F3S_OK : fail(st);
}

f3s_status_t f3s_forward(f3s_plan_t p, const void *Q, const void *K, const void *V,
                         void *O, float *lse, int32_t n_heads, int32_t d, float scale,
                         hipStream_t stream)
{
    return f3s_forward_typed(p, Q, K, V, F3S_DTYPE_F16, O, F3S_DTYPE_F32, lse, n_heads, d,
                             scale, stream);
}

f3s_status_t f3s_run_mh(f3s_plan_t p, const void *Q, const void *K, const void *V,
                        void *O, int32_t n_heads, int32_t d, float scale,
                        hipStream_t stream)
{
    return f3s_forward(p, Q, K, V, O, nullptr, n_heads, d, scale, stream);
}

f3s_status_t f3s_backward(f3s_plan_t p, f3s_plan_t pt, const void *Q, const void *K,
                          const void *V, const float *O, const void *dO, const float *lse,
                          float *row_stats, float *dQ, float *dK, float *dV, int32_t n_heads,
                          int32_t d, float scale, hipStream_t stream)
{
    return f3s_backward_typed(p, pt, Q, K, V, F3S_DTYPE_F16, O, dO, lse, row_stats, dQ, dK,
                              dV, n_heads, d, scale, stream);
}

f3s_status_t f3s_backward_typed(f3s_plan_t p, f3s_plan_t pt, const void *Q, const void *K,
                                const void *V, f3s_dtype_t in_dtype, const float *O,
                                const void *dO, const float *lse, float *row_stats, float *dQ,
                                float *dK, float *dV, int32_t n_heads, int32_t d, float scale,
                                hipStream_t stream)
{
    if (in_dtype != F3S_DTYPE_F16 && in_dtype != F3S_DTYPE_BF16)
        return fail(F3S_ERR_UNSUPPORTED);
    if (!p || !pt || n_heads < 1) return fail(F3S_ERR_INVALID_VALUE);
    if (pt->transpose_of != p->id || pt->N != p->N) return fail(F3S_ERR_INVALID_VALUE);
    if (pt->win_row) return fail(F3S_ERR_UNSUPPORTED);  // A^T's plan has 16-row windows
    if (d < 32 || d > f3s::kMaxD || d % 32 != 0) return fail(F3S_ERR_UNSUPPORTED);
    if (!isfinite(scale)) return fail(F3S_ERR_INVALID_VALUE);
    if (p->N == 0) return F3S_OK;
    if (pt->device != p->device || !on_plan_device(p, stream))
        return fail(F3S_ERR_INVALID_VALUE);
    const void *ins[] = {Q, K, V, dO};
    void *outs[] = {dQ, dK, dV};
    for (const void *x : ins)
        if (!x || !aligned16(x)) return fail(F3S_ERR_INVALID_VALUE);
    for (void *x : outs)
        if (!x || !aligned16(x)) return fail(F3S_ERR_INVALID_VALUE);
    if (!O || !aligned16(O) || !lse || !row_stats || ((uintptr_t)lse & 3u) ||
        ((uintptr_t)row_stats & 7u))
        return fail(F3S_ERR_INVALID_VALUE);
    if ((uint64_t)p->n_items * n_heads > 0x7FFFFFFFull ||
        (uint64_t)pt->n_items * n_heads > 0x7FFFFFFFull)
        return fail(F3S_ERR_UNSUPPORTED);
    const size_t elems = (size_t)p->N * n_heads * d;
    const size_t h16 = elems * 2, f32 = elems * 4, rowv = (size_t)p->N * n_heads * 4;
    // outputs must not overlap each other or any input
    struct Span { const void *p; size_t n; };
    const Span in_spans[] = {{Q, h16}, {K, h16}, {V, h16}, {dO, h16}, {O, f32}, {lse, rowv}};
    const Span out_spans[] = {{dQ, f32}, {dK, f32}, {dV, f32}, {row_stats, 2 * rowv}};
    for (const Span &o : out_spans) {
        for (const Span &x : in_spans)
            if (overlaps(o.p, o.n, x.p, x.n)) return fail(F3S_ERR_INVALID_VALUE);
        for (const Span &x : out_spans)
            if (&x != &o && overlaps(o.p, o.n, x.p, x.n)) return fail(F3S_ERR_INVALID_VALUE);
    }
    auto launch = in_dtype == F3S_DTYPE_BF16 ? f3s::launch_backward_bf16 : f3s::launch_backward;
    f3s_status_t st = from_hip(launch(*p, *pt, Q, K, V, O, dO, lse, row_stats, dQ, dK, dV,
                                      n_heads, d, scale, stream));
    return st == F3S_OK ? F3S_OK : fail(st);
}

f3s_status_t f3s_run(f3s_plan_t p, const void *Q, const void *K, const void *V,
                     void *O, int32_t d, float scale, hipStream_t stream)
{
    return f3s_run_mh(p, Q, K, V, O, 1, d, scale, stream);
}

f3s_status_t f3s_run_trace(f3s_plan_t p, const void *Q, const void *K, const void *V,
                           float *O, int32_t d, float scale, uint32_t *trace,
                           size_t trace_bytes, hipStream_t stream)
{
    if (!p) return fail(F3S_ERR_INVALID_VALUE);
    if (d < 32 || d > f3s::kMaxD || d % 32 != 0) return fail(F3S_ERR_UNSUPPORTED);
    if (p->flags & 10) return fail(F3S_ERR_UNSUPPORTED);
    if (!isfinite(scale)) return fail(F3S_ERR_INVALID_VALUE);
    if (p->N == 0) return F3S_OK;
    if (!on_plan_device(p, stream)) return fail(F3S_ERR_INVALID_VALUE);
    if (!Q || !K || !V || !O || !trace) return fail(F3S_ERR_INVALID_VALUE);
    if (!aligned16(Q) || !aligned16(K) || !aligned16(V) || !aligned16(O) || !aligned16(trace))
        return fail(F3S_ERR_INVALID_VALUE);
    const size_t elems = (size_t)p->N * (size_t)d;
    // 32-bit gather offsets only (the traced instance has no 64-bit variant)
    if (elems * 2 > 0xFFFFFFF0ull) return fail(F3S_ERR_UNSUPPORTED);
    const size_t need = 32ull * (size_t)p->n_items;
    if (trace_bytes < need) return fail(F3S_ERR_INVALID_VALUE);
    if (overlaps(O, elems * 4, Q, elems * 2) || overlaps(O, elems * 4, K, elems * 2) ||
        overlaps(O, elems * 4, V, elems * 2) || overlaps(trace, need, O, elems * 4) ||
        overlaps(trace, need, Q, elems * 2) || overlaps(trace, need, K, elems * 2) ||
        overlaps(trace, need, V, elems * 2))
        return fail(F3S_ERR_INVALID_VALUE);
    const float sl2 = (float)((double)scale * 1.4426950408889634);
    f3s_status_t st =
        from_hip(f3s::launch_fused_trace(*p, Q, K, V, O, d, sl2, trace, stream));
    return st == F3S_OK ? F3S_OK : fail(st);
}

int32_t f3s_wall_clock_khz(int32_t device)
{
    int v = 0;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeWallClockRate, device) != hipSuccess)
        return 0;
    return v;
}

}  // extern "C"
