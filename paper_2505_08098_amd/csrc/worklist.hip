// Heavy-first work list of a plan (Section 3.2), in O(T) memory: the windows
// are stably sorted by their key, largest first (radix.hip), the item counts
// are scanned in that order, and every window writes its item (or, if split,
// its merge record and first item position; its pieces are written by
// k_split_items).
#include "f3s_internal.h"

namespace f3s {
namespace {

// Window order[i] (window i without an order) starts at item pos[i].
__global__ void k_place_items(const int32_t *order, const int32_t *pos, const int32_t *nb,
                              const int32_t *blk_off, const int32_t *npieces,
                              const int32_t *slot_base, const int32_t *split_idx, int32_t T,
                              int32_t piece, WorkItem *items, int32_t *merges,
                              int32_t *split_item)
{
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= T) return;
    const int w = order ? order[i] : i, p = pos[i];
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

hipError_t launch_worklist(const int32_t *key, const int32_t *nb, const int32_t *blk_off,
                           const int32_t *npieces, const int32_t *slot_base,
                           const int32_t *split_idx, int32_t T, int32_t piece,
                           bool window_order, const WorkListScratch &ws, WorkItem *items,
                           int32_t *merges, int32_t *split_item, int32_t *n_items_out,
                           hipStream_t s)
{
    if (T == 0) return hipSuccess;
    // the window indices, sorted by key (values: the indices themselves)
    const int32_t *sorted_keys = nullptr, *order = nullptr;
    hipError_t e = hipSuccess;
    if (!window_order) {
        e = launch_radix_pairs(key, nullptr, T, piece, true, ws.radix, &sorted_keys, &order,
                               s);
        if (e != hipSuccess) return e;
    }
    // first item of each window in that order: scan of its item counts
    ScanArray a;
    a.in = npieces;
    a.gather = order;
    a.out = ws.pos;
    a.total = n_items_out;
    e = launch_scan(a, T, ws.radix.scan_tmp, s);
    if (e != hipSuccess) return e;
    k_place_items<<<blocks_for(T, 256), 256, 0, s>>>(order, ws.pos, nb, blk_off, npieces,
                                                     slot_base, split_idx, T, piece, items,
                                                     merges, split_item);
    return hipGetLastError();
}

}  // namespace f3s
