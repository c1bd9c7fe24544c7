// Work plans for the segmented reductions (built once per sparsity pattern).
//
// A plan cuts the entries of a sorted sparse operand (the rows of a CSR or
// the columns of a CSC) into work items of about L entries:
//   * a short segment (1 <= length <= S = L + min(L, 32)) is never split;
//     consecutive short segments are packed into one item while their merged
//     cost (entries + one per segment) starts inside the same window of L;
//   * a long segment (length > S) is cut into chunks of L entries, one item
//     each, whose partial sums are combined afterwards in chunk order;
//   * empty segments get no item; they are listed for a zero fill.
// Work per item is therefore bounded by L + S entries whatever the length
// distribution, and only long segments ever need a second pass.
//
// Construction (all on the GPU, with device-wide scans):
//   cost_r  = length + 1 for a short segment, L for a long one, 0 if empty;
//   pos_r   = exclusive sum of cost; window g_r = pos_r / L;
//   a short segment starts an item when the previous short segment lies in
//   another window (exclusive max-scan of g over short segments); the L added
//   for a long segment always moves the next short segment to a new window,
//   so no item spans a long segment;
//   items per segment: ceil(length / L) if long, 1 if it starts a group;
//   one more exclusive sum gives every item's index and entry offset; further
//   sums list the long segments, the huge ones (more than kHugeChunks chunks,
//   combined by a whole block instead of one wave), every chunk item, and the
//   empty segments.
#include <algorithm>

#include "nsd_internal.hpp"

namespace nsd {

constexpr int kPlanThreads = 256;
constexpr int kHugeChunks = 64;

// A segment is long (chunked) above L + min(L, 32) entries: keeping slightly
// longer segments whole spares the combine pass to most moderate lengths at
// small L, while items stay near L entries at large L (measured on MI355X).
__host__ __device__ __forceinline__ int64_t short_max(int32_t L) {
    return (int64_t)L + (L < 32 ? L : 32);
}
__device__ __forceinline__ bool seg_long(int32_t len, int32_t L) { return len > short_max(L); }

static int64_t plan_grid(int64_t n) { return ceil_div(n > 0 ? n : 1, kPlanThreads); }

__global__ void plan_cost_kernel(int32_t nseg, const int32_t *segptr, int32_t L, int32_t *cost,
                                 int32_t *is_long, int32_t *is_empty) {
    const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (r >= nseg) return;
    const int32_t len = segptr[r + 1] - segptr[r];
    const bool lg = seg_long(len, L);
    cost[r] = len == 0 ? 0 : (lg ? L : len + 1);
    is_long[r] = lg;
    is_empty[r] = len == 0;
}

__global__ void plan_window_kernel(int32_t nseg, const int32_t *segptr, int32_t L,
                                   const int32_t *pos, int32_t *win) {
    const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (r >= nseg) return;
    const int32_t len = segptr[r + 1] - segptr[r];
    win[r] = (len >= 1 && !seg_long(len, L)) ? pos[r] / L : INT32_MIN;
}

__global__ void plan_count_kernel(int32_t nseg, const int32_t *segptr, int32_t L,
                                  const int32_t *pos, const int32_t *prev_win, int32_t *nitem,
                                  int32_t *nchunk, int32_t *is_huge, int32_t *longest) {
    const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (r >= nseg) return;
    const int32_t len = segptr[r + 1] - segptr[r];
    const bool lg = seg_long(len, L);
    if (lg) {
        nitem[r] = (len + L - 1) / L;
    } else if (len >= 1) {
        nitem[r] = prev_win[r] != pos[r] / L ? 1 : 0;
    } else {
        nitem[r] = 0;
    }
    nchunk[r] = lg ? nitem[r] : 0;
    is_huge[r] = lg && nitem[r] > kHugeChunks;
    if (lg) atomicMax(longest, nitem[r]);  // integer max: order-independent
}

struct PlanScans {
    const int32_t *nitem, *ipos, *lpos, *hpos, *cpos, *epos, *is_huge;
};

__global__ void plan_fill_kernel(int32_t nseg, int32_t nnz, const int32_t *segptr, int32_t L,
                                 PlanScans sc, int32_t *item_ptr, int32_t *long_seg,
                                 int32_t *long_first, int32_t *huge_idx, int32_t *chunk_item,
                                 int32_t *chunk_ord, int32_t *empty_seg) {
    const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (r >= nseg) return;
    const int32_t *nitem = sc.nitem;
    const int32_t *ipos = sc.ipos;
    const int32_t b = segptr[r], len = segptr[r + 1] - b;
    const int32_t first = ipos[r];
    if (seg_long(len, L)) {
        for (int32_t c = 0; c < nitem[r]; ++c) {
            item_ptr[first + c] = b + c * L;
            chunk_item[sc.cpos[r] + c] = first + c;
            chunk_ord[first + c] = sc.cpos[r] + c;
        }
        long_seg[sc.lpos[r]] = (int32_t)r;
        long_first[sc.lpos[r]] = first;
        if (sc.is_huge[r]) huge_idx[sc.hpos[r]] = sc.lpos[r];
    } else if (len >= 1) {
        if (nitem[r]) {
            item_ptr[first] = b;
            chunk_ord[first] = -1;
        }
    } else {
        empty_seg[sc.epos[r]] = (int32_t)r;
    }
    if (r == nseg - 1) item_ptr[first + nitem[r]] = nnz;
}

__global__ void plan_sentinel_kernel(int32_t *item_ptr, int32_t nnz) { item_ptr[0] = nnz; }

static size_t plan_ws_bytes(int64_t nseg) {
    Carver c(nullptr);
    for (int i = 0; i < 13; ++i) c.take<int32_t>(nseg > 0 ? nseg : 1);
    c.take<int32_t>(64);
    return c.bytes() + scan_ws_bytes(nseg);
}

}  // namespace nsd

using namespace nsd;

extern "C" {

nsd_status nsd_plan_item_len(int32_t nnz, int32_t k, int32_t *item_len) {
    NSD_REQUIRE(item_len != nullptr, "item_len is NULL");
    NSD_REQUIRE(nnz >= 0 && k >= 1, "need nnz >= 0 and k >= 1");
    // about 32 waves of items per SIMD (256 CUs x 4 SIMDs), an item being
    // one slot of a wave (a slot covers min(k, 256) columns); measured on
    // MI355X this is within 2% of the best length for every workload shape
    // tried (1M to 60M entries, k = 32 to 256)
    const WidthPlan wp = width_plan(k, true);
    const int64_t slots = 32768LL * (kWave / wp.g);
    int32_t L = 16;
    while (L < 256 && (int64_t)L * 2 * slots <= nnz) L <<= 1;
    // small inputs: if 16-entry items would not give every SIMD one wave of
    // items, shorten them (down to 2) so that the serial walk of each slot,
    // not the idle chip, sets the time (10K entries at k = 1: 8.4 us per
    // launch at L = 2 against 18.1 us at L = 16)
    const int64_t fill = 1024LL * (kWave / wp.g);
    if ((int64_t)16 * fill > nnz) {
        L = 2;
        while (L < 16 && (int64_t)L * 2 * fill <= nnz) L <<= 1;
    }
    *item_len = L;
    return NSD_OK;
}

nsd_status nsd_plan_bounds(int32_t nseg, int32_t nnz, int32_t item_len, int32_t *max_items,
                           int32_t *max_long, int32_t *max_chunks, size_t *ws_bytes) {
    NSD_REQUIRE(nseg >= 0 && nnz >= 0 && item_len >= 1, "need nseg, nnz >= 0, item_len >= 1");
    NSD_REQUIRE(max_items && max_long && max_chunks && ws_bytes, "null pointer");
    if (2LL * nnz + nseg >= (1LL << 31)) return fail(NSD_ERR_TOO_LARGE, "plan cost overflows int32");
    *max_items = std::min(nseg, nnz) + 2 * (nnz / item_len) + 1;
    *max_long = nnz / (item_len + 1) + 1;
    *max_chunks = 2 * (nnz / item_len) + 1;
    *ws_bytes = plan_ws_bytes(nseg);
    return NSD_OK;
}

nsd_status nsd_plan_build(int32_t nseg, int32_t nnz, const int32_t *segptr, int32_t item_len,
                          int32_t *item_ptr, int32_t *long_seg, int32_t *long_first,
                          int32_t *huge_idx, int32_t *chunk_item, int32_t *chunk_ord,
                          int32_t *empty_seg, nsd_plan *plan, void *ws, size_t ws_bytes,
                          void *stream) {
    NSD_REQUIRE(nseg >= 0 && nnz >= 0 && item_len >= 1, "need nseg, nnz >= 0, item_len >= 1");
    NSD_REQUIRE(plan && item_ptr, "null pointer");
    NSD_REQUIRE(nseg == 0 || (segptr && long_seg && long_first && huge_idx && chunk_item &&
                              chunk_ord && empty_seg && ws),
                "null pointer");
    if (2LL * nnz + nseg >= (1LL << 31)) return fail(NSD_ERR_TOO_LARGE, "plan cost overflows int32");
    hipStream_t st = as_stream(stream);
    *plan = nsd_plan{};
    plan->item_len = item_len;
    plan->item_ptr = item_ptr;
    plan->long_seg = long_seg;
    plan->long_first = long_first;
    plan->huge_idx = huge_idx;
    plan->chunk_item = chunk_item;
    plan->chunk_ord = chunk_ord;
    plan->empty_seg = empty_seg;
    if (nseg == 0) {
        plan_sentinel_kernel<<<1, 1, 0, st>>>(item_ptr, 0);
        NSD_TRY(check_launch("plan_sentinel_kernel"));
        NSD_HIP(hipStreamSynchronize(st));
        return NSD_OK;
    }
    if (ws_bytes < plan_ws_bytes(nseg))
        return fail(NSD_ERR_WORKSPACE, "workspace %zu < %zu", ws_bytes, plan_ws_bytes(nseg));
    Carver c(ws);
    int32_t *cost = c.take<int32_t>(nseg);
    int32_t *is_long = c.take<int32_t>(nseg);
    int32_t *is_empty = c.take<int32_t>(nseg);
    int32_t *pos = c.take<int32_t>(nseg);
    int32_t *win = c.take<int32_t>(nseg);
    int32_t *nitem = c.take<int32_t>(nseg);
    int32_t *ipos = c.take<int32_t>(nseg);
    int32_t *lpos = c.take<int32_t>(nseg);
    int32_t *epos = c.take<int32_t>(nseg);
    int32_t *nchunk = c.take<int32_t>(nseg);
    int32_t *cpos = c.take<int32_t>(nseg);
    int32_t *is_huge = c.take<int32_t>(nseg);
    int32_t *hpos = c.take<int32_t>(nseg);
    int32_t *tot = c.take<int32_t>(64);
    void *scan_ws = c.base + c.bytes();
    const int64_t g = plan_grid(nseg);

    plan_cost_kernel<<<g, kPlanThreads, 0, st>>>(nseg, segptr, item_len, cost, is_long, is_empty);
    NSD_TRY(check_launch("plan_cost_kernel"));
    NSD_TRY(scan_exclusive(cost, pos, nseg, nullptr, scan_ws, st));
    plan_window_kernel<<<g, kPlanThreads, 0, st>>>(nseg, segptr, item_len, pos, win);
    NSD_TRY(check_launch("plan_window_kernel"));
    NSD_TRY(scan_exclusive_max(win, win, nseg, scan_ws, st));
    NSD_HIP(hipMemsetAsync(tot + 5, 0, sizeof(int32_t), st));
    plan_count_kernel<<<g, kPlanThreads, 0, st>>>(nseg, segptr, item_len, pos, win, nitem, nchunk,
                                                  is_huge, tot + 5);
    NSD_TRY(check_launch("plan_count_kernel"));
    NSD_TRY(scan_exclusive(nitem, ipos, nseg, tot + 0, scan_ws, st));
    NSD_TRY(scan_exclusive(is_long, lpos, nseg, tot + 1, scan_ws, st));
    NSD_TRY(scan_exclusive(is_empty, epos, nseg, tot + 2, scan_ws, st));
    NSD_TRY(scan_exclusive(nchunk, cpos, nseg, tot + 3, scan_ws, st));
    NSD_TRY(scan_exclusive(is_huge, hpos, nseg, tot + 4, scan_ws, st));
    PlanScans sc{nitem, ipos, lpos, hpos, cpos, epos, is_huge};
    plan_fill_kernel<<<g, kPlanThreads, 0, st>>>(nseg, nnz, segptr, item_len, sc, item_ptr, long_seg,
                                                 long_first, huge_idx, chunk_item, chunk_ord,
                                                 empty_seg);
    NSD_TRY(check_launch("plan_fill_kernel"));
    int32_t h[6];
    NSD_HIP(hipMemcpyAsync(h, tot, sizeof(h), hipMemcpyDeviceToHost, st));
    NSD_HIP(hipStreamSynchronize(st));
    plan->nitems = h[0];
    plan->nlong = h[1];
    plan->nempty = h[2];
    plan->nchunks = h[3];
    plan->nhuge = h[4];
    plan->longest_chunks = h[5];
    return NSD_OK;
}

}  // extern "C"
