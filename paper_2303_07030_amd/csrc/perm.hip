// A fixed permutation of fp32 values applied in two coalesced passes:
//   dst[q] = src[perm[q]]   for q < n
// (the values of a sparse operand between its CSR and CSC orders, and a
// sparse gradient back; both directions are permutations of this form).
//
// A direct gather reads one 4-byte value per random cache line.  Here the
// permutation is split, once per pattern, into two local ones of bounded
// span (a two-digit radix permutation), so every global access is a whole
// line or a run of consecutive values:
//   pass 1, per source tile of T consecutive elements: the tile is staged in
//     LDS and written out in the order of its elements' destination buckets
//     (B = T consecutive destinations each), one run per bucket, into a
//     staging array whose bucket d occupies [d T, (d + 1) T) and holds its
//     elements in source order;
//   pass 2, per destination bucket: the bucket's staging run is read
//     contiguously, placed in LDS at its local destination offsets, and the
//     bucket is written out contiguously.
// The plan stores, per element, the staging position and the local source
// index of pass 1's output slots, and the local destination offset of the
// staging slots (16-bit local indices: T = 2^15).  It is built with the
// library's stable radix sort.  The result is an exact copy (bit for bit).
#include <algorithm>

#include "nsd_internal.hpp"

namespace nsd {

#ifndef NSD_PERM_TILE
#define NSD_PERM_TILE 32768
#endif
constexpr int kPermThreads = 1024;
constexpr int kPermTile = NSD_PERM_TILE;  // T = B, the LDS span of either pass (128 KiB)
static_assert(kPermTile <= 65536, "local indices are 16-bit");

static int64_t perm_tiles(int64_t n) { return ceil_div(n, kPermTile); }

// ------------------------------------------------------------- apply

// Workgroups go to the eight XCDs round-robin (block b on XCD b mod 8), each
// XCD with its own L2.  This renumbers the blocks so that every XCD takes one
// contiguous range of the tiles: neighbouring tiles write adjacent runs of
// one output region, and with the renumbering those runs meet in one L2 and
// leave it as whole lines instead of partial ones from eight L2s.
__device__ __forceinline__ int64_t xcd_contiguous_tile() {
    const int nb = (int)gridDim.x, b = (int)blockIdx.x, x = b % 8;
    int start = 0;
    for (int y = 0; y < x; ++y) start += (nb - y + 7) / 8;  // blocks on XCDs before x
    return start + b / 8;
}


// Each thread handles kPermPer elements of its tile, strided by the block
// size, in batches of kPermBatch whose loads are all issued before any is
// used (one memory round trip per batch, not per element).  Everything read
// is read once and the result written once: those accesses are
// non-temporal, leaving the L2 to the staging runs of pass 1, which meet
// there with their neighbours' (measured on MI355X, a move of 60M values:
// 0.310 ms with ordinary accesses, 0.266 ms so; the staging stores made
// non-temporal as well, 0.433 ms).
constexpr int kPermPer = kPermTile / kPermThreads;
constexpr int kPermBatch = 8;
static_assert(kPermPer % kPermBatch == 0, "whole batches per thread");

__global__ __launch_bounds__(kPermThreads) void perm_pass1_kernel(int64_t n, const float *src,
                                                                  const int32_t *stage,
                                                                  const uint16_t *src_local,
                                                                  float *staging) {
    __shared__ float tile[kPermTile];
    const int64_t t0 = xcd_contiguous_tile() * kPermTile;
    const int len = (int)min((int64_t)kPermTile, n - t0);
    const int tid = threadIdx.x;
    for (int b = 0; b < kPermPer; b += kPermBatch) {
        float v[kPermBatch];
#pragma unroll
        for (int u = 0; u < kPermBatch; ++u) {
            const int i = tid + (b + u) * kPermThreads;
            v[u] = i < len ? __builtin_nontemporal_load(src + t0 + i) : 0.f;
        }
#pragma unroll
        for (int u = 0; u < kPermBatch; ++u) tile[tid + (b + u) * kPermThreads] = v[u];
    }
    __syncthreads();
    for (int b = 0; b < kPermPer; b += kPermBatch) {
        int32_t st[kPermBatch];
        int loc[kPermBatch];
#pragma unroll
        for (int u = 0; u < kPermBatch; ++u) {
            const int o = tid + (b + u) * kPermThreads;
            st[u] = o < len ? __builtin_nontemporal_load(stage + t0 + o) : -1;
            loc[u] = o < len ? __builtin_nontemporal_load(src_local + t0 + o) : 0;
        }
#pragma unroll
        for (int u = 0; u < kPermBatch; ++u)
            if (st[u] >= 0) staging[st[u]] = tile[loc[u]];
    }
}

__global__ __launch_bounds__(kPermThreads) void perm_pass2_kernel(int64_t n,
                                                                  const float *staging,
                                                                  const uint16_t *dst_local,
                                                                  float *dst) {
    __shared__ float bucket[kPermTile];
    const int64_t d0 = (int64_t)blockIdx.x * kPermTile;
    const int len = (int)min((int64_t)kPermTile, n - d0);
    const int tid = threadIdx.x;
    for (int b = 0; b < kPermPer; b += kPermBatch) {
        float v[kPermBatch];
        int loc[kPermBatch];
#pragma unroll
        for (int u = 0; u < kPermBatch; ++u) {
            const int s = tid + (b + u) * kPermThreads;
            v[u] = s < len ? __builtin_nontemporal_load(staging + d0 + s) : 0.f;
            loc[u] = s < len ? __builtin_nontemporal_load(dst_local + d0 + s) : -1;
        }
#pragma unroll
        for (int u = 0; u < kPermBatch; ++u)
            if (loc[u] >= 0) bucket[loc[u]] = v[u];
    }
    __syncthreads();
    for (int b = 0; b < kPermPer; b += kPermBatch) {
#pragma unroll
        for (int u = 0; u < kPermBatch; ++u) {
            const int i = tid + (b + u) * kPermThreads;
            if (i < len) __builtin_nontemporal_store(bucket[i], dst + d0 + i);
        }
    }
}

// ------------------------------------------------------------- build

// key of every destination q: its source position perm[q]; after a stable
// sort by the destination bucket (q / T) the order is (bucket, source)
__global__ void perm_bucket_kernel(int64_t n, const int32_t *order, int32_t *bucket) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) bucket[i] = (int32_t)(order[i] / kPermTile);
}

// staging slot s holds destination q = order[s]: its local offset in the bucket,
// and (for pass 1) the tile of its source and the slot's position
__global__ void perm_stage_kernel(int64_t n, const int32_t *order, const int32_t *perm,
                                  uint16_t *dst_local, int32_t *src_tile, int32_t *src_pos) {
    const int64_t s = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (s >= n) return;
    const int32_t q = order[s];
    dst_local[s] = (uint16_t)(q % kPermTile);
    const int32_t p = perm[q];
    src_tile[s] = p / kPermTile;
    src_pos[s] = p;
}

// pass-1 output slot o (tile-major, stable: within a tile in staging order)
// holds staging slot s = by_tile[o]
__global__ void perm_pass1_plan_kernel(int64_t n, const int32_t *by_tile, const int32_t *src_pos,
                                       int32_t *stage, uint16_t *src_local) {
    const int64_t o = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (o >= n) return;
    const int32_t s = by_tile[o];
    stage[o] = s;
    src_local[o] = (uint16_t)(src_pos[s] % kPermTile);
}

__global__ void perm_invert_kernel(int64_t n, const int32_t *perm, int32_t *inv) {
    const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (q < n) inv[perm[q]] = (int32_t)q;
}

__global__ void perm_check_kernel(int64_t n, const int32_t *perm, int32_t *seen, int32_t *bad) {
    const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (q >= n) return;
    const int32_t p = perm[q];
    if (p < 0 || p >= n) atomicOr(bad, 1);
    else if (atomicExch(&seen[p], 1) != 0) atomicOr(bad, 2);
}

static size_t perm_build_ws(int64_t n) {
    Carver c(nullptr);
    for (int t = 0; t < 6; ++t) c.take<int32_t>(n > 0 ? n : 1);
    c.take<int32_t>(64);
    return c.bytes() + sort_ws_bytes(n, (int32_t)std::max<int64_t>(n, 1));
}

}  // namespace nsd

using namespace nsd;

extern "C" {

nsd_status nsd_perm_plan_workspace_size(int32_t n, size_t *bytes) {
    NSD_REQUIRE(bytes != nullptr, "bytes is NULL");
    NSD_REQUIRE(n >= 0, "negative length");
    *bytes = perm_build_ws(n);
    return NSD_OK;
}

nsd_status nsd_perm_plan_build(int32_t n, const int32_t *perm, int inverse, int32_t *stage,
                               uint16_t *src_local, uint16_t *dst_local, nsd_perm_plan *plan,
                               void *ws, size_t ws_bytes, void *stream) {
    NSD_REQUIRE(n >= 0 && plan != nullptr, "negative length or NULL plan");
    NSD_REQUIRE(n == 0 || (perm && stage && src_local && dst_local && ws), "null pointer");
    *plan = nsd_perm_plan{};
    plan->n = n;
    plan->tile = kPermTile;
    plan->stage = stage;
    plan->src_local = src_local;
    plan->dst_local = dst_local;
    if (n == 0) return NSD_OK;
    const size_t need = perm_build_ws(n);
    if (ws_bytes < need) return fail(NSD_ERR_WORKSPACE, "workspace %zu < %zu", ws_bytes, need);
    hipStream_t st = as_stream(stream);
    Carver c(ws);
    int32_t *a = c.take<int32_t>(n);
    int32_t *b = c.take<int32_t>(n);
    int32_t *e = c.take<int32_t>(n);
    int32_t *f = c.take<int32_t>(n);
    int32_t *g = c.take<int32_t>(n);
    int32_t *inv = c.take<int32_t>(n);
    int32_t *flag = c.take<int32_t>(64);
    void *sort_ws = c.base + c.bytes();
    const int64_t grid = ceil_div(n, 256);
    const int32_t ntiles = (int32_t)perm_tiles(n);

    // a permutation of [0, n): every value once
    NSD_HIP(hipMemsetAsync(a, 0, sizeof(int32_t) * (size_t)n, st));
    NSD_HIP(hipMemsetAsync(flag, 0, sizeof(int32_t), st));
    perm_check_kernel<<<grid, 256, 0, st>>>(n, perm, a, flag);
    NSD_TRY(check_launch("perm_check_kernel"));
    int32_t h = 0;
    NSD_HIP(hipMemcpyAsync(&h, flag, sizeof(int32_t), hipMemcpyDeviceToHost, st));
    NSD_HIP(hipStreamSynchronize(st));
    if (h) return fail(NSD_ERR_BAD_FORMAT, "not a permutation of [0, %d)", n);
    if (inverse) {  // dst[perm[q]] = src[q] is dst[p] = src[inv[p]]
        perm_invert_kernel<<<grid, 256, 0, st>>>(n, perm, inv);
        NSD_TRY(check_launch("perm_invert_kernel"));
        perm = inv;
    }

    // destinations in source order (a sort of q by perm[q]), then stably by
    // destination bucket: the staging order (bucket, source position)
    NSD_TRY(radix_sort_pairs(n, n, perm, nullptr, b, a, sort_ws, st));  // a: q by source
    perm_bucket_kernel<<<grid, 256, 0, st>>>(n, a, e);
    NSD_TRY(check_launch("perm_bucket_kernel"));
    NSD_TRY(radix_sort_pairs(n, ntiles, e, a, f, b, sort_ws, st));     // b: staging order
    perm_stage_kernel<<<grid, 256, 0, st>>>(n, b, perm, dst_local, e, g);
    NSD_TRY(check_launch("perm_stage_kernel"));
    // pass-1 slots: staging slots stably by their source tile
    NSD_TRY(radix_sort_pairs(n, ntiles, e, nullptr, f, a, sort_ws, st));  // a: s by tile
    perm_pass1_plan_kernel<<<grid, 256, 0, st>>>(n, a, g, stage, src_local);
    NSD_TRY(check_launch("perm_pass1_plan_kernel"));
    NSD_HIP(hipStreamSynchronize(st));
    return NSD_OK;
}

nsd_status nsd_permute_f32(const nsd_perm_plan *plan, const float *src, float *dst,
                           float *staging, void *stream) {
    NSD_REQUIRE(plan != nullptr, "plan is NULL");
    NSD_REQUIRE(plan->n >= 0, "negative length");
    if (plan->n == 0) return NSD_OK;
    NSD_REQUIRE(plan->tile == kPermTile, "plan built with tile %d, library uses %d", plan->tile,
                kPermTile);
    NSD_REQUIRE(plan->stage && plan->src_local && plan->dst_local, "plan is not built");
    NSD_REQUIRE(src && dst && staging, "null pointer");
    NSD_REQUIRE(src != dst, "src and dst must not alias");
    hipStream_t st = as_stream(stream);
    const unsigned nt = (unsigned)perm_tiles(plan->n);
    probe_begin(NSD_KERNEL_PERM, st);
    perm_pass1_kernel<<<nt, kPermThreads, 0, st>>>(plan->n, src, plan->stage, plan->src_local,
                                                   staging);
    NSD_TRY(check_launch("perm_pass1_kernel"));
    perm_pass2_kernel<<<nt, kPermThreads, 0, st>>>(plan->n, staging, plan->dst_local, dst);
    probe_end(NSD_KERNEL_PERM, st);
    return check_launch("perm_pass2_kernel");
}

}  // extern "C"
