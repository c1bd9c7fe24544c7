// Tensor-times-vector of a sparse 3-tensor along its third mode and its
// vector-Jacobian product:
//   Y(i, j) = sum over stored (i, j, l) of X_ijl * v(l)
// on the projected keys {(i, j) : some (i, j, l) is stored}; it is a sum over
// X's stored keys with a singleton {(i, j) -> X_ijl v(l)} added by "+=", so Y
// is itself sparse (Logical SDQLite, Section 3; code generation, Section 5.5).
// Given the upstream gY on Y's keys:
//   dX_ijl = gY(i, j) v(l)                 on X's keys (input order)
//   dv(l)  = sum over stored (i, j, l) of X_ijl gY(i, j)
//
// The builder stably sorts X's entries by (i, j) (two counting-sort passes),
// numbers the distinct keys, and also sorts by l (a mode index); both views
// get a work plan, so the forward product and dv are k = 1 gather-reduces
// and dX is one elementwise pass.
#include <algorithm>

#include "nsd_internal.hpp"
#include "segreduce.hpp"

namespace nsd {

constexpr int kTtvThreads = 256;

static int64_t ttv_grid(int64_t n) { return ceil_div(n > 0 ? n : 1, kTtvThreads); }

__global__ void ttv_gather_kernel(int64_t n, const int32_t *perm, const int32_t *src,
                                  int32_t *dst) {
    const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (q < n) dst[q] = src[perm[q]];
}

__global__ void ttv_heads_kernel(int64_t n, const int32_t *a, const int32_t *b, int32_t *head) {
    const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (q < n) head[q] = (q == 0 || a[q] != a[q - 1] || b[q] != b[q - 1]) ? 1 : 0;
}

// seg = inclusive count of heads - 1; the head of every key writes it out;
// pair (input order) gets every entry's key index.
__global__ void ttv_keys_kernel(int64_t n, const int32_t *head, const int32_t *pos,
                                const int32_t *i_s, const int32_t *j_s, const int32_t *perm,
                                int32_t *seg, int32_t *yi, int32_t *yj, int32_t *pair) {
    const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (q >= n) return;
    const int32_t s = pos[q] + head[q] - 1;
    seg[q] = s;
    pair[perm[q]] = s;
    if (head[q]) {
        yi[s] = i_s[q];
        yj[s] = j_s[q];
    }
}

__global__ void ttv_range_kernel(int64_t n, int32_t d0, int32_t d1, int32_t d2, const int32_t *i,
                                 const int32_t *j, const int32_t *l, int32_t *flag) {
    const int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (p >= n) return;
    if (i[p] < 0 || i[p] >= d0 || j[p] < 0 || j[p] >= d1 || l[p] < 0 || l[p] >= d2)
        atomicOr(flag, 1);
}

__global__ void ttv_dx_kernel(int64_t n, const int32_t *seg, const int32_t *perm,
                              const int32_t *kidx, const float *gy, const float *v, float *dx) {
    const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (q < n) dx[perm[q]] = gy[seg[q]] * v[kidx[q]];
}

static size_t ttv_build_ws(int64_t nnz, int32_t maxdim) {
    Carver c(nullptr);
    for (int t = 0; t < 6; ++t) c.take<int32_t>(nnz > 0 ? nnz : 1);
    c.take<int32_t>(64);
    return c.bytes() + sort_ws_bytes(nnz, maxdim) + scan_ws_bytes(nnz);
}

static nsd_status check_ttv(const nsd_ttv_plan *T) {
    NSD_REQUIRE(T != nullptr, "TTV plan is NULL");
    NSD_REQUIRE(T->nnz >= 0 && T->ny >= 0 && T->dims[2] >= 1, "bad TTV plan sizes");
    if (T->nnz > 0) {
        NSD_REQUIRE(T->yptr && T->yseg && T->yperm && T->ykidx && T->lptr && T->lseg &&
                        T->lperm && T->lpair,
                    "TTV plan array is NULL");
        NSD_REQUIRE(T->yplan.item_ptr && T->yplan.nitems >= 1 && T->lplan.item_ptr &&
                        T->lplan.nitems >= 1,
                    "TTV work plans are not built (nsd_plan_build)");
    }
    return NSD_OK;
}

static size_t ttv_ws(const nsd_ttv_plan *T) {
    const size_t a = sgr_part_bytes(T->yplan, 1), b = sgr_part_bytes(T->lplan, 1);
    return ((std::max(a, b) + 255) & ~size_t(255));
}

static SgrParams ttv_sgr(int32_t nseg, int32_t nnz, const nsd_plan &plan, const int32_t *segptr,
                         const int32_t *segidx, const int32_t *idx, const float *w,
                         const int32_t *wperm, const float *X, float *out, void *ws,
                         int32_t k = 1) {
    SgrParams p;
    p.nseg = nseg;
    p.nnz = nnz;
    p.k = k;
    p.plan = plan;
    p.segptr = segptr;
    p.segidx = segidx;
    p.idx = idx;
    p.w = w;
    p.wperm = wperm;
    p.X = X;
    p.out = out;
    p.part = static_cast<float *>(ws);
    return p;
}

static size_t ttm_ws(const nsd_ttv_plan *T, int32_t R) {
    const size_t a = sgr_part_bytes(T->yplan, R), b = sgr_part_bytes(T->lplan, R);
    return ((std::max(a, b) + 255) & ~size_t(255));
}

}  // namespace nsd

using namespace nsd;

extern "C" {

nsd_status nsd_ttv_build_workspace_size(int32_t nnz, const int32_t *dims, size_t *bytes) {
    NSD_REQUIRE(dims && bytes, "null pointer");
    NSD_REQUIRE(nnz >= 0 && dims[0] >= 1 && dims[1] >= 1 && dims[2] >= 1, "bad sizes");
    *bytes = ttv_build_ws(nnz, std::max({dims[0], dims[1], dims[2]}));
    return NSD_OK;
}

nsd_status nsd_ttv_build(int32_t nnz, const int32_t *dims, const int32_t *i, const int32_t *j,
                         const int32_t *l, int32_t *yi, int32_t *yj, int32_t *yptr,
                         int32_t *yseg, int32_t *yperm, int32_t *ykidx, int32_t *lptr,
                         int32_t *lseg, int32_t *lperm, int32_t *lpair, int32_t *ny,
                         void *ws, size_t ws_bytes, void *stream) {
    NSD_REQUIRE(dims && ny && yptr && lptr, "null pointer");
    NSD_REQUIRE(nnz >= 0 && dims[0] >= 1 && dims[1] >= 1 && dims[2] >= 1, "bad sizes");
    hipStream_t st = as_stream(stream);
    if (nnz == 0) {
        NSD_TRY(segptr_from_sorted(0, 0, yseg, yptr, st));
        NSD_TRY(segptr_from_sorted(0, dims[2], lseg, lptr, st));
        NSD_HIP(hipStreamSynchronize(st));
        *ny = 0;
        return NSD_OK;
    }
    NSD_REQUIRE(i && j && l && yi && yj && yseg && yperm && ykidx && lseg && lperm && lpair && ws,
                "null pointer");
    const int32_t maxdim = std::max({dims[0], dims[1], dims[2]});
    if (ws_bytes < ttv_build_ws(nnz, maxdim))
        return fail(NSD_ERR_WORKSPACE, "workspace %zu < %zu", ws_bytes, ttv_build_ws(nnz, maxdim));
    Carver c(ws);
    int32_t *t0 = c.take<int32_t>(nnz);
    int32_t *t1 = c.take<int32_t>(nnz);
    int32_t *t2 = c.take<int32_t>(nnz);
    int32_t *t3 = c.take<int32_t>(nnz);
    int32_t *head = c.take<int32_t>(nnz);
    int32_t *pair = c.take<int32_t>(nnz);
    int32_t *flag = c.take<int32_t>(64);
    void *sort_ws = c.base + c.bytes();
    void *scan_ws = static_cast<char *>(sort_ws) + sort_ws_bytes(nnz, maxdim);
    const int64_t g = ttv_grid(nnz);

    NSD_HIP(hipMemsetAsync(flag, 0, sizeof(int32_t), st));
    ttv_range_kernel<<<g, kTtvThreads, 0, st>>>(nnz, dims[0], dims[1], dims[2], i, j, l, flag);
    NSD_TRY(check_launch("ttv_range_kernel"));
    int32_t h = 0;
    NSD_HIP(hipMemcpyAsync(&h, flag, sizeof(int32_t), hipMemcpyDeviceToHost, st));
    NSD_HIP(hipStreamSynchronize(st));
    if (h) return fail(NSD_ERR_BAD_FORMAT, "coordinate out of range");

    // (i, j) order: stable by j, then stable by i; ties keep input order
    NSD_TRY(radix_sort_pairs(nnz, dims[1], j, nullptr, t0, t1, sort_ws, st));
    ttv_gather_kernel<<<g, kTtvThreads, 0, st>>>(nnz, t1, i, t2);
    NSD_TRY(check_launch("ttv_gather_kernel"));
    NSD_TRY(radix_sort_pairs(nnz, dims[0], t2, t1, t3, yperm, sort_ws, st));  // t3 = i sorted
    ttv_gather_kernel<<<g, kTtvThreads, 0, st>>>(nnz, yperm, j, t0);          // t0 = j sorted
    ttv_gather_kernel<<<g, kTtvThreads, 0, st>>>(nnz, yperm, l, ykidx);
    ttv_heads_kernel<<<g, kTtvThreads, 0, st>>>(nnz, t3, t0, head);
    NSD_TRY(check_launch("ttv_heads_kernel"));
    NSD_TRY(scan_exclusive(head, t2, nnz, flag + 1, scan_ws, st));
    ttv_keys_kernel<<<g, kTtvThreads, 0, st>>>(nnz, head, t2, t3, t0, yperm, yseg, yi, yj, pair);
    NSD_TRY(check_launch("ttv_keys_kernel"));
    int32_t nkeys = 0;
    NSD_HIP(hipMemcpyAsync(&nkeys, flag + 1, sizeof(int32_t), hipMemcpyDeviceToHost, st));
    NSD_HIP(hipStreamSynchronize(st));
    NSD_TRY(segptr_from_sorted(nnz, nkeys, yseg, yptr, st));
    // l order
    NSD_TRY(radix_sort_pairs(nnz, dims[2], l, nullptr, lseg, lperm, sort_ws, st));
    NSD_TRY(segptr_from_sorted(nnz, dims[2], lseg, lptr, st));
    ttv_gather_kernel<<<g, kTtvThreads, 0, st>>>(nnz, lperm, pair, lpair);
    NSD_TRY(check_launch("ttv_gather_kernel"));
    NSD_HIP(hipStreamSynchronize(st));
    *ny = nkeys;
    return NSD_OK;
}

nsd_status nsd_ttv_workspace_size(const nsd_ttv_plan *T, size_t *bytes) {
    NSD_REQUIRE(bytes != nullptr, "bytes is NULL");
    NSD_TRY(check_ttv(T));
    *bytes = ttv_ws(T);
    return NSD_OK;
}

nsd_status nsd_ttv(const nsd_ttv_plan *T, const float *x, const float *v, float *y, void *ws,
                   size_t ws_bytes, void *stream) {
    NSD_TRY(check_ttv(T));
    NSD_REQUIRE(T->nnz == 0 || (x && v && y), "null pointer");
    if (ws == nullptr || ws_bytes < ttv_ws(T))
        return fail(NSD_ERR_WORKSPACE, "workspace %zu < %zu", ws_bytes, ttv_ws(T));
    if (T->ny == 0) return NSD_OK;
    hipStream_t st = as_stream(stream);
    probe_begin(NSD_KERNEL_TTV, st);
    const nsd_status s = segreduce(ttv_sgr(T->ny, T->nnz, T->yplan, T->yptr, T->yseg, T->ykidx, x,
                                           T->yperm, v, y, ws),
                                   st);
    probe_end(NSD_KERNEL_TTV, st);
    return s;
}

nsd_status nsd_ttv_vjp(const nsd_ttv_plan *T, const float *x, const float *v, const float *gy,
                       float *dx, float *dv, void *ws, size_t ws_bytes, void *stream) {
    NSD_TRY(check_ttv(T));
    NSD_REQUIRE(dv != nullptr, "dv is NULL");
    NSD_REQUIRE(T->nnz == 0 || (x && v && gy && dx), "null pointer");
    if (ws == nullptr || ws_bytes < ttv_ws(T))
        return fail(NSD_ERR_WORKSPACE, "workspace %zu < %zu", ws_bytes, ttv_ws(T));
    hipStream_t st = as_stream(stream);
    if (T->nnz > 0) {
        probe_begin(NSD_KERNEL_TTV, st);
        ttv_dx_kernel<<<ttv_grid(T->nnz), kTtvThreads, 0, st>>>(T->nnz, T->yseg, T->yperm,
                                                                T->ykidx, gy, v, dx);
        probe_end(NSD_KERNEL_TTV, st);
        NSD_TRY(check_launch("ttv_dx_kernel"));
    }
    return segreduce(ttv_sgr(T->dims[2], T->nnz, T->lplan, T->lptr, T->lseg, T->lpair, x, T->lperm,
                             gy, dv, ws),
                     st);
}

nsd_status nsd_ttm_workspace_size(const nsd_ttv_plan *T, int32_t R, size_t *bytes) {
    NSD_REQUIRE(bytes != nullptr, "bytes is NULL");
    NSD_TRY(check_ttv(T));
    NSD_REQUIRE(R >= 1, "R = %d < 1", R);
    *bytes = ttm_ws(T, R);
    return NSD_OK;
}

// Y = X x_3 U: the gather-reduce of TTV at width R (rows U[l] weighted by x).
nsd_status nsd_ttm(const nsd_ttv_plan *T, const float *x, const float *U, int32_t R, float *Y,
                   void *ws, size_t ws_bytes, void *stream) {
    NSD_TRY(check_ttv(T));
    NSD_REQUIRE(R >= 1, "R = %d < 1", R);
    NSD_REQUIRE(T->nnz == 0 || (x && U && Y), "null pointer");
    if (ws == nullptr || ws_bytes < ttm_ws(T, R))
        return fail(NSD_ERR_WORKSPACE, "workspace %zu < %zu", ws_bytes, ttm_ws(T, R));
    if (T->ny == 0) return NSD_OK;
    hipStream_t st = as_stream(stream);
    probe_begin(NSD_KERNEL_TTV, st);
    const nsd_status s = segreduce(ttv_sgr(T->ny, T->nnz, T->yplan, T->yptr, T->yseg, T->ykidx, x,
                                           T->yperm, U, Y, ws, R),
                                   st);
    probe_end(NSD_KERNEL_TTV, st);
    return s;
}

// dx = <gY[key], U[l]> per entry (an SDDMM in (i, j) order written to input
// positions), dU = the gather-reduce over l of x * gY[key].
nsd_status nsd_ttm_vjp(const nsd_ttv_plan *T, const float *x, const float *U, int32_t R,
                       const float *gY, float *dx, float *dU, void *ws, size_t ws_bytes,
                       void *stream) {
    NSD_TRY(check_ttv(T));
    NSD_REQUIRE(R >= 1, "R = %d < 1", R);
    NSD_REQUIRE(dU != nullptr, "dU is NULL");
    NSD_REQUIRE(T->nnz == 0 || (x && U && gY && dx), "null pointer");
    if (ws == nullptr || ws_bytes < ttm_ws(T, R))
        return fail(NSD_ERR_WORKSPACE, "workspace %zu < %zu", ws_bytes, ttm_ws(T, R));
    hipStream_t st = as_stream(stream);
    if (T->nnz > 0) {
        SddmmParams sp;
        sp.nnz = T->nnz;
        sp.k = R;
        sp.rowidx = T->yseg;
        sp.colind = T->ykidx;
        sp.X = gY;
        sp.Y = U;
        sp.out = dx;
        sp.operm = T->yperm;
        probe_begin(NSD_KERNEL_TTV, st);
        const nsd_status s = sddmm(sp, st);
        probe_end(NSD_KERNEL_TTV, st);
        NSD_TRY(s);
    }
    return segreduce(ttv_sgr(T->dims[2], T->nnz, T->lplan, T->lptr, T->lseg, T->lpair, x, T->lperm,
                             gY, dU, ws, R),
                     st);
}

}  // extern "C"
