// Mode-n products of a sparse order-N tensor and their vector-Jacobian
// products:
//   Y(c_{-n}) = sum over stored keys c of X(c) * v(c_n)        (TTV)
//   Y(c_{-n}, :) = sum over stored keys c of X(c) * U(c_n, :)  (TTM)
// on the projected keys {c_{-n} : some key c is stored}, c_{-n} being the key
// with coordinate n dropped; Y is a sum over X's stored keys with a
// singleton added by "+=", so it is itself sparse (Logical SDQLite,
// Section 3; code generation, Section 5.5).  Given the upstream gY on Y's
// keys:
//   dX(c) = <gY(c_{-n}), U(c_n)>              on X's keys (input order)
//   dU(l) = sum over stored keys with c_n = l of X(c) gY(c_{-n})
//
// The builder stably sorts X's entries by their other coordinates (one
// counting-sort pass per mode, last mode first), numbers the distinct keys,
// and also sorts by the mode-n coordinate; both views get a work plan, so the
// products and dU are gather-reduces and dX is one sampled product.
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

// The key-sorted coordinates of the modes other than n (up to 5 arrays).
struct KeyCols {
    const int32_t *c[NSD_MAX_ORDER - 1];
    int32_t n;
};

__global__ void ttv_heads_kernel(int64_t n, KeyCols k, int32_t *head) {
    const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (q >= n) return;
    bool h = q == 0;
    for (int o = 0; o < k.n && !h; ++o) h = k.c[o][q] != k.c[o][q - 1];
    head[q] = h ? 1 : 0;
}

struct KeyOut {
    int32_t *c[NSD_MAX_ORDER - 1];
};

// seg = inclusive count of heads - 1; the head of every key writes its
// coordinates; pair (input order) gets every entry's key index.
__global__ void ttv_keys_kernel(int64_t n, const int32_t *head, const int32_t *pos, KeyCols k,
                                const int32_t *perm, int32_t *seg, KeyOut y, int32_t *pair) {
    const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (q >= n) return;
    const int32_t s = pos[q] + head[q] - 1;
    seg[q] = s;
    pair[perm[q]] = s;
    if (head[q])
        for (int o = 0; o < k.n; ++o) y.c[o][s] = k.c[o][q];
}

__global__ void ttv_range_kernel(int64_t n, int32_t dim, const int32_t *c, int32_t *flag) {
    const int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (p < n && (c[p] < 0 || c[p] >= dim)) atomicOr(flag, 1);
}

__global__ void ttv_dx_kernel(int64_t n, const int32_t *seg, const int32_t *perm,
                              const int32_t *kidx, const float *gy, const float *v, float *dx) {
    const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (q < n) dx[perm[q]] = gy[seg[q]] * v[kidx[q]];
}

// Scratch of the builder: the N - 1 key-sorted coordinate arrays, two
// permutations, the head flags, the key of every entry and a flag word.
static size_t ttv_build_ws(int32_t order, int64_t nnz, int32_t maxdim) {
    Carver c(nullptr);
    for (int t = 0; t < order - 1 + 4; ++t) c.take<int32_t>(nnz > 0 ? nnz : 1);
    c.take<int32_t>(64);
    return c.bytes() + sort_ws_bytes(nnz, maxdim) + scan_ws_bytes(nnz);
}

static nsd_status check_ttv(const nsd_ttv_plan *T) {
    NSD_REQUIRE(T != nullptr, "TTV plan is NULL");
    NSD_REQUIRE(T->order >= 3 && T->order <= NSD_MAX_ORDER && T->mode >= 0 &&
                    T->mode < T->order,
                "TTV plan of order %d along mode %d", T->order, T->mode);
    NSD_REQUIRE(T->nnz >= 0 && T->ny >= 0 && T->dims[T->mode] >= 1, "bad TTV plan sizes");
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

static nsd_status check_build_sizes(int32_t order, const int32_t *dims, int32_t nnz) {
    NSD_REQUIRE(dims != nullptr, "dims is NULL");
    NSD_REQUIRE(order >= 3 && order <= NSD_MAX_ORDER, "order %d outside [3, %d]", order,
                NSD_MAX_ORDER);
    NSD_REQUIRE(nnz >= 0, "negative nnz");
    for (int m = 0; m < order; ++m) NSD_REQUIRE(dims[m] >= 1, "dims[%d] = %d < 1", m, dims[m]);
    return NSD_OK;
}

nsd_status nsd_ttv_build_workspace_size(int32_t order, const int32_t *dims, int32_t nnz,
                                        size_t *bytes) {
    NSD_REQUIRE(bytes != nullptr, "bytes is NULL");
    NSD_TRY(check_build_sizes(order, dims, nnz));
    *bytes = ttv_build_ws(order, nnz, *std::max_element(dims, dims + order));
    return NSD_OK;
}

nsd_status nsd_ttv_build(int32_t order, const int32_t *dims, int32_t nnz,
                         const int32_t *const *coords, int32_t mode, int32_t *const *ykey,
                         int32_t *yptr, int32_t *yseg, int32_t *yperm, int32_t *ykidx,
                         int32_t *lptr, int32_t *lseg, int32_t *lperm, int32_t *lpair,
                         int32_t *ny, void *ws, size_t ws_bytes, void *stream) {
    NSD_TRY(check_build_sizes(order, dims, nnz));
    NSD_REQUIRE(mode >= 0 && mode < order, "mode %d of an order-%d tensor", mode, order);
    NSD_REQUIRE(ny && yptr && lptr, "null pointer");
    hipStream_t st = as_stream(stream);
    if (nnz == 0) {
        NSD_TRY(segptr_from_sorted(0, 0, yseg, yptr, st));
        NSD_TRY(segptr_from_sorted(0, dims[mode], lseg, lptr, st));
        NSD_HIP(hipStreamSynchronize(st));
        *ny = 0;
        return NSD_OK;
    }
    NSD_REQUIRE(coords && ykey && yseg && yperm && ykidx && lseg && lperm && lpair && ws,
                "null pointer");
    int others[NSD_MAX_ORDER - 1];
    for (int m = 0, o = 0; m < order; ++m) {
        NSD_REQUIRE(coords[m] != nullptr, "coordinate array %d is NULL", m);
        if (m != mode) {
            NSD_REQUIRE(ykey[o] != nullptr, "key array %d is NULL", o);
            others[o++] = m;
        }
    }
    const int nk = order - 1;
    const int32_t maxdim = *std::max_element(dims, dims + order);
    const size_t need = ttv_build_ws(order, nnz, maxdim);
    if (ws_bytes < need) return fail(NSD_ERR_WORKSPACE, "workspace %zu < %zu", ws_bytes, need);
    Carver c(ws);
    KeyCols kc;
    kc.n = nk;
    int32_t *sorted[NSD_MAX_ORDER - 1];
    for (int o = 0; o < nk; ++o) kc.c[o] = sorted[o] = c.take<int32_t>(nnz);
    int32_t *pa = c.take<int32_t>(nnz);
    int32_t *pb = c.take<int32_t>(nnz);
    int32_t *head = c.take<int32_t>(nnz);
    int32_t *pair = c.take<int32_t>(nnz);
    int32_t *flag = c.take<int32_t>(64);
    void *sort_ws = c.base + c.bytes();
    void *scan_ws = static_cast<char *>(sort_ws) + sort_ws_bytes(nnz, maxdim);
    const int64_t g = ttv_grid(nnz);

    NSD_HIP(hipMemsetAsync(flag, 0, sizeof(int32_t), st));
    for (int m = 0; m < order; ++m) {
        ttv_range_kernel<<<g, kTtvThreads, 0, st>>>(nnz, dims[m], coords[m], flag);
        NSD_TRY(check_launch("ttv_range_kernel"));
    }
    int32_t h = 0;
    NSD_HIP(hipMemcpyAsync(&h, flag, sizeof(int32_t), hipMemcpyDeviceToHost, st));
    NSD_HIP(hipStreamSynchronize(st));
    if (h) return fail(NSD_ERR_BAD_FORMAT, "coordinate out of range");

    // lexicographic order of the other coordinates: stable passes from the
    // last other mode to the first; ties keep input order.  perm ends in
    // yperm, each pass's sorted keys in a scratch array.
    int32_t *perm = nullptr;  // identity before the first pass
    for (int o = nk - 1; o >= 0; --o) {
        const int m = others[o];
        const int32_t *key = coords[m];
        if (perm) {
            ttv_gather_kernel<<<g, kTtvThreads, 0, st>>>(nnz, perm, coords[m], head);
            NSD_TRY(check_launch("ttv_gather_kernel"));
            key = head;
        }
        int32_t *out = o == 0 ? yperm : (perm == pa ? pb : pa);
        NSD_TRY(radix_sort_pairs(nnz, dims[m], key, perm, sorted[o], out, sort_ws, st));
        perm = out;
    }
    // the key-sorted coordinates of the other modes, and l
    for (int o = 1; o < nk; ++o) {
        ttv_gather_kernel<<<g, kTtvThreads, 0, st>>>(nnz, yperm, coords[others[o]], sorted[o]);
        NSD_TRY(check_launch("ttv_gather_kernel"));
    }
    ttv_gather_kernel<<<g, kTtvThreads, 0, st>>>(nnz, yperm, coords[mode], ykidx);
    NSD_TRY(check_launch("ttv_gather_kernel"));
    ttv_heads_kernel<<<g, kTtvThreads, 0, st>>>(nnz, kc, head);
    NSD_TRY(check_launch("ttv_heads_kernel"));
    NSD_TRY(scan_exclusive(head, pa, nnz, flag + 1, scan_ws, st));
    KeyOut yo;
    for (int o = 0; o < nk; ++o) yo.c[o] = ykey[o];
    ttv_keys_kernel<<<g, kTtvThreads, 0, st>>>(nnz, head, pa, kc, yperm, yseg, yo, pair);
    NSD_TRY(check_launch("ttv_keys_kernel"));
    int32_t nkeys = 0;
    NSD_HIP(hipMemcpyAsync(&nkeys, flag + 1, sizeof(int32_t), hipMemcpyDeviceToHost, st));
    NSD_HIP(hipStreamSynchronize(st));
    NSD_TRY(segptr_from_sorted(nnz, nkeys, yseg, yptr, st));
    // mode-n order
    NSD_TRY(radix_sort_pairs(nnz, dims[mode], coords[mode], nullptr, lseg, lperm, sort_ws, st));
    NSD_TRY(segptr_from_sorted(nnz, dims[mode], lseg, lptr, st));
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
    return segreduce(ttv_sgr(T->dims[T->mode], T->nnz, T->lplan, T->lptr, T->lseg, T->lpair, x,
                             T->lperm, gy, dv, ws),
                     st);
}

nsd_status nsd_ttm_workspace_size(const nsd_ttv_plan *T, int32_t R, size_t *bytes) {
    NSD_REQUIRE(bytes != nullptr, "bytes is NULL");
    NSD_TRY(check_ttv(T));
    NSD_REQUIRE(R >= 1, "R = %d < 1", R);
    *bytes = ttm_ws(T, R);
    return NSD_OK;
}

// Y = X x_n U: the gather-reduce of TTV at width R (rows U[l] weighted by x).
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

// dx = <gY[key], U[l]> per entry (an SDDMM in key order written to input
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
    return segreduce(ttv_sgr(T->dims[T->mode], T->nnz, T->lplan, T->lptr, T->lseg, T->lpair, x,
                             T->lperm, gY, dU, ws, R),
                     st);
}

}  // extern "C"
