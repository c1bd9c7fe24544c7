// Hot-path entry points: forward products, VJP primitives and the fused
// loss + gradient calls.  Each one validates its arguments on the host, then
// enqueues kernels on the caller's stream and returns without waiting.
#include <algorithm>

#include "nsd_internal.hpp"
#include "segreduce.hpp"

namespace nsd {

static nsd_status check_csr(const nsd_csr *A, bool need_val) {
    NSD_REQUIRE(A != nullptr, "CSR descriptor is NULL");
    NSD_REQUIRE(A->nrows >= 0 && A->ncols >= 0 && A->nnz >= 0, "negative CSR size");
    NSD_REQUIRE(A->rowptr != nullptr, "CSR rowptr is NULL");
    if (A->nnz > 0) {
        NSD_REQUIRE(A->nrows > 0 && A->ncols > 0, "nnz > 0 in an empty shape");
        NSD_REQUIRE(A->rowidx && A->colind, "CSR rowidx/colind is NULL");
        NSD_REQUIRE(!need_val || A->val, "CSR val is NULL");
    }
    return NSD_OK;
}

static nsd_status check_csc(const nsd_csc *At, const nsd_csr *A) {
    NSD_REQUIRE(At != nullptr, "CSC descriptor is NULL");
    NSD_REQUIRE(At->nrows == A->nrows && At->ncols == A->ncols && At->nnz == A->nnz,
                "CSC shape (%d x %d, %d) differs from CSR (%d x %d, %d)", At->nrows, At->ncols,
                At->nnz, A->nrows, A->ncols, A->nnz);
    NSD_REQUIRE(At->colptr != nullptr, "CSC colptr is NULL");
    if (At->nnz > 0) NSD_REQUIRE(At->colidx && At->rowind && At->perm, "CSC array is NULL");
    return NSD_OK;
}

// Workspace: one gather-reduce carry region (reused by every reduction of a
// call, which run in stream order) followed by the loss partials.
static size_t sgr_region_bytes(int64_t nnz, int k) {
    size_t best = 0;
    for (int kk : {k, 1}) {
        Carver c(nullptr);
        sgr_carve(c, nnz, kk, nullptr);
        best = std::max(best, c.bytes());
    }
    return best;
}

static size_t part_count(int64_t nnz, int k) {
    int64_t m = 1;
    for (int kk : {k, 1})
        for (bool v : {true, false}) m = std::max(m, sddmm_shape(nnz, kk, v).nblocks);
    return (size_t)m;
}

static size_t compute_ws_bytes(int64_t nnz, int k) {
    return sgr_region_bytes(nnz, k) + ((part_count(nnz, k) * sizeof(double) + 255) & ~size_t(255));
}

struct ComputeWs {
    void *sgr;
    double *part;
};

static nsd_status carve_compute(void *ws, size_t ws_bytes, int64_t nnz, int k, ComputeWs *out) {
    const size_t need = compute_ws_bytes(nnz, k);
    if (ws == nullptr || ws_bytes < need)
        return fail(NSD_ERR_WORKSPACE, "workspace %zu bytes at %p, need %zu", ws_bytes, ws, need);
    out->sgr = ws;
    out->part = reinterpret_cast<double *>(static_cast<char *>(ws) + sgr_region_bytes(nnz, k));
    return NSD_OK;
}

static SgrParams rows_params(const nsd_csr *A, const float *X, int k, float alpha, float *out,
                             void *region) {
    SgrParams p;
    p.nseg = A->nrows;
    p.nnz = A->nnz;
    p.k = k;
    p.segptr = A->rowptr;
    p.segidx = A->rowidx;
    p.idx = A->colind;
    p.w = A->val;
    p.X = X;
    p.alpha = alpha;
    p.out = out;
    Carver c(region);
    sgr_carve(c, A->nnz, k, &p);
    return p;
}

static SgrParams cols_params(const nsd_csr *A, const nsd_csc *At, const float *G, int k,
                             float alpha, float *out, void *region) {
    SgrParams p;
    p.nseg = A->ncols;
    p.nnz = A->nnz;
    p.k = k;
    p.segptr = At->colptr;
    p.segidx = At->colidx;
    p.idx = At->rowind;
    p.w = A->val;
    p.wperm = At->perm;
    p.X = G;
    p.alpha = alpha;
    p.out = out;
    Carver c(region);
    sgr_carve(c, A->nnz, k, &p);
    return p;
}

static SddmmParams sddmm_params(const nsd_csr *A, const float *X, const float *Y, int k,
                                float alpha, float *out) {
    SddmmParams p;
    p.nnz = A->nnz;
    p.k = k;
    p.rowidx = A->rowidx;
    p.colind = A->colind;
    p.X = X;
    p.Y = Y;
    p.alpha = alpha;
    p.out = out;
    return p;
}

// The loss partial count of a fused SDDMM; with nnz == 0 the loss is 0.
static nsd_status finish_loss(const SddmmParams &p, double *loss, hipStream_t st) {
    // with nnz == 0 there are no partials and the finaliser writes 0
    return loss_finalize(p.part, sddmm_shape(p.nnz, p.k, sddmm_vec_ok(p)).nblocks, loss, st);
}

}  // namespace nsd

using namespace nsd;

extern "C" {

nsd_status nsd_workspace_size(int32_t nnz, int32_t nseg, int32_t k, size_t *bytes) {
    NSD_REQUIRE(bytes != nullptr, "bytes is NULL");
    NSD_REQUIRE(nnz >= 0 && nseg >= 0 && k >= 1, "need nnz >= 0, nseg >= 0, k >= 1");
    *bytes = compute_ws_bytes(nnz, k);
    return NSD_OK;
}

nsd_status nsd_spmv(const nsd_csr *A, const float *x, float *y, void *ws, size_t ws_bytes,
                    void *stream) {
    NSD_TRY(check_csr(A, true));
    NSD_REQUIRE(A->nrows == 0 || y != nullptr, "y is NULL");
    NSD_REQUIRE(A->nnz == 0 || x != nullptr, "x is NULL");
    ComputeWs w;
    NSD_TRY(carve_compute(ws, ws_bytes, A->nnz, 1, &w));
    return segreduce(rows_params(A, x, 1, 1.f, y, w.sgr), as_stream(stream));
}

nsd_status nsd_spmm(const nsd_csr *A, const float *B, int32_t k, float *C, void *ws,
                    size_t ws_bytes, void *stream) {
    NSD_TRY(check_csr(A, true));
    NSD_REQUIRE(k >= 1, "k = %d < 1", k);
    NSD_REQUIRE(A->nrows == 0 || C != nullptr, "C is NULL");
    NSD_REQUIRE(A->nnz == 0 || B != nullptr, "B is NULL");
    ComputeWs w;
    NSD_TRY(carve_compute(ws, ws_bytes, A->nnz, k, &w));
    return segreduce(rows_params(A, B, k, 1.f, C, w.sgr), as_stream(stream));
}

nsd_status nsd_sddmm(const nsd_csr *A, const float *X, const float *Y, int32_t k, float alpha,
                     float *out, void *stream) {
    NSD_TRY(check_csr(A, false));
    NSD_REQUIRE(k >= 1, "k = %d < 1", k);
    NSD_REQUIRE(A->nnz == 0 || (Y != nullptr && out != nullptr), "Y/out is NULL");
    return sddmm(sddmm_params(A, X, Y, k, alpha, out), as_stream(stream));
}

nsd_status nsd_spmm_t(const nsd_csr *A, const nsd_csc *At, const float *G, int32_t k,
                      float alpha, float *out, void *ws, size_t ws_bytes, void *stream) {
    NSD_TRY(check_csr(A, true));
    NSD_TRY(check_csc(At, A));
    NSD_REQUIRE(k >= 1, "k = %d < 1", k);
    NSD_REQUIRE(A->ncols == 0 || out != nullptr, "out is NULL");
    ComputeWs w;
    NSD_TRY(carve_compute(ws, ws_bytes, A->nnz, k, &w));
    return segreduce(cols_params(A, At, G, k, alpha, out, w.sgr), as_stream(stream));
}

nsd_status nsd_loss_sum_spmv(const nsd_csr *A, const nsd_csc *At, const float *x, float seed,
                             double *loss, float *dA, float *dx, void *ws, size_t ws_bytes,
                             void *stream) {
    NSD_TRY(check_csr(A, true));
    NSD_TRY(check_csc(At, A));
    NSD_REQUIRE(loss != nullptr, "loss is NULL");
    NSD_REQUIRE(A->nnz == 0 || (x && dA), "x/dA is NULL");
    NSD_REQUIRE(A->ncols == 0 || dx != nullptr, "dx is NULL");
    ComputeWs w;
    NSD_TRY(carve_compute(ws, ws_bytes, A->nnz, 1, &w));
    hipStream_t st = as_stream(stream);
    // dA[p] = seed * x[col]; loss = sum_p A_p * x[col]
    SddmmParams sp = sddmm_params(A, nullptr, x, 1, seed, dA);
    sp.w = A->val;
    sp.beta = 1.0;
    sp.part = w.part;
    NSD_TRY(sddmm(sp, st));
    NSD_TRY(finish_loss(sp, loss, st));
    // dx = seed * A^T 1
    return segreduce(cols_params(A, At, nullptr, 1, seed, dx, w.sgr), st);
}

nsd_status nsd_loss_frob_spmm(const nsd_csr *A, const nsd_csc *At, const float *B, int32_t k,
                              float seed, float *C, double *loss, float *dA, float *dB,
                              void *ws, size_t ws_bytes, void *stream) {
    NSD_TRY(check_csr(A, true));
    NSD_TRY(check_csc(At, A));
    NSD_REQUIRE(k >= 1, "k = %d < 1", k);
    NSD_REQUIRE(loss != nullptr, "loss is NULL");
    NSD_REQUIRE(A->nrows == 0 || C != nullptr, "C is NULL");
    NSD_REQUIRE(A->ncols == 0 || dB != nullptr, "dB is NULL");
    NSD_REQUIRE(A->nnz == 0 || (B && dA), "B/dA is NULL");
    ComputeWs w;
    NSD_TRY(carve_compute(ws, ws_bytes, A->nnz, k, &w));
    hipStream_t st = as_stream(stream);
    // forward: C = A B
    NSD_TRY(segreduce(rows_params(A, B, k, 1.f, C, w.sgr), st));
    // dA = seed * <C_i, B_j> on the pattern; loss = 1/2 sum_p A_p <C_i, B_j> = 1/2 ||C||^2
    SddmmParams sp = sddmm_params(A, C, B, k, seed, dA);
    sp.w = A->val;
    sp.beta = 0.5;
    sp.part = w.part;
    NSD_TRY(sddmm(sp, st));
    NSD_TRY(finish_loss(sp, loss, st));
    // dB = seed * A^T C
    return segreduce(cols_params(A, At, C, k, seed, dB, w.sgr), st);
}

nsd_status nsd_loss_bilinear(const nsd_csr *A, const nsd_csc *At, const float *H,
                             const float *G, int32_t k, float seed, double *loss, float *dA,
                             float *dH, void *ws, size_t ws_bytes, void *stream) {
    NSD_TRY(check_csr(A, true));
    NSD_TRY(check_csc(At, A));
    NSD_REQUIRE(k >= 1, "k = %d < 1", k);
    NSD_REQUIRE(loss != nullptr, "loss is NULL");
    NSD_REQUIRE(A->ncols == 0 || dH != nullptr, "dH is NULL");
    NSD_REQUIRE(A->nnz == 0 || (H && G && dA), "H/G/dA is NULL");
    ComputeWs w;
    NSD_TRY(carve_compute(ws, ws_bytes, A->nnz, k, &w));
    hipStream_t st = as_stream(stream);
    // dA = seed * <G_i, H_j>; loss = sum_p A_p <G_i, H_j>
    SddmmParams sp = sddmm_params(A, G, H, k, seed, dA);
    sp.w = A->val;
    sp.beta = 1.0;
    sp.part = w.part;
    NSD_TRY(sddmm(sp, st));
    NSD_TRY(finish_loss(sp, loss, st));
    // dH = seed * A^T G
    return segreduce(cols_params(A, At, G, k, seed, dH, w.sgr), st);
}

}  // extern "C"
