// Hot-path entry points: forward products, VJP primitives and the fused
// loss + gradient calls.  Each one validates its arguments on the host, then
// enqueues kernels on the caller's stream and returns without waiting.
#include <algorithm>
#include <mutex>

#include "nsd_internal.hpp"
#include "segreduce.hpp"
#include "wide.hpp"

namespace nsd {

static nsd_status check_plan(const nsd_plan &pl, int32_t nnz, const char *what) {
    if (nnz == 0) return NSD_OK;
    NSD_REQUIRE(pl.item_ptr && pl.nitems >= 1 && pl.nlong >= 0 && pl.nempty >= 0 &&
                    pl.item_len >= 1,
                "%s plan is not built (nsd_plan_build)", what);
    NSD_REQUIRE(pl.nlong == 0 || pl.long_first, "%s plan long_first is NULL", what);
    NSD_REQUIRE(pl.nempty == 0 || pl.empty_seg, "%s plan empty_seg is NULL", what);
    return NSD_OK;
}

static nsd_status check_csr(const nsd_csr *A, bool need_val, bool need_plan) {
    NSD_REQUIRE(A != nullptr, "CSR descriptor is NULL");
    NSD_REQUIRE(A->nrows >= 0 && A->ncols >= 0 && A->nnz >= 0, "negative CSR size");
    NSD_REQUIRE(A->rowptr != nullptr, "CSR rowptr is NULL");
    if (A->nnz > 0) {
        NSD_REQUIRE(A->nrows > 0 && A->ncols > 0, "nnz > 0 in an empty shape");
        NSD_REQUIRE(A->rowidx && A->colind, "CSR rowidx/colind is NULL");
        NSD_REQUIRE(!need_val || A->val, "CSR val is NULL");
    }
    if (need_plan) NSD_TRY(check_plan(A->plan, A->nnz, "row"));
    return NSD_OK;
}

static nsd_status check_csc(const nsd_csc *At, const nsd_csr *A) {
    NSD_REQUIRE(At != nullptr, "CSC descriptor is NULL");
    NSD_REQUIRE(At->nrows == A->nrows && At->ncols == A->ncols && At->nnz == A->nnz,
                "CSC shape (%d x %d, %d) differs from CSR (%d x %d, %d)", At->nrows, At->ncols,
                At->nnz, A->nrows, A->ncols, A->nnz);
    NSD_REQUIRE(At->colptr != nullptr, "CSC colptr is NULL");
    if (At->nnz > 0) NSD_REQUIRE(At->colidx && At->rowind && At->perm, "CSC array is NULL");
    return check_plan(At->plan, At->nnz, "column");
}

static size_t round256(size_t b) { return (b + 255) & ~size_t(255); }

// Workspace: the chunk partials of the row plan, then of the column plan
// (passes that run in one launch need both), then the loss partials and the
// long-row loss partials.
static size_t row_part_bytes(const nsd_csr *A, int k) {
    return round256(sgr_part_bytes(A->plan, std::max(k, 1)));
}

static size_t part_region_bytes(const nsd_csr *A, const nsd_csc *At, int k) {
    size_t b = row_part_bytes(A, k);
    if (At) b += round256(sgr_part_bytes(At->plan, std::max(k, 1)));
    return b;
}

static size_t loss_part_count(const nsd_csr *A, const nsd_csc *At, int k) {
    int64_t m = std::max<int64_t>(1, frob_row_blocks(A->plan, k));
    for (int kk : {k, 1})
        for (bool v : {true, false}) m = std::max(m, sddmm_shape(A->nnz, kk, v).nblocks);
    if (At) {
        const nsd_plan *both[2] = {&A->plan, &At->plan};
        for (bool v : {true, false}) m = std::max(m, dual_blocks(both, 2, k, v));
    }
    return (size_t)m;
}

// Widths that a fused factorisation pass may not hold (above 64 columns
// without float4 rows, above 256 with them) form the residual once, one
// float per stored entry.
static size_t resid_buf_bytes(const nsd_csr *A, int k) {
    return k > 64 ? round256((size_t)std::max(A->nnz, 1) * sizeof(float)) : 0;
}

// A CSC carrying both two-pass forms of its perm moves A's values to CSC
// order and the sparse gradient back through them (three arrays of nnz
// floats: the values, the gradient in CSC order, the staging of a move).
static bool has_perm_plans(const nsd_csc *At) {
    return At && At->nnz > 0 && At->to_csc.n == At->nnz && At->to_csr.n == At->nnz;
}

static size_t perm_bufs_bytes(const nsd_csr *A, const nsd_csc *At) {
    return has_perm_plans(At) ? 3 * round256((size_t)A->nnz * sizeof(float)) : 0;
}

static size_t compute_ws_bytes(const nsd_csr *A, const nsd_csc *At, int k) {
    return part_region_bytes(A, At, k) + round256(loss_part_count(A, At, k) * sizeof(double)) +
           round256(std::max<size_t>(A->plan.nlong, 1) * sizeof(double)) +
           resid_buf_bytes(A, k) + perm_bufs_bytes(A, At);
}

struct ComputeWs {
    float *part;      // row-plan partials (also used alone by single passes)
    float *part_col;  // column-plan partials for passes sharing a launch
    double *loss_part;
    double *seg_loss;
    float *rbuf;      // residual per stored entry (wide factorisation only)
    float *valT, *gradT, *staging;  // with the CSC's perm plans only
};

static nsd_status carve_compute(void *ws, size_t ws_bytes, const nsd_csr *A, const nsd_csc *At,
                                int k, ComputeWs *out) {
    const size_t need = compute_ws_bytes(A, At, k);
    if (ws == nullptr || ws_bytes < need)
        return fail(NSD_ERR_WORKSPACE, "workspace %zu bytes at %p, need %zu", ws_bytes, ws, need);
    char *b = static_cast<char *>(ws);
    out->part = reinterpret_cast<float *>(b);
    out->part_col = reinterpret_cast<float *>(b + row_part_bytes(A, k));
    b += part_region_bytes(A, At, k);
    out->loss_part = reinterpret_cast<double *>(b);
    b += round256(loss_part_count(A, At, k) * sizeof(double));
    out->seg_loss = reinterpret_cast<double *>(b);
    b += round256(std::max<size_t>(A->plan.nlong, 1) * sizeof(double));
    out->rbuf = resid_buf_bytes(A, k) ? reinterpret_cast<float *>(b) : nullptr;
    b += resid_buf_bytes(A, k);
    out->valT = out->gradT = out->staging = nullptr;
    if (has_perm_plans(At)) {
        const size_t one = round256((size_t)A->nnz * sizeof(float));
        out->valT = reinterpret_cast<float *>(b);
        out->gradT = reinterpret_cast<float *>(b + one);
        out->staging = reinterpret_cast<float *>(b + 2 * one);
    }
    return NSD_OK;
}

static SgrParams rows_params(const nsd_csr *A, const float *X, int k, float alpha, float *out,
                             float *part) {
    SgrParams p;
    p.nseg = A->nrows;
    p.nnz = A->nnz;
    p.k = k;
    p.plan = A->plan;
    p.segptr = A->rowptr;
    p.segidx = A->rowidx;
    p.idx = A->colind;
    p.w = A->val;
    p.X = X;
    p.alpha = alpha;
    p.out = out;
    p.part = part;
    return p;
}

static SgrParams cols_params(const nsd_csr *A, const nsd_csc *At, const float *G, int k,
                             float alpha, float *out, float *part) {
    SgrParams p;
    p.nseg = A->ncols;
    p.nnz = A->nnz;
    p.k = k;
    p.plan = At->plan;
    p.segptr = At->colptr;
    p.segidx = At->colidx;
    p.idx = At->rowind;
    p.w = A->val;
    p.wperm = At->perm;
    p.X = G;
    p.alpha = alpha;
    p.out = out;
    p.part = part;
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

// Linear dual pass over A's columns: own row O[j], gathered row X[i] (NULL:
// ones), w = A's values through perm;  out = alpha * A^T X,
// sdd[p] = sdd_alpha * <X_i, O_j> at A's storage position p.
static DualPass col_dual(const nsd_csr *A, const nsd_csc *At, const float *X, const float *O,
                         int k, float alpha, float *out, float *part, float *sdd,
                         float sdd_alpha, bool count_loss) {
    DualPass d;
    d.s = cols_params(A, At, X, k, alpha, out, part);
    d.own = O;
    d.sdd = sdd;
    d.sdd_alpha = sdd_alpha;
    d.count_loss = count_loss ? 1 : 0;
    return d;
}

// One linear dual pass over the columns with its loss, then the loss total.
static nsd_status col_dual_loss(const DualPass &pass, double *loss_part, double *loss,
                                hipStream_t st) {
    DualParams f;
    f.pass[0] = pass;
    f.npass = 1;
    f.loss_part = loss_part;
    LossJob job;
    job.loss = loss;  // sums the dual kernel's own block partials
    return dual_fused(kDualLin, f, NSD_KERNEL_DUAL, job, st);
}

static bool col_dual_ok(const DualPass &pass) {
    DualParams f;
    f.pass[0] = pass;
    return dual_supported(pass.s.k, dual_vec_ok(f));
}

static nsd_status check_bilinear(const nsd_csr *A, const nsd_csc *At, const float *H,
                                 const float *G, int k, const double *loss, const float *dA,
                                 const float *dH) {
    NSD_TRY(check_csr(A, true, false));
    NSD_TRY(check_csc(At, A));
    NSD_REQUIRE(k >= 1, "k = %d < 1", k);
    NSD_REQUIRE(loss != nullptr, "loss is NULL");
    NSD_REQUIRE(A->ncols == 0 || dH != nullptr, "dH is NULL");
    NSD_REQUIRE(A->nnz == 0 || (H && G && dA), "H/G/dA is NULL");
    return NSD_OK;
}

// Loss partials of the bilinear layer: one per block of its fused column
// pass, or of the unfused SDDMM (widths a fused slot does not hold).
static int64_t bilinear_loss_parts(const nsd_csr *A, const nsd_csc *At, int k) {
    const nsd_plan *cols[1] = {&At->plan};
    int64_t m = 1;
    for (bool v : {true, false})
        m = std::max({m, dual_blocks(cols, 1, k, v), sddmm_shape(A->nnz, k, v).nblocks});
    return m;
}

// The loss total of an unfused SDDMM's block partials; with nnz == 0 the
// loss is 0.
static nsd_status finish_loss(const SddmmParams &p, double *loss, hipStream_t st);

// The bilinear layer L = sum (A H) o G with its gradients, given the chunk
// partials of the column plan and the loss partials; with valT, gradT and
// staging (nnz floats each) A's values are moved to CSC order and the sparse
// gradient back by the CSC's two-pass permutations.
// With the CSC's two-pass permutations (large patterns), a column pass reads
// A's values moved to CSC order and writes its sampled products there, so
// its entry positions are its own slots; csc_order_after moves the products
// back to A's order.  Without them the pass reads and writes through perm.
static nsd_status csc_order_before(const nsd_csr *A, const nsd_csc *At, float *valT,
                                   float *gradT, float *staging, DualPass &pass, hipStream_t st) {
    if (!valT) return NSD_OK;
    NSD_TRY(nsd_permute_f32(&At->to_csc, A->val, valT, staging, st));
    pass.s.w = valT;
    pass.s.wperm = nullptr;
    pass.sdd = gradT;
    return NSD_OK;
}

static nsd_status csc_order_after(const nsd_csc *At, float *valT, const float *gradT,
                                  float *staging, float *dA, hipStream_t st) {
    if (!valT) return NSD_OK;
    return nsd_permute_f32(&At->to_csr, gradT, dA, staging, st);
}

static nsd_status bilinear_run(const nsd_csr *A, const nsd_csc *At, const float *H,
                               const float *G, int k, float seed, double *loss, float *dA,
                               float *dH, float *part_col, double *loss_part, hipStream_t st,
                               float *valT = nullptr, float *gradT = nullptr,
                               float *staging = nullptr) {
    if (A->nnz > 0) {
        // one pass over the columns: own row H_j, gathered row G_i:
        // dA[p] = seed <G_i, H_j>, loss = sum_p A_p <G_i, H_j>, dH = seed A^T G
        DualPass pass = col_dual(A, At, G, H, k, seed, dH, part_col, dA, seed, true);
        if (col_dual_ok(pass)) {
            NSD_TRY(csc_order_before(A, At, valT, gradT, staging, pass, st));
            NSD_TRY(col_dual_loss(pass, loss_part, loss, st));
            return csc_order_after(At, valT, gradT, staging, dA, st);
        }
    }
    // dA = seed * <G_i, H_j>; loss = sum_p A_p <G_i, H_j>
    SddmmParams sp = sddmm_params(A, G, H, k, seed, dA);
    sp.w = A->val;
    sp.beta = 1.0;
    sp.part = loss_part;
    NSD_TRY(sddmm(sp, st));
    NSD_TRY(finish_loss(sp, loss, st));
    // dH = seed * A^T G
    return segreduce(cols_params(A, At, G, k, seed, dH, part_col), st);
}

// ------------------------------------------------------ static scratch

// Scratch of the entry points that allocate nothing (for callers that
// cannot allocate: code under graph capture, serving loops): a file-scope
// device array, one copy per GPU that the library runs on, held until the
// process ends.  Host code never uses the array's name as an address: the
// device address is looked up once per device (hipGetSymbolAddress, with that
// device current, on the first call made there) and kept.
constexpr size_t kScratchBytes = size_t(64) << 20;
__device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
static std::mutex g_scratch_mu;
static void *g_scratch[kMaxDevices];

static nsd_status scratch_base(char **out) {
    int dev = 0;
    NSD_HIP(hipGetDevice(&dev));
    if (dev < 0 || dev >= kMaxDevices) return fail(NSD_ERR_UNSUPPORTED, "device %d", dev);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (g_scratch[dev] == nullptr) {
        void *p = nullptr;
        NSD_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
        g_scratch[dev] = p;
    }
    *out = static_cast<char *>(g_scratch[dev]);
    return NSD_OK;
}

// The loss partial count of a fused SDDMM; with nnz == 0 the loss is 0.
static nsd_status finish_loss(const SddmmParams &p, double *loss, hipStream_t st) {
    // with nnz == 0 there are no partials and the finaliser writes 0
    return loss_finalize(p.part, sddmm_shape(p.nnz, p.k, sddmm_vec_ok(p)).nblocks, loss, st);
}

}  // namespace nsd

using namespace nsd;

extern "C" {

nsd_status nsd_workspace_size(const nsd_csr *A, const nsd_csc *At, int32_t k, size_t *bytes) {
    NSD_REQUIRE(bytes != nullptr, "bytes is NULL");
    NSD_REQUIRE(k >= 1, "k = %d < 1", k);
    NSD_TRY(check_csr(A, false, false));
    if (At) NSD_TRY(check_csc(At, A));
    *bytes = compute_ws_bytes(A, At, k);
    return NSD_OK;
}

nsd_status nsd_spmv(const nsd_csr *A, const float *x, float *y, void *ws, size_t ws_bytes,
                    void *stream) {
    NSD_TRY(check_csr(A, true, true));
    NSD_REQUIRE(A->nrows == 0 || y != nullptr, "y is NULL");
    NSD_REQUIRE(A->nnz == 0 || x != nullptr, "x is NULL");
    ComputeWs w;
    NSD_TRY(carve_compute(ws, ws_bytes, A, nullptr, 1, &w));
    return segreduce(rows_params(A, x, 1, 1.f, y, w.part), as_stream(stream));
}

nsd_status nsd_spmm(const nsd_csr *A, const float *B, int32_t k, float *C, void *ws,
                    size_t ws_bytes, void *stream) {
    NSD_TRY(check_csr(A, true, true));
    NSD_REQUIRE(k >= 1, "k = %d < 1", k);
    NSD_REQUIRE(A->nrows == 0 || C != nullptr, "C is NULL");
    NSD_REQUIRE(A->nnz == 0 || B != nullptr, "B is NULL");
    ComputeWs w;
    NSD_TRY(carve_compute(ws, ws_bytes, A, nullptr, k, &w));
    return segreduce(rows_params(A, B, k, 1.f, C, w.part), as_stream(stream));
}

nsd_status nsd_sddmm(const nsd_csr *A, const float *X, const float *Y, int32_t k, float alpha,
                     float *out, void *stream) {
    NSD_TRY(check_csr(A, false, false));
    NSD_REQUIRE(k >= 1, "k = %d < 1", k);
    NSD_REQUIRE(A->nnz == 0 || (Y != nullptr && out != nullptr), "Y/out is NULL");
    return sddmm(sddmm_params(A, X, Y, k, alpha, out), as_stream(stream));
}

nsd_status nsd_spmm_t(const nsd_csr *A, const nsd_csc *At, const float *G, int32_t k,
                      float alpha, float *out, void *ws, size_t ws_bytes, void *stream) {
    NSD_TRY(check_csr(A, true, false));
    NSD_TRY(check_csc(At, A));
    NSD_REQUIRE(k >= 1, "k = %d < 1", k);
    NSD_REQUIRE(A->ncols == 0 || out != nullptr, "out is NULL");
    ComputeWs w;
    NSD_TRY(carve_compute(ws, ws_bytes, A, At, k, &w));
    return segreduce(cols_params(A, At, G, k, alpha, out, w.part_col), as_stream(stream));
}

nsd_status nsd_loss_sum_spmv(const nsd_csr *A, const nsd_csc *At, const float *x, float seed,
                             double *loss, float *dA, float *dx, void *ws, size_t ws_bytes,
                             void *stream) {
    NSD_TRY(check_csr(A, true, false));
    NSD_TRY(check_csc(At, A));
    NSD_REQUIRE(loss != nullptr, "loss is NULL");
    NSD_REQUIRE(A->nnz == 0 || (x && dA), "x/dA is NULL");
    NSD_REQUIRE(A->ncols == 0 || dx != nullptr, "dx is NULL");
    ComputeWs w;
    NSD_TRY(carve_compute(ws, ws_bytes, A, At, 1, &w));
    hipStream_t st = as_stream(stream);
    if (A->nnz > 0) {
        // one pass over the columns: own row x[j], gathered row 1:
        // dA[p] = seed * x[j], loss = sum_p A_p x[j], dx = seed * A^T 1
        return col_dual_loss(col_dual(A, At, nullptr, x, 1, seed, dx, w.part_col, dA, seed, true),
                             w.loss_part, loss, st);
    }
    // dA[p] = seed * x[col]; loss = sum_p A_p * x[col]
    SddmmParams sp = sddmm_params(A, nullptr, x, 1, seed, dA);
    sp.w = A->val;
    sp.beta = 1.0;
    sp.part = w.loss_part;
    NSD_TRY(sddmm(sp, st));
    NSD_TRY(finish_loss(sp, loss, st));
    // dx = seed * A^T 1
    return segreduce(cols_params(A, At, nullptr, 1, seed, dx, w.part_col), st);
}

nsd_status nsd_loss_frob_spmm(const nsd_csr *A, const nsd_csc *At, const float *B, int32_t k,
                              float seed, float *C, double *loss, float *dA, float *dB,
                              void *ws, size_t ws_bytes, void *stream) {
    NSD_TRY(check_csr(A, true, true));
    NSD_TRY(check_csc(At, A));
    NSD_REQUIRE(k >= 1, "k = %d < 1", k);
    NSD_REQUIRE(loss != nullptr, "loss is NULL");
    NSD_REQUIRE(A->nrows == 0 || C != nullptr, "C is NULL");
    NSD_REQUIRE(A->ncols == 0 || dB != nullptr, "dB is NULL");
    NSD_REQUIRE(A->nnz == 0 || (B && dA), "B/dA is NULL");
    ComputeWs w;
    NSD_TRY(carve_compute(ws, ws_bytes, A, At, k, &w));
    hipStream_t st = as_stream(stream);
    if (A->nnz > 0 && frob_fused_ok(k, B, C, dB)) {
        // row pass (C and the loss), long-row combine, one column pass (dB
        // and dA, with B_j the column's own row), long-column combine, total
        FrobParams f;
        f.rows = rows_params(A, B, k, 1.f, C, w.part);
        f.cols = col_dual(A, At, C, B, k, seed, dB, w.part_col, dA, seed, false);
        f.loss_part = w.loss_part;
        f.seg_loss = w.seg_loss;
        f.loss = loss;
        NSD_TRY(csc_order_before(A, At, w.valT, w.gradT, w.staging, f.cols, st));
        NSD_TRY(frob_fused(f, st));
        return csc_order_after(At, w.valT, w.gradT, w.staging, dA, st);
    }
    // forward: C = A B
    NSD_TRY(segreduce(rows_params(A, B, k, 1.f, C, w.part), st));
    // dA = seed * <C_i, B_j> on the pattern; loss = 1/2 sum_p A_p <C_i, B_j> = 1/2 ||C||^2
    SddmmParams sp = sddmm_params(A, C, B, k, seed, dA);
    sp.w = A->val;
    sp.beta = 0.5;
    sp.part = w.loss_part;
    NSD_TRY(sddmm(sp, st));
    NSD_TRY(finish_loss(sp, loss, st));
    // dB = seed * A^T C
    return segreduce(cols_params(A, At, C, k, seed, dB, w.part_col), st);
}

nsd_status nsd_loss_bilinear(const nsd_csr *A, const nsd_csc *At, const float *H,
                             const float *G, int32_t k, float seed, double *loss, float *dA,
                             float *dH, void *ws, size_t ws_bytes, void *stream) {
    NSD_TRY(check_bilinear(A, At, H, G, k, loss, dA, dH));
    ComputeWs w;
    NSD_TRY(carve_compute(ws, ws_bytes, A, At, k, &w));
    return bilinear_run(A, At, H, G, k, seed, loss, dA, dH, w.part_col, w.loss_part,
                        as_stream(stream), w.valT, w.gradT, w.staging);
}

nsd_status nsd_loss_bilinear_noalloc(const nsd_csr *A, const nsd_csc *At, const float *H,
                                     const float *G, int32_t k, float seed, double *loss,
                                     float *dA, float *dH, void *stream) {
    NSD_TRY(check_bilinear(A, At, H, G, k, loss, dA, dH));
    // the layout in the static scratch: the column plan's chunk partials,
    // then the loss partials of the fused pass (or of the unfused SDDMM)
    const size_t part = round256(sgr_part_bytes(At->plan, k));
    const size_t need = part + round256(bilinear_loss_parts(A, At, k) * sizeof(double));
    if (need > kScratchBytes)
        return fail(NSD_ERR_WORKSPACE,
                    "this operand needs %zu bytes of scratch; the static scratch holds %zu "
                    "(use nsd_loss_bilinear with a workspace)", need, kScratchBytes);
    char *b = nullptr;
    NSD_TRY(scratch_base(&b));
    return bilinear_run(A, At, H, G, k, seed, loss, dA, dH, reinterpret_cast<float *>(b),
                        reinterpret_cast<double *>(b + part), as_stream(stream));
}

nsd_status nsd_spmm_vjp(const nsd_csr *A, const nsd_csc *At, const float *X, const float *G,
                        int32_t k, float *dA, float *dX, void *ws, size_t ws_bytes, void *stream) {
    NSD_TRY(check_csr(A, true, false));
    NSD_TRY(check_csc(At, A));
    NSD_REQUIRE(k >= 1, "k = %d < 1", k);
    NSD_REQUIRE(A->ncols == 0 || dX != nullptr, "dX is NULL");
    NSD_REQUIRE(A->nnz == 0 || (X && dA), "X/dA is NULL");
    ComputeWs w;
    NSD_TRY(carve_compute(ws, ws_bytes, A, At, k, &w));
    hipStream_t st = as_stream(stream);
    if (A->nnz > 0) {
        // one pass over the columns: own row X_j, gathered row G_i (NULL:
        // ones): dA[p] = <G_i, X_j>, dX = A^T G; no loss
        DualPass pass = col_dual(A, At, G, X, k, 1.f, dX, w.part_col, dA, 1.f, false);
        if (col_dual_ok(pass)) {
            NSD_TRY(csc_order_before(A, At, w.valT, w.gradT, w.staging, pass, st));
            DualParams f;
            f.pass[0] = pass;
            f.npass = 1;
            f.loss_part = w.loss_part;
            NSD_TRY(dual_fused(kDualLin, f, NSD_KERNEL_DUAL, LossJob{}, st));
            return csc_order_after(At, w.valT, w.gradT, w.staging, dA, st);
        }
        NSD_TRY(sddmm(sddmm_params(A, G, X, k, 1.f, dA), st));
    }
    return segreduce(cols_params(A, At, G, k, 1.f, dX, w.part_col), st);
}

nsd_status nsd_spmv_vjp(const nsd_csr *A, const nsd_csc *At, const float *x, const float *gy,
                        float *dA, float *dx, void *ws, size_t ws_bytes, void *stream) {
    return nsd_spmm_vjp(A, At, x, gy, 1, dA, dx, ws, ws_bytes, stream);
}

nsd_status nsd_dot(int64_t n, const float *x, const float *y, double alpha, int accumulate,
                   double *out, void *ws, size_t ws_bytes, void *stream) {
    NSD_REQUIRE(n >= 0, "negative length");
    NSD_REQUIRE(out != nullptr, "out is NULL");
    NSD_REQUIRE(n == 0 || x != nullptr, "x is NULL");
    const size_t need = dot_blocks(n) * sizeof(double);
    if (ws == nullptr || ws_bytes < need)
        return fail(NSD_ERR_WORKSPACE, "workspace %zu bytes at %p, need %zu", ws_bytes, ws, need);
    return dot(n, x, y, alpha, accumulate != 0, static_cast<double *>(ws), out,
               as_stream(stream));
}

nsd_status nsd_axpby(int64_t n, float alpha, const float *x, float beta, float *y,
                     void *stream) {
    NSD_REQUIRE(n >= 0, "negative length");
    NSD_REQUIRE(n == 0 || y != nullptr, "y is NULL");
    return axpby(n, alpha, x, beta, y, as_stream(stream));
}

nsd_status nsd_diag_keys(const nsd_csr *A, float alpha, float *out, void *stream) {
    NSD_TRY(check_csr(A, false, false));
    NSD_REQUIRE(A->nnz == 0 || out != nullptr, "out is NULL");
    return diag_keys(A->nnz, A->rowidx, A->colind, alpha, out, as_stream(stream));
}

nsd_status nsd_loss_mf(const nsd_csr *A, const nsd_csc *At, const float *valT, const float *U,
                       const float *V, int32_t k, float seed, double *loss, float *dU, float *dV,
                       void *ws, size_t ws_bytes, void *stream) {
    NSD_TRY(check_csr(A, true, true));
    NSD_TRY(check_csc(At, A));
    NSD_REQUIRE(k >= 1, "k = %d < 1", k);
    NSD_REQUIRE(loss != nullptr, "loss is NULL");
    NSD_REQUIRE(A->nrows == 0 || dU != nullptr, "dU is NULL");
    NSD_REQUIRE(A->ncols == 0 || dV != nullptr, "dV is NULL");
    NSD_REQUIRE(A->nnz == 0 || (U && V), "U/V is NULL");
    const bool vec = k % 4 == 0 && aligned16(U) && aligned16(V) && aligned16(dU) && aligned16(dV);
    ComputeWs w;
    NSD_TRY(carve_compute(ws, ws_bytes, A, At, k, &w));
    hipStream_t st = as_stream(stream);
    if (!dual_supported(k, vec)) {
        // wider than a fused slot: r_ij once (CSR order) with the loss,
        // then dU over the rows and dV over the columns with r as weights
        ResidParams r;
        r.nnz = A->nnz;
        r.k = k;
        r.order = 2;
        r.coord[0] = A->rowidx;
        r.coord[1] = A->colind;
        r.fac[0] = U;
        r.fac[1] = V;
        r.x = A->val;
        r.rbuf = w.rbuf;
        r.part = w.loss_part;
        NSD_TRY(resid_pass(r, vec, st));
        SgrParams rows = rows_params(A, V, k, -2.f * seed, dU, w.part);
        rows.w = w.rbuf;
        NSD_TRY(segreduce(rows, st));
        SgrParams cols = cols_params(A, At, U, k, -2.f * seed, dV, w.part_col);
        cols.w = w.rbuf;  // through At->perm
        NSD_TRY(segreduce(cols, st));
        return loss_finalize(w.loss_part, resid_blocks(A->nnz, k, vec), loss, st);
    }
    // row pass: dU = -2 seed sum_j r_ij V_j with the loss; column pass:
    // dV = -2 seed sum_i r_ij U_i, r recomputed; both in one launch
    DualParams f;
    f.npass = 2;
    f.pass[0].s = rows_params(A, V, k, -2.f * seed, dU, w.part);
    f.pass[0].own = U;
    f.pass[0].count_loss = 1;
    f.pass[1].s = cols_params(A, At, U, k, -2.f * seed, dV, w.part_col);
    if (valT) {
        f.pass[1].s.w = valT;
        f.pass[1].s.wperm = nullptr;
    }
    f.pass[1].own = V;
    f.loss_part = w.loss_part;
    LossJob job;
    job.loss = loss;  // sums the dual kernel's own block partials
    return dual_fused(kDualMf, f, NSD_KERNEL_MF, job, st);
}

static nsd_status check_coo3(const nsd_coo3 *X) {
    NSD_REQUIRE(X != nullptr, "COO3 descriptor is NULL");
    NSD_REQUIRE(X->nnz >= 0 && X->dims[0] >= 0 && X->dims[1] >= 0 && X->dims[2] >= 0,
                "negative COO3 size");
    for (int n = 0; n < 3; ++n) {
        const nsd_coo3_mode &m = X->mode[n];
        NSD_REQUIRE(m.mode == n, "mode[%d] holds mode %d", n, m.mode);
        NSD_REQUIRE(m.segptr != nullptr, "mode %d segptr is NULL", n);
        if (X->nnz > 0) {
            NSD_REQUIRE(X->dims[0] > 0 && X->dims[1] > 0 && X->dims[2] > 0,
                        "nnz > 0 in an empty shape");
            NSD_REQUIRE(m.segidx && m.idx_a && m.idx_b && m.val && m.perm,
                        "mode %d array is NULL", n);
        }
        NSD_TRY(check_plan(m.plan, X->nnz, "mode"));
    }
    return NSD_OK;
}

// Per-mode chunk partials, the loss partials, and (ranks above 64, which a
// fused slot may not hold) the residual of every stored entry.
static size_t cp_ws_bytes(const nsd_coo3 *X, int rank) {
    size_t b = 0;
    nsd_plan plans[3];
    for (int n = 0; n < 3; ++n) {
        b += round256(sgr_part_bytes(X->mode[n].plan, std::max(rank, 1)));
        plans[n] = X->mode[n].plan;
    }
    int64_t blocks = std::max(cp_blocks(plans, rank, true), cp_blocks(plans, rank, false));
    if (rank > 64)
        blocks = std::max({blocks, resid_blocks(X->nnz, rank, true),
                           resid_blocks(X->nnz, rank, false)});
    b += round256(std::max<int64_t>(blocks, 1) * sizeof(double));
    if (rank > 64) b += round256((size_t)std::max(X->nnz, 1) * sizeof(float));
    return b;
}

// CP gradient of a rank wider than a fused slot: the residual once in mode
// 0's order (written to dX and, unscaled, to a buffer in X's input order),
// then one mode pass per mode reading it through the mode's permutation.
static nsd_status cp_wide(const nsd_coo3 *X, const float *const *F, int rank, float seed,
                          double *loss, float *dX, float *const *dF, bool vec, char *b,
                          hipStream_t st) {
    float *part[3];
    for (int n = 0; n < 3; ++n) {
        part[n] = reinterpret_cast<float *>(b);
        b += round256(sgr_part_bytes(X->mode[n].plan, rank));
    }
    double *loss_part = reinterpret_cast<double *>(b);
    nsd_plan plans[3] = {X->mode[0].plan, X->mode[1].plan, X->mode[2].plan};
    const int64_t blocks = std::max({cp_blocks(plans, rank, true), cp_blocks(plans, rank, false),
                                     resid_blocks(X->nnz, rank, true),
                                     resid_blocks(X->nnz, rank, false)});
    b += round256(std::max<int64_t>(blocks, 1) * sizeof(double));
    float *rbuf = reinterpret_cast<float *>(b);
    const nsd_coo3_mode &m0 = X->mode[0];
    ResidParams r;
    r.nnz = X->nnz;
    r.k = rank;
    r.order = 3;
    r.coord[0] = m0.segidx;
    r.coord[1] = m0.idx_a;
    r.coord[2] = m0.idx_b;
    for (int n = 0; n < 3; ++n) r.fac[n] = F[n];
    r.x = m0.val;
    r.perm = m0.perm;
    r.rbuf = rbuf;
    r.resid = dX;
    r.seed = seed;
    r.lscale = 0.5;
    r.part = loss_part;
    NSD_TRY(resid_pass(r, vec, st));
    for (int n = 0; n < 3; ++n) {
        const nsd_coo3_mode &md = X->mode[n];
        MttkrpParams m;
        m.s.nseg = X->dims[n];
        m.s.nnz = X->nnz;
        m.s.k = rank;
        m.s.plan = md.plan;
        m.s.segptr = md.segptr;
        m.s.segidx = md.segidx;
        m.s.idx = md.idx_a;
        m.s.w = rbuf;
        m.s.wperm = md.perm;
        m.s.alpha = -seed;
        m.s.out = dF[n];
        m.s.part = part[n];
        m.other[0] = md.idx_a;
        m.other[1] = md.idx_b;
        m.fac[0] = F[(n + 1) % 3];
        m.fac[1] = F[(n + 2) % 3];
        NSD_TRY(mttkrp_pass(m, 3, vec, st));
    }
    return loss_finalize(loss_part, resid_blocks(X->nnz, rank, vec), loss, st);
}

nsd_status nsd_cp_workspace_size(const nsd_coo3 *X, int32_t rank, size_t *bytes) {
    NSD_REQUIRE(bytes != nullptr, "bytes is NULL");
    NSD_REQUIRE(rank >= 1, "rank = %d < 1", rank);
    NSD_TRY(check_coo3(X));
    *bytes = cp_ws_bytes(X, rank);
    return NSD_OK;
}

nsd_status nsd_loss_cp(const nsd_coo3 *X, const float *F1, const float *F2, const float *F3,
                       int32_t rank, float seed, double *loss, float *dX, float *dF1,
                       float *dF2, float *dF3, void *ws, size_t ws_bytes, void *stream) {
    NSD_TRY(check_coo3(X));
    NSD_REQUIRE(rank >= 1, "rank = %d < 1", rank);
    NSD_REQUIRE(loss != nullptr, "loss is NULL");
    const float *F[3] = {F1, F2, F3};
    float *dF[3] = {dF1, dF2, dF3};
    for (int n = 0; n < 3; ++n) {
        NSD_REQUIRE(X->dims[n] == 0 || dF[n] != nullptr, "dF%d is NULL", n + 1);
        NSD_REQUIRE(X->nnz == 0 || F[n] != nullptr, "F%d is NULL", n + 1);
    }
    NSD_REQUIRE(X->nnz == 0 || dX != nullptr, "dX is NULL");
    bool vec = rank % 4 == 0;
    for (int n = 0; n < 3; ++n) vec = vec && aligned16(F[n]) && aligned16(dF[n]);
    const size_t need = cp_ws_bytes(X, rank);
    if (ws == nullptr || ws_bytes < need)
        return fail(NSD_ERR_WORKSPACE, "workspace %zu bytes at %p, need %zu", ws_bytes, ws, need);
    char *b = static_cast<char *>(ws);
    if (vec ? rank > 256 : rank > 64) return cp_wide(X, F, rank, seed, loss, dX, dF, vec, b,
                                                     as_stream(stream));
    CpParams f;
    for (int n = 0; n < 3; ++n) {
        const nsd_coo3_mode &md = X->mode[n];
        CpMode &m = f.m[n];
        m.s.nseg = X->dims[n];
        m.s.nnz = X->nnz;
        m.s.k = rank;
        m.s.plan = md.plan;
        m.s.segptr = md.segptr;
        m.s.segidx = md.segidx;
        m.s.idx = md.idx_a;
        m.s.w = md.val;
        m.s.alpha = -seed;
        m.s.out = dF[n];
        m.s.part = reinterpret_cast<float *>(b);
        b += round256(sgr_part_bytes(md.plan, rank));
        m.idx_b = md.idx_b;
        m.own = F[n];
        m.fa = F[(n + 1) % 3];
        m.fb = F[(n + 2) % 3];
        m.perm = md.perm;
        m.resid = dX;
        m.seed = seed;
    }
    f.loss_part = reinterpret_cast<double *>(b);
    return cp_fused(f, vec, loss, as_stream(stream));
}

}  // extern "C"
