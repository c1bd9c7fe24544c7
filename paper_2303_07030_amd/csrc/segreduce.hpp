// Internal interface of the gather-reduce and SDDMM kernels.
#pragma once

#include "nsd_internal.hpp"

namespace nsd {

struct SgrParams {
    int32_t nseg = 0, nnz = 0, k = 0;
    nsd_plan plan{};                  // work items over the segments
    const int32_t *segptr = nullptr;  // [nseg+1]
    const int32_t *segidx = nullptr;  // [nnz] segment of each entry, sorted
    const int32_t *idx = nullptr;     // [nnz] row of X gathered by each entry
    const float *w = nullptr;         // weights (NULL: 1)
    const int32_t *wperm = nullptr;   // weight of entry p is w[wperm[p]]
    const float *X = nullptr;         // gathered dense operand (NULL: ones)
    float alpha = 1.f;
    float *out = nullptr;             // [nseg x k]
    float *part = nullptr;            // [plan.nitems x k] chunk partials
    // Rows of `part` that hold a long segment's partials: its first chunk's
    // and, past it, those of the chunks at item indexes divisible by
    // chunk_stride (1: every chunk's; chunk_group<G>(): one per group of
    // slots, the group's chunks of a segment added together first, see
    // store_chunk_partial)
    int32_t chunk_stride = 1;
    int32_t item_blocks = 0;          // set by the launcher
};

struct SddmmParams {
    int32_t nnz = 0, k = 0, L = 0, nslots = 0;
    const int32_t *rowidx = nullptr;
    const int32_t *colind = nullptr;
    const float *X = nullptr;  // [nrows x k] (NULL: ones)
    const float *Y = nullptr;  // [ncols x k]
    float alpha = 1.f;
    float *out = nullptr;      // [nnz]
    const int32_t *operm = nullptr;  // entry p goes to out[operm[p]] (NULL: out[p])
    const float *w = nullptr;  // fused loss weights (NULL: no loss)
    double beta = 1.0;         // loss += beta * sum_p w_p * <X_i, Y_j>
    double *part = nullptr;    // [nblocks] block partials of the loss
};

struct SddmmShape {
    WidthPlan wp;
    int L;
    int64_t nslots, nblocks;
};

int choose_slot_len(int64_t nnz, int slots_per_wave);
size_t sgr_part_bytes(const nsd_plan &plan, int k);
nsd_status segreduce(SgrParams a, hipStream_t st);

// The loss total, run by one extra block of the last kernel of a call:
// *loss = sum of p1[0, n1) + sum of p2[0, n2) in a fixed order.
struct LossJob {
    const double *p1 = nullptr;
    int64_t n1 = 0;
    const double *p2 = nullptr;
    int64_t n2 = 0;
    double *loss = nullptr;  // NULL: no job
};

// A pass over a segmented sparse operand that also uses each segment's own
// dense row `own` (see dual.hip):
//   d_p = <own[seg_p], X[idx_p]>,  out[seg] = alpha * sum_p c_p X[idx_p],
// with c_p = w_p (kDualLin; then sdd[pos_p] = sdd_alpha * d_p when sdd is
// set, and loss += w_p d_p when count_loss) or c_p = w_p - d_p (kDualMf;
// loss += c_p^2 when count_loss).  pos_p = wperm[p] when the weights are
// permuted, else p.
constexpr int kDualLin = 0;
constexpr int kDualMf = 1;

struct DualPass {
    SgrParams s;
    const float *own = nullptr;  // [nseg x k]
    float *sdd = nullptr;        // [nnz] sampled products at pos_p (kDualLin)
    float sdd_alpha = 1.f;
    int32_t count_loss = 0;
    int32_t item_blocks = 0, empty_blocks = 0;  // set by the launcher
};

struct DualParams {
    DualPass pass[2];
    int32_t npass = 1;
    double *loss_part = nullptr;  // [dual_blocks] block partials (NULL: no loss)
    double loss_beta = 1.0;       // scale of every block partial
    LossJob early;                // a loss total over partials of earlier launches,
                                  // run by one extra block (when early.loss is set)
};

int64_t dual_blocks(const nsd_plan *const *plans, int npass, int k, bool vec);
bool dual_vec_ok(const DualParams &f);
bool dual_supported(int k, bool vec);
// Launches the passes and their long-segment combines, the last of which
// also runs `job` (when job.loss is set); a job without p1 sums the block
// partials of the dual kernel itself (f.loss_part).
nsd_status dual_fused(int kind, DualParams f, int probe_id, LossJob job, hipStream_t st);

// Fused SpMM-gradient passes (L = 1/2 ||A B||^2): rows = C = A B over the
// row plan with the loss; cols = a linear dual pass over the column plan
// (own = B, X = C): dB = seed A^T C and dA = seed <C_i, B_j>.
struct FrobParams {
    SgrParams rows;
    DualPass cols;
    double *loss_part = nullptr;  // [frob_row_blocks] row-pass block partials
    double *seg_loss = nullptr;   // [rows.plan.nlong] long-row partials
    double *loss = nullptr;
};

// One mode pass of the CP gradient: s is the gather-reduce over the mode's
// plan (segidx = mode coordinate, idx = coordinate of mode n+1, w = values,
// out = dF_n, alpha = -seed, k = rank); own = F_n, fa / fb = the factors of
// modes n+1 / n+2.  The first pass also writes the residual through perm.
struct CpMode {
    SgrParams s;
    const int32_t *idx_b = nullptr;
    const float *own = nullptr, *fa = nullptr, *fb = nullptr;
    const int32_t *perm = nullptr;
    float *resid = nullptr;
    float seed = 1.f;
    int32_t item_blocks = 0, empty_blocks = 0;  // set by the launcher
};

struct CpParams {
    CpMode m[3];
    double *loss_part = nullptr;
};

int64_t cp_blocks(const nsd_plan *plans, int rank, bool vec);
nsd_status cp_fused(CpParams f, bool vec, double *loss, hipStream_t st);

int64_t frob_row_blocks(const nsd_plan &rows, int k);
bool frob_fused_ok(int k, const void *B, const void *C, const void *dB);
nsd_status frob_fused(FrobParams f, hipStream_t st);

SddmmShape sddmm_shape(int64_t nnz, int k, bool vec_ok);
bool sddmm_vec_ok(const SddmmParams &a);
nsd_status sddmm(SddmmParams a, hipStream_t st);

nsd_status loss_finalize(const double *part, int64_t n, double *loss, hipStream_t st);

// *out = alpha * sum x_i y_i (y NULL: ones) in fp64, fixed order, plus the
// old *out when accumulating; part holds dot_blocks(n) doubles.
int64_t dot_blocks(int64_t n);
nsd_status dot(int64_t n, const float *x, const float *y, double alpha, bool accumulate,
               double *part, double *out, hipStream_t st);

// y = alpha x + beta y elementwise (x NULL: ones; beta 0: y is not read).
nsd_status axpby(int64_t n, float alpha, const float *x, float beta, float *y, hipStream_t st);
// out[p] = alpha where entry p's row equals its column, else 0.
nsd_status diag_keys(int64_t n, const int32_t *rowidx, const int32_t *colind, float alpha,
                     float *out, hipStream_t st);

}  // namespace nsd
