// Internal interface of the gather-reduce and SDDMM kernels.
#pragma once

#include "nsd_internal.hpp"

namespace nsd {

struct SgrParams {
    int32_t nseg = 0, nnz = 0, k = 0, L = 0, nslots = 0;
    const int32_t *segptr = nullptr;  // [nseg+1]
    const int32_t *segidx = nullptr;  // [nnz] segment of each entry, sorted
    const int32_t *idx = nullptr;     // [nnz] row of X gathered by each entry
    const float *w = nullptr;         // weights (NULL: 1)
    const int32_t *wperm = nullptr;   // weight of entry p is w[wperm[p]]
    const float *X = nullptr;         // gathered dense operand (NULL: ones)
    float alpha = 1.f;
    float *out = nullptr;             // [nseg x k]
    float *pfirst = nullptr;          // [nslots x k] carry-in partials
    float *plast = nullptr;           // [nslots x k] carry-out partials
    int32_t *span = nullptr;          // [nslots] row continuing past the slot, or -1
};

struct SgrShape {
    WidthPlan wp;
    int L;
    int64_t nslots;
};

struct SddmmParams {
    int32_t nnz = 0, k = 0, L = 0, nslots = 0;
    const int32_t *rowidx = nullptr;
    const int32_t *colind = nullptr;
    const float *X = nullptr;  // [nrows x k] (NULL: ones)
    const float *Y = nullptr;  // [ncols x k]
    float alpha = 1.f;
    float *out = nullptr;      // [nnz]
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
SgrShape sgr_shape(int64_t nnz, int k);
SgrShape sgr_shape_vec1(int64_t nnz, int k);
void sgr_carve(Carver &c, int64_t nnz, int k, SgrParams *p);
nsd_status segreduce(SgrParams a, hipStream_t st);

SddmmShape sddmm_shape(int64_t nnz, int k, bool vec_ok);
bool sddmm_vec_ok(const SddmmParams &a);
nsd_status sddmm(SddmmParams a, hipStream_t st);

nsd_status loss_finalize(const double *part, int64_t n, double *loss, hipStream_t st);

}  // namespace nsd
