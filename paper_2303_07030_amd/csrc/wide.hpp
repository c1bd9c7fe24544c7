// Internal interface of the wide-rank factorisation and CP passes (wide.hip).
#pragma once

#include "nsd_internal.hpp"
#include "segreduce.hpp"

namespace nsd {

// Residual of a rank-k model at every stored entry p of one storage order:
//   res_p = x[p] - sum_r prod_{n < order} fac[n][coord[n][p], r]
// rbuf[pos] = res_p and, when resid is set, resid[pos] = seed * res_p, with
// pos = perm[p] (NULL: p); part[b] = the block's sum of lscale * res_p^2.
struct ResidParams {
    int32_t nnz = 0, k = 0, order = 2;
    int32_t L = 0, nslots = 0;  // set by resid_pass
    const int32_t *coord[NSD_MAX_ORDER] = {};
    const float *fac[NSD_MAX_ORDER] = {};
    const float *x = nullptr;
    const int32_t *perm = nullptr;
    float *rbuf = nullptr;
    float *resid = nullptr;
    float seed = 1.f;
    double lscale = 1.0;
    double *part = nullptr;  // [resid_blocks]
};

// Loss partials resid_pass writes (one per block).
int64_t resid_blocks(int64_t nnz, int k, bool vec);
// Needs a slot of a whole wave: k > 64, or k > 256 with float4 rows.
nsd_status resid_pass(ResidParams a, bool vec, hipStream_t st);

// Mode pass of a CP gradient of an order-`order` tensor from a formed
// residual: s is the gather-reduce over the mode's plan (segidx = mode
// coordinate, idx = other[0], w = residuals, wperm = their positions,
// alpha = -seed, out = dF_n); the gathered row of an entry is the product of
// fac[o][other[o][p], :] over o < order - 1.
struct MttkrpParams {
    SgrParams s;
    const int32_t *other[NSD_MAX_ORDER - 1] = {};
    const float *fac[NSD_MAX_ORDER - 1] = {};
};

nsd_status mttkrp_pass(MttkrpParams m, int order, bool vec, hipStream_t st);

}  // namespace nsd
