// Products taken key by key on stored keys: what remains of a differentiated
// program's term once multiplication normalisation (Section 5) has turned
// its tensor products into loops and no index is summed.  Such a term is
// the product of at most two value arrays on one set of stored keys (one of
// them possibly a dense operand read at each key's row, column or index),
// at most two reals of the program (inputs or results, kept on the device)
// and a constant.  The Jacobians of the evaluation's vector kernels
// (Section 7.1) and of matrix-valued programs on a matrix's keys are of this
// form.  HBM-bound: one read of each operand and one write per key.
#include <algorithm>

#include "nsd_internal.hpp"

namespace nsd {

constexpr int kEwBlock = 256;

// y[yi] = c * x1[i] * x2[x2i] + beta * y[yi], c = alpha * s1 * s2, in double
// and rounded once.
__global__ __launch_bounds__(kEwBlock) void scale_kernel(int64_t n, double alpha,
                                                         const double *s1, const double *s2,
                                                         const float *x1, const float *x2,
                                                         const int32_t *x2_idx, float beta,
                                                         float *y, const int32_t *y_idx) {
    const double c = alpha * (s1 ? *s1 : 1.0) * (s2 ? *s2 : 1.0);
    const int64_t stride = (int64_t)gridDim.x * kEwBlock;
    for (int64_t i = (int64_t)blockIdx.x * kEwBlock + threadIdx.x; i < n; i += stride) {
        double v = c;
        if (x1) v *= (double)x1[i];
        if (x2) v *= (double)x2[x2_idx ? (int64_t)x2_idx[i] : i];
        const int64_t o = y_idx ? (int64_t)y_idx[i] : i;
        if (beta != 0.f) v += (double)beta * (double)y[o];
        y[o] = (float)v;
    }
}

__global__ __launch_bounds__(64) void scale_real_kernel(double alpha, const double *s1,
                                                        const double *s2, const double *x,
                                                        double beta, double *y) {
    if (threadIdx.x != 0) return;
    double v = alpha * (s1 ? *s1 : 1.0) * (s2 ? *s2 : 1.0) * (x ? *x : 1.0);
    if (beta != 0.0) v += beta * *y;
    *y = v;
}

}  // namespace nsd

using namespace nsd;

extern "C" {

nsd_status nsd_scale(int64_t n, double alpha, const double *s1, const double *s2,
                     const float *x1, const float *x2, const int32_t *x2_idx, float beta,
                     float *y, const int32_t *y_idx, void *stream) {
    NSD_REQUIRE(n >= 0, "negative length");
    if (n == 0) return NSD_OK;
    NSD_REQUIRE(y != nullptr, "y is NULL");
    NSD_REQUIRE(x2_idx == nullptr || x2 != nullptr, "x2_idx without x2");
    const int64_t nb = std::min<int64_t>(ceil_div(n, kEwBlock), 8192);
    scale_kernel<<<(unsigned)nb, kEwBlock, 0, as_stream(stream)>>>(n, alpha, s1, s2, x1, x2,
                                                                   x2_idx, beta, y, y_idx);
    return check_launch("scale_kernel");
}

nsd_status nsd_scale_real(double alpha, const double *s1, const double *s2, const double *x,
                          double beta, double *y, void *stream) {
    NSD_REQUIRE(y != nullptr, "y is NULL");
    scale_real_kernel<<<1, 64, 0, as_stream(stream)>>>(alpha, s1, s2, x, beta, y);
    return check_launch("scale_real_kernel");
}

}  // extern "C"
