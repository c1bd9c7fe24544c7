// Fused loss and gradients of sparse matrix factorisation:
//   L  = sum over stored (i, j) of r_ij^2,   r_ij = A(i, j) - <U[i,:], V[j,:]>
//   dU[i,:] = -2 seed sum_j r_ij V[j,:]     (row pass, over A's row plan)
//   dV[j,:] = -2 seed sum_i r_ij U[i,:]     (column pass, over the column plan)
// The residual is the paper's `sum` over the stored keys of A with the
// factor rows looked up by key (Logical SDQLite, Section 3); its gradient is
// keyed by the stored entries only (Section 4.3).
//
// Both passes are gather-reduces whose weight is computed on the fly: per
// entry the other factor's row is gathered once and used twice, for the dot
// product that gives r (reduced across the slot's lanes with a transposing
// butterfly and broadcast back) and for the accumulation r * row.  The two
// passes are independent and share one launch (disjoint block ranges); the
// residual is recomputed in the column pass instead of being stored.  The
// loss is counted in the row pass only.  Long rows and columns use the
// chunk partials and the shared combine kernel.
#include "nsd_internal.hpp"
#include "segreduce.hpp"
#include "segreduce_dev.hpp"

namespace nsd {

template <int VEC, int G, int U>
__device__ __forceinline__ void mf_walk(const MfPass &m, int64_t s, int lane, bool count_loss,
                                        double &lsum) {
    const SgrParams &a = m.s;
    const int g = lane % G;
    const int col = g * VEC;  // k <= G * VEC on this path
    const bool on = col < a.k;
    const int64_t k = a.k;
    const int64_t a0 = a.plan.item_ptr[s];
    const int64_t b0 = a.plan.item_ptr[s + 1];
    const int last_r = a.segidx[b0 - 1];
    const int last_c = a.idx[b0 - 1];
    int row = a.segidx[a0];
    bool carry = a0 > 0 && a.segidx[a0 - 1] == row;

    Vec<VEC> acc;
    acc.zero();
    auto flush = [&]() {
        if (!on) return;
        if (carry) {
            acc.store(a.part + s * k + col);
        } else {
            Vec<VEC> t = acc;
            t.scale(a.alpha);
            t.store(a.out + (int64_t)row * k + col);
        }
    };

    Meta<U> cur, nxt;
    load_meta(a, a0, b0, last_r, last_c, cur);
    for (int64_t p = a0; p < b0; p += U) {
        if (p + U < b0) load_meta(a, p + U, b0, last_r, last_c, nxt);
        Vec<VEC> xv[U], ov[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (on) {
                xv[u].load(a.X + (int64_t)cur.c[u] * k + col);
                ov[u].load(m.own + (int64_t)cur.r[u] * k + col);
            } else {
                xv[u].zero();
                ov[u].zero();
            }
        }
        float d[U];
#pragma unroll
        for (int u = 0; u < U; ++u) d[u] = ov[u].dot(xv[u]);
        float rr[U];
        if constexpr (G == 1) {
#pragma unroll
            for (int u = 0; u < U; ++u) rr[u] = p + u < b0 ? cur.w[u] - d[u] : 0.f;
        } else {
            const float tot = transpose_reduce<G, U>(d, lane);
            constexpr int kRep = G / U;
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const float t = __shfl(tot, u * kRep, G);
                rr[u] = p + u < b0 ? cur.w[u] - t : 0.f;
            }
        }
        if (count_loss && g == 0)
#pragma unroll
            for (int u = 0; u < U; ++u) lsum += (double)rr[u] * rr[u];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (cur.r[u] != row) {
                flush();
                row = cur.r[u];
                carry = false;
                acc.zero();
            }
            acc.fma(rr[u], xv[u]);
        }
        cur = nxt;
    }
    if (b0 == a.nnz || a.segidx[b0] != row) {
        flush();
    } else if (on) {
        acc.store(a.part + s * k + col);
    }
}

template <int VEC, int G, int U>
__device__ __forceinline__ void mf_block(const MfPass &m, int b, bool count_loss, double &lsum) {
    constexpr int kSlots = kBlock / G;
    const int lane = threadIdx.x % kWave;
    const int g = threadIdx.x % G;
    if (b < m.item_blocks) {
        const int64_t s = (int64_t)b * kSlots + threadIdx.x / G;
        if (s < m.s.plan.nitems) mf_walk<VEC, G, U>(m, s, lane, count_loss, lsum);
    } else {
        zero_segment<VEC>(m.s, (int64_t)(b - m.item_blocks) * kSlots + threadIdx.x / G, g * VEC,
                          g * VEC < m.s.k);
    }
}

template <int VEC, int G, int U>
__global__ __launch_bounds__(kBlock) void mf_kernel(MfParams f) {
    const int row_blocks = f.rows.item_blocks + f.rows.empty_blocks;
    double lsum = 0.0;
    if ((int)blockIdx.x < row_blocks) mf_block<VEC, G, U>(f.rows, blockIdx.x, true, lsum);
    else mf_block<VEC, G, U>(f.cols, (int)blockIdx.x - row_blocks, false, lsum);
    const double t = block_sum(lsum);
    if (threadIdx.x == 0) f.loss_part[blockIdx.x] = t;
}

template <int G>
constexpr int mf_unroll_c() {
    return G >= 4 ? 4 : (G == 1 ? 4 : G);
}

int64_t mf_blocks(const nsd_plan &rows, const nsd_plan &cols, int k, bool vec) {
    const WidthPlan wp = width_plan(k, vec);
    const int slots = kBlock / wp.g;
    return ceil_div(rows.nitems, slots) + ceil_div(rows.nempty, slots) +
           ceil_div(cols.nitems, slots) + ceil_div(cols.nempty, slots);
}

template <int VEC, int G>
static nsd_status launch_mf(MfParams f, double *loss, hipStream_t st) {
    constexpr int kSlots = kBlock / G;
    for (MfPass *m : {&f.rows, &f.cols}) {
        m->item_blocks = (int32_t)ceil_div(m->s.plan.nitems, kSlots);
        m->empty_blocks = (int32_t)ceil_div(m->s.plan.nempty, kSlots);
    }
    const int grid = f.rows.item_blocks + f.rows.empty_blocks + f.cols.item_blocks +
                     f.cols.empty_blocks;
    if (grid == 0) return loss_finalize(f.loss_part, 0, loss, st);
    probe_begin(NSD_KERNEL_MF, st);
    mf_kernel<VEC, G, mf_unroll_c<G>()><<<grid, kBlock, 0, st>>>(f);
    probe_end(NSD_KERNEL_MF, st);
    NSD_TRY(check_launch("mf_kernel"));
    NSD_TRY((launch_fix<VEC, G>(f.rows.s, nullptr, 0.0, st)));
    NSD_TRY((launch_fix<VEC, G>(f.cols.s, nullptr, 0.0, st)));
    return loss_finalize(f.loss_part, grid, loss, st);
}

struct MfLauncher {
    MfParams f;
    double *loss;
    hipStream_t st;
    template <int VEC, int G>
    nsd_status operator()() { return launch_mf<VEC, G>(f, loss, st); }
};

bool mf_vec_ok(int k, const void *U, const void *V, const void *dU, const void *dV) {
    return k % 4 == 0 && aligned16(U) && aligned16(V) && aligned16(dU) && aligned16(dV);
}

nsd_status mf_fused(MfParams f, double *loss, hipStream_t st) {
    const bool vec = mf_vec_ok(f.rows.s.k, f.rows.own, f.cols.own, f.rows.s.out, f.cols.s.out);
    MfLauncher fn{f, loss, st};
    return dispatch_width(width_plan(f.rows.s.k, vec), fn);
}

}  // namespace nsd
