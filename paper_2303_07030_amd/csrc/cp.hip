// Fused loss and gradients of a rank-R CP model of a sparse 3-tensor X:
//   m_ijl = sum_r F1[i,r] F2[j,r] F3[l,r],  R_ijl = X_ijl - m_ijl on X's keys
//   L = 1/2 sum over stored (i, j, l) of R_ijl^2
//   dX on X's keys = seed * R                    (written in X's input order)
//   dF1[i,:] = -seed sum R_ijl (F2[j,:] o F3[l,:])   and cyclically for
//   dF2 and dF3: the negated mode-n MTTKRPs of R.
// X is an order-3 `tensor` of the paper (nested dictionaries, Section 3); the
// factor gradients come from its tensorized AD applied to the sum over X's
// stored keys, so they stay O(nnz) (Section 4.2).
//
// The three mode passes run in one launch on disjoint block ranges.  Pass n
// walks X sorted by the mode-n coordinate (a mode index, built once), over
// that mode's work plan: per entry it gathers the two other factor rows
// (small, cache-resident), forms their elementwise product t, reduces
// <F_n[seg], t> across the slot's lanes to get R, and accumulates R * t into
// the segment's gradient row; long segments leave chunk partials combined by
// the shared kernel.  Pass 0 also writes the residual through the mode's
// permutation and counts the loss.
#include "nsd_internal.hpp"
#include "segreduce.hpp"
#include "segreduce_dev.hpp"

namespace nsd {

template <int U>
struct CpMeta {
    int r[U], ca[U], cb[U], pp[U];
    float x[U];
};

template <int U>
__device__ __forceinline__ void cp_meta(const CpMode &m, int64_t p, int64_t b0, int last_r,
                                        int last_a, int last_b, bool with_perm, CpMeta<U> &t) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int64_t q = p + u;
        if (q < b0) {
            t.r[u] = m.s.segidx[q];
            t.ca[u] = m.s.idx[q];
            t.cb[u] = m.idx_b[q];
            t.x[u] = m.s.w[q];
            t.pp[u] = with_perm ? m.perm[q] : 0;
        } else {
            t.r[u] = last_r;
            t.ca[u] = last_a;
            t.cb[u] = last_b;
            t.x[u] = 0.f;
            t.pp[u] = 0;
        }
    }
}

template <int VEC, int G, int U>
__device__ __forceinline__ void cp_walk(const CpMode &m, int64_t s, int lane, bool first_mode,
                                        double &lsum) {
    const SgrParams &a = m.s;
    const int g = lane % G;
    const int col = g * VEC;  // rank <= G * VEC
    const bool on = col < a.k;
    const int64_t k = a.k;
    const int64_t a0 = a.plan.item_ptr[s];
    const int64_t b0 = a.plan.item_ptr[s + 1];
    const int last_r = a.segidx[b0 - 1], last_a = a.idx[b0 - 1], last_b = m.idx_b[b0 - 1];
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

    CpMeta<U> cur, nxt;
    cp_meta(m, a0, b0, last_r, last_a, last_b, first_mode, cur);
    for (int64_t p = a0; p < b0; p += U) {
        if (p + U < b0) cp_meta(m, p + U, b0, last_r, last_a, last_b, first_mode, nxt);
        Vec<VEC> t[U], ow[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (on) {
                Vec<VEC> fb;
                t[u].load(m.fa + (int64_t)cur.ca[u] * k + col);
                fb.load(m.fb + (int64_t)cur.cb[u] * k + col);
                ow[u].load(m.own + (int64_t)cur.r[u] * k + col);
#pragma unroll
                for (int e = 0; e < VEC; ++e) t[u].v[e] *= fb.v[e];
            } else {
                t[u].zero();
                ow[u].zero();
            }
        }
        float d[U];
#pragma unroll
        for (int u = 0; u < U; ++u) d[u] = ow[u].dot(t[u]);
        float res[U];
        if constexpr (G == 1) {
#pragma unroll
            for (int u = 0; u < U; ++u) res[u] = p + u < b0 ? cur.x[u] - d[u] : 0.f;
        } else {
            const float tot = transpose_reduce<G, U>(d, lane);
            constexpr int kRep = G / U;
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const float mv = __shfl(tot, u * kRep, G);
                res[u] = p + u < b0 ? cur.x[u] - mv : 0.f;
            }
        }
        if (first_mode && g == 0) {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if (p + u < b0) {
                    m.resid[cur.pp[u]] = m.seed * res[u];
                    lsum += 0.5 * (double)res[u] * res[u];
                }
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (cur.r[u] != row) {
                flush();
                row = cur.r[u];
                carry = false;
                acc.zero();
            }
            acc.fma(res[u], t[u]);
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
__device__ __forceinline__ void cp_block(const CpMode &m, int b, bool first_mode, double &lsum) {
    constexpr int kSlots = kBlock / G;
    const int lane = threadIdx.x % kWave;
    const int g = threadIdx.x % G;
    if (b < m.item_blocks) {
        const int64_t s = (int64_t)b * kSlots + threadIdx.x / G;
        if (s < m.s.plan.nitems) cp_walk<VEC, G, U>(m, s, lane, first_mode, lsum);
    } else {
        zero_segment<VEC>(m.s, (int64_t)(b - m.item_blocks) * kSlots + threadIdx.x / G, g * VEC,
                          g * VEC < m.s.k);
    }
}

template <int VEC, int G, int U>
__global__ __launch_bounds__(kBlock) void cp_kernel(CpParams f) {
    const int b0 = f.m[0].item_blocks + f.m[0].empty_blocks;
    const int b1 = b0 + f.m[1].item_blocks + f.m[1].empty_blocks;
    double lsum = 0.0;
    if ((int)blockIdx.x < b0) cp_block<VEC, G, U>(f.m[0], blockIdx.x, true, lsum);
    else if ((int)blockIdx.x < b1) cp_block<VEC, G, U>(f.m[1], blockIdx.x - b0, false, lsum);
    else cp_block<VEC, G, U>(f.m[2], blockIdx.x - b1, false, lsum);
    const double t = block_sum(lsum);
    if (threadIdx.x == 0) f.loss_part[blockIdx.x] = t;
}

template <int G>
constexpr int cp_unroll() {
#ifdef NSD_CP_UNROLL
    return reduce_unroll<G, NSD_CP_UNROLL>();
#else
    return reduce_unroll<G, 4>();
#endif
}

int64_t cp_blocks(const nsd_plan *plans, int rank, bool vec) {
    const WidthPlan wp = width_plan(rank, vec);
    const int slots = kBlock / wp.g;
    int64_t n = 0;
    for (int i = 0; i < 3; ++i) n += ceil_div(plans[i].nitems, slots) + ceil_div(plans[i].nempty, slots);
    return n;
}

template <int VEC, int G>
static nsd_status launch_cp(CpParams f, double *loss, hipStream_t st) {
    constexpr int kSlots = kBlock / G;
    int grid = 0;
    for (int i = 0; i < 3; ++i) {
        f.m[i].item_blocks = (int32_t)ceil_div(f.m[i].s.plan.nitems, kSlots);
        f.m[i].empty_blocks = (int32_t)ceil_div(f.m[i].s.plan.nempty, kSlots);
        grid += f.m[i].item_blocks + f.m[i].empty_blocks;
    }
    if (grid == 0) return loss_finalize(f.loss_part, 0, loss, st);
    probe_begin(NSD_KERNEL_CP, st);
    cp_kernel<VEC, G, cp_unroll<G>()><<<grid, kBlock, 0, st>>>(f);
    probe_end(NSD_KERNEL_CP, st);
    NSD_TRY(check_launch("cp_kernel"));
    // the loss total rides on the last combine launch
    LossJob job;
    job.p1 = f.loss_part;
    job.n1 = grid;
    job.loss = loss;
    for (int i = 0; i < 3; ++i)
        NSD_TRY((launch_fix<VEC, G>(f.m[i].s, nullptr, 0.0, st, i == 2 ? job : LossJob{})));
    return NSD_OK;
}

struct CpLauncher {
    CpParams f;
    double *loss;
    hipStream_t st;
    template <int VEC, int G>
    nsd_status operator()() { return launch_cp<VEC, G>(f, loss, st); }
};

nsd_status cp_fused(CpParams f, bool vec, double *loss, hipStream_t st) {
    CpLauncher fn{f, loss, st};
    return dispatch_width(width_plan(f.m[0].s.k, vec), fn);
}

}  // namespace nsd
