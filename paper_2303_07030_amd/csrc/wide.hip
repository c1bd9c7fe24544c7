// Wide-rank form of the factorisation and CP losses: any rank, also above
// what one slot of the fused kernels holds (256 columns with 16-byte aligned
// rows, 64 otherwise).
//
// The fused kernels recompute an entry's residual in every pass from the
// dense rows they hold in registers; with more columns than a slot holds,
// the residual is formed once instead and the gradient passes read it:
//   1. resid_kernel: for every stored entry p (any storage order),
//        m_p = sum_r prod_n F_n[c_n(p), r],  res_p = x_p - m_p,
//      written unscaled to rbuf[pos_p] (and seed * res_p to the caller's
//      residual output when there is one), lscale * res_p^2 into the block's
//      loss partial.  A slot of a whole wave walks a run of entries, the
//      columns in chunks of the slot's width.
//   2. one gather-reduce per mode over that mode's work plan, the weight of
//      an entry read through the mode's permutation from rbuf:
//        dF_n[s, :] = alpha * sum_{p in s} res_p * (o_{m != n} F_m[c_m(p), :])
//      (for a matrix the ordinary gather-reduce with res as its weights).
//   3. the loss total over the block partials.
// These are the same sums over the stored keys as the fused passes (the
// reverse gradients that the tensorized forward mode of Section 4.2
// computes); only where the residual lives differs.
#include <algorithm>

#include "nsd_internal.hpp"
#include "segreduce.hpp"
#include "segreduce_dev.hpp"
#include "wide.hpp"

namespace nsd {

// ------------------------------------------------------------ residual

template <int N, int VEC, int G, int U>
__global__ __launch_bounds__(kBlock) void resid_kernel(ResidParams a) {
    static_assert(G == kWave, "one slot per wave");
    constexpr int kSlots = kBlock / G;
    const int lane = threadIdx.x % kWave;
    const int g = lane % G;
    const int64_t s = (int64_t)blockIdx.x * kSlots + threadIdx.x / G;
    const int64_t k = a.k;
    double lsum = 0.0;
    if (s < a.nslots) {
        const int64_t a0 = s * a.L;
        const int64_t b0 = min(a0 + (int64_t)a.L, (int64_t)a.nnz);
        for (int64_t p = a0; p < b0; p += U) {
            int c[U][N];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int64_t q = min(p + u, b0 - 1);  // padding repeats the last entry
#pragma unroll
                for (int n = 0; n < N; ++n) c[u][n] = a.coord[n][q];
            }
            float part[U];
#pragma unroll
            for (int u = 0; u < U; ++u) part[u] = 0.f;
            for (int c0 = 0; c0 < a.k; c0 += G * VEC) {
                const int col = c0 + g * VEC;
                if (col < a.k) {
                    Vec<VEC> t[U];
#pragma unroll
                    for (int u = 0; u < U; ++u) t[u].load(a.fac[0] + (int64_t)c[u][0] * k + col);
#pragma unroll
                    for (int n = 1; n < N; ++n) {
#pragma unroll
                        for (int u = 0; u < U; ++u) {
                            Vec<VEC> f;
                            f.load(a.fac[n] + (int64_t)c[u][n] * k + col);
#pragma unroll
                            for (int e = 0; e < VEC; ++e) t[u].v[e] *= f.v[e];
                        }
                    }
#pragma unroll
                    for (int u = 0; u < U; ++u)
#pragma unroll
                        for (int e = 0; e < VEC; ++e) part[u] += t[u].v[e];
                }
            }
            // lane g ends with the model value of entry g / (G / U)
            const float m = transpose_reduce<G, U>(part, lane);
            constexpr int kRep = G / U;
            const int64_t q = p + g / kRep;
            if (g % kRep == 0 && q < b0) {
                const float r = a.x[q] - m;
                const int64_t pos = a.perm ? a.perm[q] : q;
                a.rbuf[pos] = r;
                if (a.resid) a.resid[pos] = a.seed * r;
                lsum += a.lscale * (double)r * r;
            }
        }
    }
    const double t = block_sum(lsum);
    if (threadIdx.x == 0) a.part[blockIdx.x] = t;
}

template <int N, int VEC>
static nsd_status launch_resid(ResidParams a, int64_t nblocks, hipStream_t st) {
    resid_kernel<N, VEC, kWave, 4><<<(unsigned)nblocks, kBlock, 0, st>>>(a);
    return check_launch("resid_kernel");
}

template <int VEC>
static nsd_status resid_order(ResidParams a, int64_t nblocks, hipStream_t st) {
    switch (a.order) {
        case 2: return launch_resid<2, VEC>(a, nblocks, st);
        case 3: return launch_resid<3, VEC>(a, nblocks, st);
        case 4: return launch_resid<4, VEC>(a, nblocks, st);
        case 5: return launch_resid<5, VEC>(a, nblocks, st);
        default: return launch_resid<6, VEC>(a, nblocks, st);
    }
}

int64_t resid_blocks(int64_t nnz, int k, bool vec) { return sddmm_shape(nnz, k, vec).nblocks; }

nsd_status resid_pass(ResidParams a, bool vec, hipStream_t st) {
    const SddmmShape sh = sddmm_shape(a.nnz, a.k, vec);
    if (sh.nblocks == 0) return NSD_OK;
    if (sh.wp.g != kWave)
        return fail(NSD_ERR_UNSUPPORTED, "residual pass of width %d below one wave", a.k);
    a.L = sh.L;
    a.nslots = (int32_t)sh.nslots;
    return sh.wp.vec == 4 ? resid_order<4>(a, sh.nblocks, st) : resid_order<1>(a, sh.nblocks, st);
}

// ------------------------------------------------------ mode gather-reduce

// One slot's gather-reduce over an item of a mode pass whose gathered row is
// the elementwise product of N-1 factor rows (the first coordinate comes
// from the walk, the others are read per batch).
template <int N, int VEC, int G, int U>
struct MttkrpSlot {
    const MttkrpParams &m;
    int64_t k, b0;
    int col;
    bool on;
    int row;
    bool carry;
    bool pend = false;  // acc is a chunk partial of segment `row`, not yet stored
    Vec<VEC> acc;

    __device__ __forceinline__ MttkrpSlot(const MttkrpParams &m_, int64_t a0, int64_t b0_, int col_)
        : m(m_), k(m_.s.k), b0(b0_), col(col_) {
        on = col < m.s.k;
        row = m.s.segidx[a0];
        carry = a0 > 0 && m.s.segidx[a0 - 1] == row;
        acc.zero();
    }

    __device__ __forceinline__ void flush() {
        if (carry) {
            pend = true;
        } else if (on) {
            Vec<VEC> t = acc;
            t.scale(m.s.alpha);
            t.store(m.s.out + (int64_t)row * k + col);
        }
    }

    __device__ __forceinline__ void batch(int64_t p, const int (&r)[U], const int (&c)[U],
                                          const int (&)[U], const float (&w)[U], int, float) {
        const int cl = on ? col : 0;  // lanes past the width read column 0, dropped
        Vec<VEC> t[U];
#pragma unroll
        for (int u = 0; u < U; ++u) t[u].load(m.fac[0] + (int64_t)c[u] * k + cl);
#pragma unroll
        for (int o = 1; o < N - 1; ++o) {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int64_t q = min(p + u, b0 - 1);
                Vec<VEC> f;
                f.load(m.fac[o] + (int64_t)m.other[o][q] * k + cl);
#pragma unroll
                for (int e = 0; e < VEC; ++e) t[u].v[e] *= f.v[e];
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (r[u] != row) {
                flush();
                row = r[u];
                carry = false;
                acc.zero();
            }
            acc.fma(w[u], t[u]);  // w is 0 on padding
        }
    }

    __device__ __forceinline__ void finish() {
        if (b0 == m.s.nnz || m.s.segidx[b0] != row) flush();
        else pend = true;
    }
};

template <int N, int VEC, int G, int U>
__global__ __launch_bounds__(kBlock) void mttkrp_kernel(MttkrpParams m) {
    constexpr int kSlots = kBlock / G;
    const SgrParams &a = m.s;
    const int g = threadIdx.x % G;
    const int col = blockIdx.y * (G * VEC) + g * VEC;
    const bool on = col < a.k;
    if ((int)blockIdx.x >= a.item_blocks) {
        zero_segment<VEC>(a, (int64_t)(blockIdx.x - a.item_blocks) * kSlots + threadIdx.x / G,
                          col, on);
        return;
    }
    const int64_t s = (int64_t)blockIdx.x * kSlots + threadIdx.x / G;
    Vec<VEC> pacc;
    pacc.zero();
    int pseg = -1;
    if (s < a.plan.nitems) {
        const int64_t a0 = a.plan.item_ptr[s], b0 = a.plan.item_ptr[s + 1];
        MttkrpSlot<N, VEC, G, U> st(m, a0, b0, col);
        walk_item<G, U>(a, a0, b0, g, st);
        st.finish();
        pacc = st.acc;
        pseg = st.pend ? st.row : -1;
    }
    store_chunk_partial<VEC, G>(pseg, pacc, a.part, a.plan.chunk_ord, s, a.k, col, on);
}

template <int N, int VEC>
static nsd_status launch_mttkrp(MttkrpParams m, hipStream_t st) {
    constexpr int G = kWave;
    constexpr int kSlots = kBlock / G;
    m.s.item_blocks = (int32_t)ceil_div(m.s.plan.nitems, kSlots);
    m.s.chunk_stride = chunk_group<G>();
    const int64_t empty_blocks = ceil_div(m.s.plan.nempty, kSlots);
    dim3 grid((unsigned)(m.s.item_blocks + empty_blocks), (unsigned)ceil_div(m.s.k, G * VEC));
    mttkrp_kernel<N, VEC, G, 4><<<grid, kBlock, 0, st>>>(m);
    NSD_TRY(check_launch("mttkrp_kernel"));
    return launch_fix<VEC, G>(m.s, nullptr, 0.0, st);
}

template <int VEC>
static nsd_status mttkrp_order(MttkrpParams m, int order, hipStream_t st) {
    switch (order) {
        case 3: return launch_mttkrp<3, VEC>(m, st);
        case 4: return launch_mttkrp<4, VEC>(m, st);
        case 5: return launch_mttkrp<5, VEC>(m, st);
        default: return launch_mttkrp<6, VEC>(m, st);
    }
}

nsd_status mttkrp_pass(MttkrpParams m, int order, bool vec, hipStream_t st) {
    if (m.s.nnz == 0) return segreduce(m.s, st);  // zero fill
    const WidthPlan wp = width_plan(m.s.k, vec);
    if (wp.g != kWave)
        return fail(NSD_ERR_UNSUPPORTED, "mode pass of width %d below one wave", m.s.k);
    return wp.vec == 4 ? mttkrp_order<4>(m, order, st) : mttkrp_order<1>(m, order, st);
}

}  // namespace nsd
