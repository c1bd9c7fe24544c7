// Segment passes that use the segment's own dense row: one gather per entry
// serves both a sampled dot product and a gather-reduce.
//
// A pass walks a sorted sparse operand over its work plan (segments = the
// rows of a CSR, or the columns of its CSC).  For entry p of segment s, with
// gathered row X[idx_p] and the segment's own row O[s]:
//     d_p = <O[s], X[idx_p]>                  (reduced across the slot's lanes)
//     out[s] = alpha * sum_{p in s} c_p X[idx_p]
// where the coefficient c_p depends on the kind of pass:
//   linear (kDualLin):   c_p = w_p; optionally sdd[pos_p] = sdd_alpha * d_p
//                        and loss += w_p d_p.  With O = B, X = C = A B over
//                        A's columns this is dB = A^T C together with
//                        dA = <C_i, B_j> of L = 1/2 ||A B||^2; with O = H,
//                        X = G it is the whole bilinear layer
//                        L = sum (A H) o G: dA = <G_i, H_j>, dH = A^T G.
//   residual (kDualMf):  c_p = r_p = w_p - d_p, loss += r_p^2: the row and
//                        column passes of sparse matrix factorisation.
// These are the paper's sums over the stored keys of A with the dense rows
// looked up by key (Logical SDQLite, Section 3); the sampled product keeps
// the gradient of A on A's keys (Section 4.2), the `+=` of the code
// generation (Section 5.5) becomes a fixed-order segmented sum.
//
// pos_p is the entry's position in the sparse operand's storage order
// (perm[p] for a CSC pass), so the sampled product is written aligned with
// A's own pattern.  Up to two passes share one launch on disjoint block
// ranges; long segments leave chunk partials combined by the shared kernel.
#include "nsd_internal.hpp"
#include "segreduce.hpp"
#include "segreduce_dev.hpp"

namespace nsd {

// State of one slot walking one work item: the open segment, its sum, and
// the per-batch arithmetic shared by both ways of fetching entry metadata.
template <int KIND, int VEC, int G, int U>
struct DualSlot {
    const DualPass &m;
    int64_t s, k, b0;
    int lane, g, col;
    bool on;
    int row;
    bool carry;    // the open segment started before this item (a later chunk)
    bool pend = false;  // acc is a chunk partial of segment `row`, not yet stored
    Vec<VEC> acc;
    Vec<VEC> ownv; // own[row] when kKeepOwn: the open segment's own dense row
    double &lsum;

    // Keeping the open segment's own row pays for slots of 32 lanes or more
    // (measured on MI355X: full-wave slots and the 32-lane slots of k = 128);
    // with four slots per wave the branches on segment boundaries diverge
    // more, and per-entry loads (L1 hits) measured faster.  Build-time knob:
    // NSD_KEEP_OWN_MIN.
#ifdef NSD_KEEP_OWN_MIN
    static constexpr bool kKeepOwn = G >= NSD_KEEP_OWN_MIN;
#else
    static constexpr bool kKeepOwn = G >= 32;
#endif

    __device__ __forceinline__ DualSlot(const DualPass &m_, int64_t s_, int lane_, double &ls)
        : m(m_), s(s_), k(m_.s.k), lane(lane_), g(lane_ % G), col((lane_ % G) * VEC), lsum(ls) {
        const SgrParams &a = m.s;
        on = col < a.k;  // k <= G * VEC on this path
        const int64_t a0 = a.plan.item_ptr[s];
        b0 = a.plan.item_ptr[s + 1];
        row = a.segidx[a0];
        carry = a0 > 0 && a.segidx[a0 - 1] == row;
        acc.zero();
        if (kKeepOwn && on) ownv.load_nt(m.own + (int64_t)row * k + col);
        else ownv.zero();
    }

    __device__ __forceinline__ void flush() {
        if (carry) {
            pend = true;  // a chunk item holds one segment: this is its end
        } else if (on) {
            Vec<VEC> t = acc;
            t.scale(m.s.alpha);
            t.store_nt(m.s.out + (int64_t)row * k + col);  // written once
        }
    }

    // Entries [p, p + U) with metadata r, c, pos, w (padding past b0 has
    // weight 0, the last entry's segment and gathered row).
    // For a linear pass with G > 1, ps / ws are the position and weight of
    // entry g / (G / U) of the batch, the one whose dot product this lane
    // ends up holding.
    __device__ __forceinline__ void batch(int64_t p, const int (&r)[U], const int (&c)[U],
                                          const int (&pos)[U], const float (&w)[U], int ps,
                                          float ws) {
        const SgrParams &a = m.s;
        Vec<VEC> xv[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (on) {
                if (a.X) xv[u].load(a.X + (int64_t)c[u] * k + col);
                else xv[u].ones();
            } else {
                xv[u].zero();
            }
        }
        float d[U];
        if constexpr (kKeepOwn) {
            // the open segment's own row is kept; a batch that ends in
            // another segment loads that one (ownn); an entry in neither (a
            // segment that starts and ends inside the batch) loads its own
            const bool same = r[U - 1] == row;  // segments are sorted in an item
            Vec<VEC> ownn = ownv;
            if (!same && on) ownn.load_nt(m.own + (int64_t)r[U - 1] * k + col);
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if (!on) {
                    d[u] = 0.f;
                } else if (r[u] == row) {
                    d[u] = ownv.dot(xv[u]);
                } else if (r[u] == r[U - 1]) {
                    d[u] = ownn.dot(xv[u]);
                } else {
                    Vec<VEC> o;
                    o.load(m.own + (int64_t)r[u] * k + col);
                    d[u] = o.dot(xv[u]);
                }
            }
            ownv = ownn;  // own row of the last entry's segment
        } else {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                Vec<VEC> o;
                if (on) o.load(m.own + (int64_t)r[u] * k + col);
                else o.zero();
                d[u] = o.dot(xv[u]);
            }
        }
        float coef[U];
        if constexpr (KIND == kDualMf) {
            if constexpr (G == 1) {
#pragma unroll
                for (int u = 0; u < U; ++u) coef[u] = p + u < b0 ? w[u] - d[u] : 0.f;
            } else {
                float t[U];
                slot_totals<G, U>(transpose_reduce<G, U>(d, lane), lane, t);
#pragma unroll
                for (int u = 0; u < U; ++u) coef[u] = p + u < b0 ? w[u] - t[u] : 0.f;
            }
            if (m.count_loss && g == 0)
#pragma unroll
                for (int u = 0; u < U; ++u) lsum += (double)coef[u] * coef[u];
        } else {
#pragma unroll
            for (int u = 0; u < U; ++u) coef[u] = w[u];  // 0 on padding
            if constexpr (G == 1) {
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    if (p + u < b0) {
                        if (m.sdd) m.sdd[pos[u]] = m.sdd_alpha * d[u];
                        if (m.count_loss) lsum += (double)w[u] * d[u];
                    }
                }
            } else {
                const float tot = transpose_reduce<G, U>(d, lane);
                constexpr int kRep = G / U;
                const int us = g / kRep;  // the entry whose total this lane holds
                if (g % kRep == 0 && p + us < b0) {
                    if (m.sdd) m.sdd[ps] = m.sdd_alpha * tot;
                    if (m.count_loss) lsum += (double)ws * tot;
                }
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
            acc.fma(coef[u], xv[u]);
        }
    }

    __device__ __forceinline__ void finish() {
        const SgrParams &a = m.s;
        if (b0 == a.nnz || a.segidx[b0] != row) flush();
        else pend = true;  // a chunk of a long segment that goes on
    }
};

// Walks item s; returns the segment of the chunk partial left in `part_acc`
// (stored with store_chunk_partial), or -1.
template <int KIND, int VEC, int G, int U>
__device__ __forceinline__ int dual_walk(const DualPass &m, int64_t s, int lane, double &lsum,
                                         Vec<VEC> &part_acc) {
    DualSlot<KIND, VEC, G, U> st(m, s, lane, lsum);
    walk_item<G, U>(m.s, m.s.plan.item_ptr[s], st.b0, st.g, st);
    st.finish();
    part_acc = st.acc;
    return st.pend ? st.row : -1;
}

template <int KIND, int VEC, int G, int U>
__device__ __forceinline__ void dual_block(const DualPass &m, int b, double &lsum) {
    constexpr int kSlots = kBlock / G;
    const int lane = threadIdx.x % kWave;
    const int g = threadIdx.x % G;
    if (b < m.item_blocks) {
        const int64_t s = (int64_t)b * kSlots + threadIdx.x / G;
        Vec<VEC> pacc;
        pacc.zero();
        int pseg = -1;
        if (s < m.s.plan.nitems) pseg = dual_walk<KIND, VEC, G, U>(m, s, lane, lsum, pacc);
        store_chunk_partial<VEC, G>(pseg, pacc, m.s.part, m.s.plan.chunk_ord, s, m.s.k, g * VEC,
                                    g * VEC < m.s.k);
    } else {
        zero_segment<VEC>(m.s, (int64_t)(b - m.item_blocks) * kSlots + threadIdx.x / G, g * VEC,
                          g * VEC < m.s.k);
    }
}

// Occupancy floor (waves per SIMD), a build-time tuning knob.
#ifdef NSD_DUAL_WAVES
#define NSD_DUAL_OCCUPANCY __attribute__((amdgpu_waves_per_eu(NSD_DUAL_WAVES, 8)))
#else
#define NSD_DUAL_OCCUPANCY
#endif

template <int KIND, int VEC, int G, int U>
__global__ __launch_bounds__(kBlock) NSD_DUAL_OCCUPANCY void dual_kernel(DualParams f) {
    if (f.early.loss && blockIdx.x == gridDim.x - 1) {
        loss_total_block<4>(f.early);  // a few thousand row partials; keeps VGPRs low
        return;
    }
    const int first = f.pass[0].item_blocks + f.pass[0].empty_blocks;
    double lsum = 0.0;
    if ((int)blockIdx.x < first) dual_block<KIND, VEC, G, U>(f.pass[0], blockIdx.x, lsum);
    else dual_block<KIND, VEC, G, U>(f.pass[1], (int)blockIdx.x - first, lsum);
    if (f.loss_part) {
        const double t = block_sum(lsum);
        if (threadIdx.x == 0) f.loss_part[blockIdx.x] = f.loss_beta * t;
    }
}

template <int G>
constexpr int dual_unroll() {
#ifdef NSD_DUAL_UNROLL
    return reduce_unroll<G, NSD_DUAL_UNROLL>();
#else
    // measured on MI355X: eight entries per batch for full-wave slots
    // (k > 128), four for 32- and 16-lane slots (the SpMM column pass at
    // k = 64: 54.8 us against 57.6 with two, 62.5 with eight), two for
    // narrower ones, four for single-lane slots
    return reduce_unroll<G, G >= 64 ? 8 : (G >= 16 || G == 1 ? 4 : 2)>();
#endif
}

int64_t dual_blocks(const nsd_plan *const *plans, int npass, int k, bool vec) {
    const WidthPlan wp = width_plan(k, vec);
    const int slots = kBlock / wp.g;
    int64_t n = 0;
    for (int i = 0; i < npass; ++i)
        n += ceil_div(plans[i]->nitems, slots) + ceil_div(plans[i]->nempty, slots);
    return n;
}

template <int KIND, int VEC, int G>
static nsd_status launch_dual(DualParams f, int probe_id, LossJob job, hipStream_t st) {
    constexpr int kSlots = kBlock / G;
    int64_t grid = 0;
    for (int i = 0; i < 2; ++i) {
        DualPass &m = f.pass[i];
        if (i >= f.npass) {
            m.item_blocks = m.empty_blocks = 0;
            continue;
        }
        m.item_blocks = (int32_t)ceil_div(m.s.plan.nitems, kSlots);
        m.empty_blocks = (int32_t)ceil_div(m.s.plan.nempty, kSlots);
        m.s.chunk_stride = chunk_group<G>();
        grid += m.item_blocks + m.empty_blocks;
    }
    if (job.loss && !job.p1) {
        job.p1 = f.loss_part;
        job.n1 = grid;
    }
    const int64_t launch = grid + (f.early.loss ? 1 : 0);
    if (launch > 0) {
        probe_begin(probe_id, st);
        dual_kernel<KIND, VEC, G, dual_unroll<G>()><<<(unsigned)launch, kBlock, 0, st>>>(f);
        probe_end(probe_id, st);
        NSD_TRY(check_launch("dual_kernel"));
    }
    FixJobs fx;
    for (int i = 0; i < f.npass; ++i) add_fix(fx, f.pass[i].s);
    fx.loss = job;
    return launch_fixes<VEC, G>(fx, st);
}

template <int KIND>
struct DualLauncher {
    DualParams f;
    int probe_id;
    LossJob job;
    hipStream_t st;
    template <int VEC, int G>
    nsd_status operator()() { return launch_dual<KIND, VEC, G>(f, probe_id, job, st); }
};

bool dual_vec_ok(const DualParams &f) {
    bool ok = f.pass[0].s.k % 4 == 0;
    for (int i = 0; i < f.npass; ++i) {
        const DualPass &m = f.pass[i];
        ok = ok && aligned16(m.own) && aligned16(m.s.out) && (!m.s.X || aligned16(m.s.X));
    }
    return ok;
}

bool dual_supported(int k, bool vec) { return vec ? k <= 256 : k <= 64; }

nsd_status dual_fused(int kind, DualParams f, int probe_id, LossJob job, hipStream_t st) {
    const bool vec = dual_vec_ok(f);
    const WidthPlan wp = width_plan(f.pass[0].s.k, vec);
    if (!dual_supported(f.pass[0].s.k, vec))
        return fail(NSD_ERR_UNSUPPORTED, "dense width k = %d on a fused pass", f.pass[0].s.k);
    if (kind == kDualMf) {
        DualLauncher<kDualMf> fn{f, probe_id, job, st};
        return dispatch_width(wp, fn);
    }
    DualLauncher<kDualLin> fn{f, probe_id, job, st};
    return dispatch_width(wp, fn);
}

}  // namespace nsd
