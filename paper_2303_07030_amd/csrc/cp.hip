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

// State of one slot walking one work item of a mode pass.
template <int VEC, int G, int U>
struct CpSlot {
    const CpMode &m;
    int64_t s, k, b0;
    int lane, g, col;
    bool on, first_mode;
    int row;
    bool carry;     // the open segment started before this item (a later chunk)
    bool pend = false;  // acc is a chunk partial of segment `row`, not yet stored
    Vec<VEC> acc;   // sum of R * (fa o fb) over the open segment
    Vec<VEC> ownv;  // own[row]: the open segment's own factor row
    double &lsum;

    __device__ __forceinline__ CpSlot(const CpMode &m_, int64_t s_, int lane_, bool fm,
                                      double &ls)
        : m(m_), s(s_), k(m_.s.k), lane(lane_), g(lane_ % G), col((lane_ % G) * VEC),
          first_mode(fm), lsum(ls) {
        const SgrParams &a = m.s;
        on = col < a.k;  // rank <= G * VEC
        const int64_t a0 = a.plan.item_ptr[s];
        b0 = a.plan.item_ptr[s + 1];
        row = a.segidx[a0];
        carry = a0 > 0 && a.segidx[a0 - 1] == row;
        acc.zero();
        if (on) ownv.load(m.own + (int64_t)row * k + col);
        else ownv.zero();
    }

    __device__ __forceinline__ void flush() {
        if (carry) {
            pend = true;  // a chunk item holds one segment: this is its end
        } else if (on) {
            Vec<VEC> t = acc;
            t.scale(m.s.alpha);
            t.store(m.s.out + (int64_t)row * k + col);
        }
    }

    // Entries [p, p + U): segment r, coordinates ca / cb of the two other
    // modes, value x, input position pp (padding past b0 repeats the last
    // entry; its residual is zeroed here).
    __device__ __forceinline__ void batch(int64_t p, const int (&r)[U], const int (&ca)[U],
                                          const int (&cb)[U], const float (&x)[U],
                                          const int (&pp)[U]) {
        // segments are long in most tensors: the own row is reused while the
        // whole batch stays in the open segment, else loaded per entry
        bool same = true;
#pragma unroll
        for (int u = 0; u < U; ++u) same = same && r[u] == row;
        // Every load of the batch is issued before any of them is used: the
        // addresses are always valid (a lane past the rank reads column 0 and
        // its data is dropped), so no load sits in a branch that must wait.
        const int cl = on ? col : 0;
        Vec<VEC> t[U], fb[U], ow[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            t[u].load(m.fa + (int64_t)ca[u] * k + cl);
            fb[u].load(m.fb + (int64_t)cb[u] * k + cl);
        }
        if (!same) {
#pragma unroll
            for (int u = 0; u < U; ++u) ow[u].load(m.own + (int64_t)r[u] * k + cl);
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
#pragma unroll
            for (int e = 0; e < VEC; ++e) t[u].v[e] = on ? t[u].v[e] * fb[u].v[e] : 0.f;
        }
        float d[U];
#pragma unroll
        for (int u = 0; u < U; ++u) d[u] = (same || !on) ? ownv.dot(t[u]) : ow[u].dot(t[u]);
        float res[U];
        if constexpr (G == 1) {
#pragma unroll
            for (int u = 0; u < U; ++u) res[u] = p + u < b0 ? x[u] - d[u] : 0.f;
        } else {
            float mv[U];
            slot_totals<G, U>(transpose_reduce<G, U>(d, lane), lane, mv);
#pragma unroll
            for (int u = 0; u < U; ++u) res[u] = p + u < b0 ? x[u] - mv[u] : 0.f;
        }
        if (first_mode && g == 0) {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if (p + u < b0) {
                    m.resid[pp[u]] = m.seed * res[u];
                    lsum += 0.5 * (double)res[u] * res[u];
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
            acc.fma(res[u], t[u]);
        }
        if (!same && on) ownv = ow[U - 1];  // own row of the segment now open
    }

    __device__ __forceinline__ void finish() {
        const SgrParams &a = m.s;
        if (b0 == a.nnz || a.segidx[b0] != row) flush();
        else pend = true;  // a chunk of a long segment that goes on
    }
};

// One slot's walk over item s of a mode pass.  Slots of 8 or more lanes read
// the entries' metadata in tiles of G (lane g loads entry g of a tile, each
// batch takes its fields by broadcast); narrow slots load them per entry.
// The next tile's (batch's) metadata is in flight under the current one.
template <int VEC, int G, int U>
__device__ __forceinline__ int cp_walk(const CpMode &m, int64_t s, int lane, bool first_mode,
                                       double &lsum, Vec<VEC> &part_acc) {
    const SgrParams &a = m.s;
    CpSlot<VEC, G, U> st(m, s, lane, first_mode, lsum);
    const int64_t a0 = a.plan.item_ptr[s], b0 = st.b0;
    // Fields of entry q; past the item they are those of its last entry
    // (every load unconditional, so none is consumed before its batch); the
    // batch zeroes the padding's residual by position.
    auto fields = [&](int64_t q, int &r, int &ca, int &cb, float &x, int &pp) {
        const int64_t qc = min(q, b0 - 1);
        r = a.segidx[qc];
        ca = a.idx[qc];
        cb = m.idx_b[qc];
        x = a.w[qc];
        pp = first_mode ? m.perm[qc] : 0;
    };
    if constexpr (G >= 8) {
        static_assert(G % U == 0, "a tile holds whole batches");
        const int g = st.g;
        int tr, ta, tb, tp, nr = 0, na = 0, nb = 0, np = 0;
        float tx, nx = 0.f;
        fields(a0 + g, tr, ta, tb, tx, tp);
        for (int64_t t = a0; t < b0; t += G) {
            if (t + G < b0) fields(t + G + g, nr, na, nb, nx, np);
            for (int base = 0; base < G && t + base < b0; base += U) {
                int r[U], ca[U], cb[U], pp[U];
                float x[U];
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    r[u] = slot_bcast<G>(tr, base + u);
                    ca[u] = slot_bcast<G>(ta, base + u);
                    cb[u] = slot_bcast<G>(tb, base + u);
                    x[u] = slot_bcast<G>(tx, base + u);
                    pp[u] = first_mode ? slot_bcast<G>(tp, base + u) : 0;
                }
                st.batch(t + base, r, ca, cb, x, pp);
            }
            tr = nr;
            ta = na;
            tb = nb;
            tx = nx;
            tp = np;
        }
    } else {
        int r[U], ca[U], cb[U], pp[U], nr[U], na[U], nb[U], np[U];
        float x[U], nx[U];
#pragma unroll
        for (int u = 0; u < U; ++u) fields(a0 + u, r[u], ca[u], cb[u], x[u], pp[u]);
        for (int64_t p = a0; p < b0; p += U) {
            if (p + U < b0)
#pragma unroll
                for (int u = 0; u < U; ++u) fields(p + U + u, nr[u], na[u], nb[u], nx[u], np[u]);
            st.batch(p, r, ca, cb, x, pp);
#pragma unroll
            for (int u = 0; u < U; ++u) {
                r[u] = nr[u];
                ca[u] = na[u];
                cb[u] = nb[u];
                x[u] = nx[u];
                pp[u] = np[u];
            }
        }
    }
    st.finish();
    part_acc = st.acc;
    return st.pend ? st.row : -1;  // a chunk partial, stored by store_chunk_partial
}

template <int VEC, int G, int U>
__device__ __forceinline__ void cp_block(const CpMode &m, int b, bool first_mode, double &lsum) {
    constexpr int kSlots = kBlock / G;
    const int lane = threadIdx.x % kWave;
    const int g = threadIdx.x % G;
    if (b < m.item_blocks) {
        const int64_t s = (int64_t)b * kSlots + threadIdx.x / G;
        Vec<VEC> pacc;
        pacc.zero();
        int pseg = -1;
        if (s < m.s.plan.nitems) pseg = cp_walk<VEC, G, U>(m, s, lane, first_mode, lsum, pacc);
        store_chunk_partial<VEC, G>(pseg, pacc, m.s.part, m.s.plan.chunk_ord, s, m.s.k, g * VEC,
                                    g * VEC < m.s.k);
    } else {
        zero_segment<VEC>(m.s, (int64_t)(b - m.item_blocks) * kSlots + threadIdx.x / G, g * VEC,
                          g * VEC < m.s.k);
    }
}

// Occupancy floor (waves per SIMD), a build-time tuning knob.
#ifdef NSD_CP_WAVES
#define NSD_CP_OCCUPANCY __attribute__((amdgpu_waves_per_eu(NSD_CP_WAVES, 8)))
#else
#define NSD_CP_OCCUPANCY
#endif

template <int VEC, int G, int U>
__global__ __launch_bounds__(kBlock) NSD_CP_OCCUPANCY void cp_kernel(CpParams f) {
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
    // measured on MI355X (rank 32): two entries per batch beat four and eight
    return reduce_unroll<G, (G >= 64 || G == 1) ? 4 : 2>();
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
        f.m[i].s.chunk_stride = chunk_group<G>();
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
    FixJobs fx;
    for (int i = 0; i < 3; ++i) add_fix(fx, f.m[i].s);
    fx.loss = job;
    return launch_fixes<VEC, G>(fx, st);
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
