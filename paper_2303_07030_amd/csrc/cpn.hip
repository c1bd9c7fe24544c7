// Fused loss and gradients of a rank-R CP model of a sparse order-N tensor X
// (3 <= N <= NSD_MAX_ORDER), the order-N form of the CP gradient:
//   m = sum_r prod_n F_n[c_n, r],  R = x - m on X's keys,  L = 1/2 sum R^2
//   dX on X's keys = seed * R (in X's input order)
//   dF_n[c_n, :] = -seed sum R * (o_{m != n} F_m[c_m, :])  (negated MTTKRPs)
// X is an order-N `tensor` of the paper (N nested dictionaries, Section 3);
// the factor gradients are its tensorized AD over the sum of X's stored keys
// (Section 4.2).
//
// The N mode passes run in one launch on consecutive block ranges.  Pass n
// walks X in mode n's order (a mode index built once per pattern) over the
// mode's work plan; per entry it gathers the N-1 other factor rows, forms
// their elementwise product t, reduces <F_n[seg], t> across the slot's lanes
// to get R, and accumulates R * t into the segment's gradient row.  Entry
// metadata is read in tiles (lane g loads entry g's fields, batches take
// them by broadcast); the open segment's own factor row is kept while a
// batch stays in it.  Pass 0 also writes the residual through the mode's
// permutation and counts the loss.  Long segments leave chunk partials
// combined by the shared kernel.
#include <algorithm>

#include "nsd_internal.hpp"
#include "segreduce.hpp"
#include "segreduce_dev.hpp"
#include "wide.hpp"

namespace nsd {

template <int N>
struct CpnMode {
    SgrParams s;                     // segidx, w = values, out = dF_n, part, plan
    const int32_t *other[N - 1];     // coordinates of modes n+1 .. n+N-1 (mod N)
    const float *own = nullptr;      // F_n
    const float *fac[N - 1];         // F_{n+1} .. F_{n+N-1}
    const int32_t *perm = nullptr;   // input position of each slot (pass 0)
    float *resid = nullptr;          // dX (pass 0)
    float seed = 1.f;
    int32_t fiber = 0;               // other[0] is the fiber coordinate (a run level)
    int32_t item_blocks = 0, empty_blocks = 0;
};

template <int N>
struct CpnParams {
    CpnMode<N> m[N];
    double *loss_part = nullptr;
};

template <int N, int VEC, int G, int U>
struct CpnSlot {
    const CpnMode<N> &m;
    int64_t s, k, b0;
    int lane, g, col;
    bool on, first_mode;
    int row;
    bool carry;
    bool pend = false;  // acc is a chunk partial of segment `row`, not yet stored
    Vec<VEC> acc, ownv;
    double &lsum;

    __device__ __forceinline__ CpnSlot(const CpnMode<N> &m_, int64_t s_, int lane_, bool fm,
                                       double &ls)
        : m(m_), s(s_), k(m_.s.k), lane(lane_), g(lane_ % G), col((lane_ % G) * VEC),
          first_mode(fm), lsum(ls) {
        const SgrParams &a = m.s;
        on = col < a.k;
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

    // Entries [p, p + U): segment r, other coordinates c[0..N-2], value x,
    // input position pp (pass 0); padding past b0 repeats the last entry and
    // its residual is zeroed here.
    __device__ __forceinline__ void batch(int64_t p, const int (&r)[U], const int (&c)[N - 1][U],
                                          const float (&x)[U], const int (&pp)[U]) {
        bool same = true;
#pragma unroll
        for (int u = 0; u < U; ++u) same = same && r[u] == row;
        // All gathers of the batch are issued before any is used (a lane past
        // the rank reads column 0 and drops it), as in the order-3 kernel.
        const int cl = on ? col : 0;
        Vec<VEC> t[U], h[N - 2][U], ow[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            t[u].load(m.fac[0] + (int64_t)c[0][u] * k + cl);
#pragma unroll
            for (int f = 1; f < N - 1; ++f) h[f - 1][u].load(m.fac[f] + (int64_t)c[f][u] * k + cl);
        }
        if (!same) {
#pragma unroll
            for (int u = 0; u < U; ++u) ow[u].load(m.own + (int64_t)r[u] * k + cl);
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
#pragma unroll
            for (int f = 0; f < N - 2; ++f) {
#pragma unroll
                for (int e = 0; e < VEC; ++e) t[u].v[e] *= h[f][u].v[e];
            }
            if (!on) t[u].zero();
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
        if (!same && on) ownv = ow[U - 1];
    }

    __device__ __forceinline__ void finish() {
        const SgrParams &a = m.s;
        if (b0 == a.nnz || a.segidx[b0] != row) flush();
        else pend = true;  // a chunk of a long segment that goes on
    }
};

// The same pass with a fiber level (the second level of a compressed-fiber
// tree): entries of a slice come in runs of equal coordinate other[0] (a
// fiber), whose factor row fac[0] is gathered once per fiber.  With
// t' = the product of the other N - 2 gathered rows,
//   model = <own o fac0[fiber], t'>,  fiber sum += R t',
// and at the fiber's end the slice's sum gets fac0[fiber] o (fiber sum),
// which is sum R (fac0 o t') regrouped by fiber.  The open fiber keeps its
// factor row fv and the partial product pv = own o fv, so an entry in it
// needs N - 2 gathers and one dot product.
template <int N, int VEC, int G, int U>
struct CpnFiberSlot {
    const CpnMode<N> &m;
    int64_t s, k, b0;
    int lane, g, col;
    bool on, first_mode;
    int row;
    bool carry;
    bool pend = false;
    int fib = -1;          // coordinate of the open fiber (-1: none open)
    Vec<VEC> acc, ownv, fv, pv, accf;
    double &lsum;

    __device__ __forceinline__ CpnFiberSlot(const CpnMode<N> &m_, int64_t s_, int lane_, bool fm,
                                            double &ls)
        : m(m_), s(s_), k(m_.s.k), lane(lane_), g(lane_ % G), col((lane_ % G) * VEC),
          first_mode(fm), lsum(ls) {
        const SgrParams &a = m.s;
        on = col < a.k;
        const int64_t a0 = a.plan.item_ptr[s];
        b0 = a.plan.item_ptr[s + 1];
        row = a.segidx[a0];
        carry = a0 > 0 && a.segidx[a0 - 1] == row;
        acc.zero();
        accf.zero();
        fv.zero();
        pv.zero();
        if (on) ownv.load(m.own + (int64_t)row * k + col);
        else ownv.zero();
    }

    // the open fiber's sum into the slice's sum
    __device__ __forceinline__ void close_fiber() {
        if (fib >= 0) {
#pragma unroll
            for (int e = 0; e < VEC; ++e) acc.v[e] = __builtin_fmaf(fv.v[e], accf.v[e], acc.v[e]);
            accf.zero();
            fib = -1;
        }
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

    __device__ __forceinline__ void batch(int64_t p, const int (&r)[U], const int (&c)[N - 1][U],
                                          const float (&x)[U], const int (&pp)[U]) {
        bool same = true, samef = true;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            same = same && r[u] == row;
            samef = samef && c[0][u] == fib;
        }
        samef = samef && same;
        const int cl = on ? col : 0;
        Vec<VEC> t[U], h[N - 2][U], ow[U], fr[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if constexpr (N >= 3) t[u].load(m.fac[1] + (int64_t)c[1][u] * k + cl);
#pragma unroll
            for (int f = 2; f < N - 1; ++f) h[f - 2][u].load(m.fac[f] + (int64_t)c[f][u] * k + cl);
        }
        if (!samef) {
#pragma unroll
            for (int u = 0; u < U; ++u) fr[u].load(m.fac[0] + (int64_t)c[0][u] * k + cl);
        }
        if (!same) {
#pragma unroll
            for (int u = 0; u < U; ++u) ow[u].load(m.own + (int64_t)r[u] * k + cl);
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
#pragma unroll
            for (int f = 0; f < N - 3; ++f) {
#pragma unroll
                for (int e = 0; e < VEC; ++e) t[u].v[e] *= h[f][u].v[e];
            }
            if (!on) t[u].zero();
        }
        float d[U];
        if (samef) {
#pragma unroll
            for (int u = 0; u < U; ++u) d[u] = pv.dot(t[u]);
        } else {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const Vec<VEC> &o = same ? ownv : ow[u];
                Vec<VEC> q;
#pragma unroll
                for (int e = 0; e < VEC; ++e) q.v[e] = o.v[e] * fr[u].v[e];
                d[u] = q.dot(t[u]);
            }
        }
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
        if (samef) {
#pragma unroll
            for (int u = 0; u < U; ++u) accf.fma(res[u], t[u]);
        } else {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if (r[u] != row) {
                    close_fiber();
                    flush();
                    row = r[u];
                    carry = false;
                    acc.zero();
                }
                if (c[0][u] != fib) {
                    close_fiber();
                    fib = c[0][u];
                    fv = fr[u];
                }
                accf.fma(res[u], t[u]);
            }
            if (!same && on) ownv = ow[U - 1];
#pragma unroll
            for (int e = 0; e < VEC; ++e) pv.v[e] = ownv.v[e] * fv.v[e];
        }
    }

    __device__ __forceinline__ void finish() {
        const SgrParams &a = m.s;
        close_fiber();
        if (b0 == a.nnz || a.segidx[b0] != row) flush();
        else pend = true;
    }
};

// One slot's walk over item s of a mode pass; G >= 8 reads the metadata in
// tiles of G entries, narrower slots per entry and lane.
template <int N, int VEC, int G, int U, class Slot>
__device__ __forceinline__ int cpn_walk(const CpnMode<N> &m, int64_t s, int lane,
                                        bool first_mode, double &lsum, Vec<VEC> &part_acc) {
    const SgrParams &a = m.s;
    Slot st(m, s, lane, first_mode, lsum);
    const int64_t a0 = a.plan.item_ptr[s], b0 = st.b0;
    // Fields of entry q, past the item those of its last entry (every load
    // unconditional, so none is consumed before its batch); the batch zeroes
    // the padding's residual by position.
    auto fields = [&](int64_t q, int &r, int (&c)[N - 1], float &x, int &pp) {
        const int64_t qc = min(q, b0 - 1);
        r = a.segidx[qc];
#pragma unroll
        for (int f = 0; f < N - 1; ++f) c[f] = m.other[f][qc];
        x = a.w[qc];
        pp = first_mode ? m.perm[qc] : 0;
    };
    if constexpr (G >= 8) {
        static_assert(G % U == 0, "a tile holds whole batches");
        const int g = st.g;
        int tr, tc[N - 1], tp, nr = 0, nc[N - 1], np = 0;
        float tx, nx = 0.f;
#pragma unroll
        for (int f = 0; f < N - 1; ++f) nc[f] = 0;
        fields(a0 + g, tr, tc, tx, tp);
        for (int64_t t = a0; t < b0; t += G) {
            if (t + G < b0) fields(t + G + g, nr, nc, nx, np);
            for (int base = 0; base < G && t + base < b0; base += U) {
                int r[U], c[N - 1][U], pp[U];
                float x[U];
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    r[u] = slot_bcast<G>(tr, base + u);
#pragma unroll
                    for (int f = 0; f < N - 1; ++f) c[f][u] = slot_bcast<G>(tc[f], base + u);
                    x[u] = slot_bcast<G>(tx, base + u);
                    pp[u] = first_mode ? slot_bcast<G>(tp, base + u) : 0;
                }
                st.batch(t + base, r, c, x, pp);
            }
            tr = nr;
#pragma unroll
            for (int f = 0; f < N - 1; ++f) tc[f] = nc[f];
            tx = nx;
            tp = np;
        }
    } else {
        int r[U], c[N - 1][U], pp[U], nr[U], nc[N - 1][U], np[U];
        float x[U], nx[U];
        auto load = [&](int64_t p, int (&rr)[U], int (&cc)[N - 1][U], float (&xx)[U],
                        int (&qq)[U]) {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                int cu[N - 1];
                fields(p + u, rr[u], cu, xx[u], qq[u]);
#pragma unroll
                for (int f = 0; f < N - 1; ++f) cc[f][u] = cu[f];
            }
        };
        load(a0, r, c, x, pp);
        for (int64_t p = a0; p < b0; p += U) {
            if (p + U < b0) load(p + U, nr, nc, nx, np);
            st.batch(p, r, c, x, pp);
#pragma unroll
            for (int u = 0; u < U; ++u) {
                r[u] = nr[u];
#pragma unroll
                for (int f = 0; f < N - 1; ++f) c[f][u] = nc[f][u];
                x[u] = nx[u];
                pp[u] = np[u];
            }
        }
    }
    st.finish();
    part_acc = st.acc;
    return st.pend ? st.row : -1;  // a chunk partial, stored by store_chunk_partial
}

template <int N, int VEC, int G, int U>
__device__ __forceinline__ void cpn_block(const CpnMode<N> &m, int b, bool first_mode,
                                          double &lsum) {
    constexpr int kSlots = kBlock / G;
    const int lane = threadIdx.x % kWave;
    const int g = threadIdx.x % G;
    if (b < m.item_blocks) {
        const int64_t s = (int64_t)b * kSlots + threadIdx.x / G;
        Vec<VEC> pacc;
        pacc.zero();
        int pseg = -1;
        if (s < m.s.plan.nitems) {
            if (m.fiber)
                pseg = cpn_walk<N, VEC, G, U, CpnFiberSlot<N, VEC, G, U>>(m, s, lane, first_mode,
                                                                          lsum, pacc);
            else
                pseg = cpn_walk<N, VEC, G, U, CpnSlot<N, VEC, G, U>>(m, s, lane, first_mode, lsum,
                                                                     pacc);
        }
        store_chunk_partial<VEC, G>(pseg, pacc, m.s.part, m.s.plan.chunk_ord, s, m.s.k, g * VEC,
                                    g * VEC < m.s.k);
    } else {
        zero_segment<VEC>(m.s, (int64_t)(b - m.item_blocks) * kSlots + threadIdx.x / G, g * VEC,
                          g * VEC < m.s.k);
    }
}

// Block b belongs to the first mode whose block range holds it (modes in
// order; compile-time mode indices keep the kernel arguments addressed
// statically).
template <int M, int N, int VEC, int G, int U>
__device__ __forceinline__ void cpn_dispatch(const CpnParams<N> &f, int b, double &lsum) {
    const int nb = f.m[M].item_blocks + f.m[M].empty_blocks;
    if (b < nb) {
        cpn_block<N, VEC, G, U>(f.m[M], b, M == 0, lsum);
    } else if constexpr (M + 1 < N) {
        cpn_dispatch<M + 1, N, VEC, G, U>(f, b - nb, lsum);
    }
}

template <int N, int VEC, int G, int U>
__global__ __launch_bounds__(kBlock) void cpn_kernel(CpnParams<N> f) {
    double lsum = 0.0;
    cpn_dispatch<0, N, VEC, G, U>(f, blockIdx.x, lsum);
    const double t = block_sum(lsum);
    if (threadIdx.x == 0) f.loss_part[blockIdx.x] = t;
}

template <int G>
constexpr int cpn_unroll() {
#ifdef NSD_CPN_UNROLL
    return reduce_unroll<G, NSD_CPN_UNROLL>();
#else
    return reduce_unroll<G, (G >= 64 || G == 1) ? 4 : 2>();
#endif
}

template <int N, int VEC, int G>
static nsd_status launch_cpn(CpnParams<N> f, double *loss, hipStream_t st) {
    constexpr int kSlots = kBlock / G;
    int grid = 0;
    for (int i = 0; i < N; ++i) {
        f.m[i].item_blocks = (int32_t)ceil_div(f.m[i].s.plan.nitems, kSlots);
        f.m[i].empty_blocks = (int32_t)ceil_div(f.m[i].s.plan.nempty, kSlots);
        f.m[i].s.chunk_stride = chunk_group<G>();
        grid += f.m[i].item_blocks + f.m[i].empty_blocks;
    }
    if (grid == 0) return loss_finalize(f.loss_part, 0, loss, st);
    probe_begin(NSD_KERNEL_CPN, st);
    cpn_kernel<N, VEC, G, cpn_unroll<G>()><<<grid, kBlock, 0, st>>>(f);
    probe_end(NSD_KERNEL_CPN, st);
    NSD_TRY(check_launch("cpn_kernel"));
    LossJob job;
    job.p1 = f.loss_part;
    job.n1 = grid;
    job.loss = loss;
    FixJobs fx;
    for (int i = 0; i < N; ++i) add_fix(fx, f.m[i].s);
    fx.loss = job;
    return launch_fixes<VEC, G>(fx, st);
}

template <int N>
struct CpnLauncher {
    CpnParams<N> f;
    double *loss;
    hipStream_t st;
    template <int VEC, int G>
    nsd_status operator()() { return launch_cpn<N, VEC, G>(f, loss, st); }
};

static int64_t cpn_blocks(const nsd_coon *X, int rank, bool vec) {
    const WidthPlan wp = width_plan(rank, vec);
    const int slots = kBlock / wp.g;
    int64_t n = 0;
    for (int i = 0; i < X->order; ++i)
        n += ceil_div(X->mode[i].plan.nitems, slots) + ceil_div(X->mode[i].plan.nempty, slots);
    return n;
}

static size_t rnd256(size_t b) { return (b + 255) & ~size_t(255); }

// Loss partials of either form (ranks above 64, which a fused slot may not
// hold, form the residual once in its own pass).
static int64_t cpn_loss_parts(const nsd_coon *X, int rank) {
    int64_t blocks = std::max(cpn_blocks(X, rank, true), cpn_blocks(X, rank, false));
    if (rank > 64)
        blocks = std::max({blocks, resid_blocks(X->nnz, rank, true),
                           resid_blocks(X->nnz, rank, false)});
    return std::max<int64_t>(blocks, 1);
}

// Per-mode chunk partials, the loss partials and, for ranks above 64, the
// residual of every stored entry.
static size_t cpn_ws_bytes(const nsd_coon *X, int rank) {
    size_t b = 0;
    for (int n = 0; n < X->order; ++n) b += rnd256(sgr_part_bytes(X->mode[n].plan, rank));
    b += rnd256(cpn_loss_parts(X, rank) * sizeof(double));
    if (rank > 64) b += rnd256((size_t)std::max(X->nnz, 1) * sizeof(float));
    return b;
}

// The gradient of a rank wider than a fused slot: the residual once in mode
// 0's order (to dX and, unscaled, to a buffer in X's input order), then one
// mode pass per mode reading it through the mode's permutation.
static nsd_status cpn_wide(const nsd_coon *X, const float *const *F, int32_t rank, float seed,
                           double *loss, float *dX, float *const *dF, bool vec, char *b,
                           hipStream_t st) {
    const int N = X->order;
    float *part[NSD_MAX_ORDER];
    for (int n = 0; n < N; ++n) {
        part[n] = reinterpret_cast<float *>(b);
        b += rnd256(sgr_part_bytes(X->mode[n].plan, rank));
    }
    double *loss_part = reinterpret_cast<double *>(b);
    b += rnd256(cpn_loss_parts(X, rank) * sizeof(double));
    float *rbuf = reinterpret_cast<float *>(b);
    const nsd_coon_mode &m0 = X->mode[0];
    ResidParams r;
    r.nnz = X->nnz;
    r.k = rank;
    r.order = N;
    r.coord[0] = m0.segidx;
    for (int o = 0; o < N - 1; ++o) r.coord[o + 1] = m0.idx[o];  // mode o + 1
    for (int n = 0; n < N; ++n) r.fac[n] = F[n];
    r.x = m0.val;
    r.perm = m0.perm;
    r.rbuf = rbuf;
    r.resid = dX;
    r.seed = seed;
    r.lscale = 0.5;
    r.part = loss_part;
    NSD_TRY(resid_pass(r, vec, st));
    for (int n = 0; n < N; ++n) {
        const nsd_coon_mode &md = X->mode[n];
        MttkrpParams m;
        m.s.nseg = X->dims[n];
        m.s.nnz = X->nnz;
        m.s.k = rank;
        m.s.plan = md.plan;
        m.s.segptr = md.segptr;
        m.s.segidx = md.segidx;
        m.s.idx = md.idx[0];
        m.s.w = rbuf;
        m.s.wperm = md.perm;
        m.s.alpha = -seed;
        m.s.out = dF[n];
        m.s.part = part[n];
        for (int o = 0; o < N - 1; ++o) {
            m.other[o] = md.idx[o];
            m.fac[o] = F[(n + 1 + o) % N];
        }
        NSD_TRY(mttkrp_pass(m, N, vec, st));
    }
    return loss_finalize(loss_part, resid_blocks(X->nnz, rank, vec), loss, st);
}

static nsd_status check_coon(const nsd_coon *X) {
    NSD_REQUIRE(X != nullptr, "tensor descriptor is NULL");
    NSD_REQUIRE(X->order >= 3 && X->order <= NSD_MAX_ORDER, "order %d outside [3, %d]",
                X->order, NSD_MAX_ORDER);
    NSD_REQUIRE(X->nnz >= 0, "negative nnz");
    for (int n = 0; n < X->order; ++n) {
        NSD_REQUIRE(X->dims[n] >= 0, "negative dimension");
        const nsd_coon_mode &md = X->mode[n];
        NSD_REQUIRE(md.mode == n, "mode[%d] holds mode %d", n, md.mode);
        NSD_REQUIRE(md.segptr != nullptr, "mode %d segptr is NULL", n);
        if (X->nnz > 0) {
            NSD_REQUIRE(X->dims[n] > 0, "nnz > 0 in an empty shape");
            NSD_REQUIRE(md.segidx && md.val && md.perm, "mode %d array is NULL", n);
            for (int f = 0; f < X->order - 1; ++f)
                NSD_REQUIRE(md.idx[f] != nullptr, "mode %d coordinate %d is NULL", n, f);
            NSD_REQUIRE(md.plan.item_ptr && md.plan.nitems >= 1,
                        "mode %d plan is not built (nsd_plan_build)", n);
        }
    }
    return NSD_OK;
}

template <int N>
static nsd_status cpn_run(const nsd_coon *X, const float *const *F, int32_t rank, float seed,
                          double *loss, float *dX, float *const *dF, bool vec, char *b,
                          hipStream_t st) {
    CpnParams<N> f;
    for (int n = 0; n < N; ++n) {
        const nsd_coon_mode &md = X->mode[n];
        CpnMode<N> &m = f.m[n];
        m.s.nseg = X->dims[n];
        m.s.nnz = X->nnz;
        m.s.k = rank;
        m.s.plan = md.plan;
        m.s.segptr = md.segptr;
        m.s.segidx = md.segidx;
        m.s.idx = md.idx[0];
        m.s.w = md.val;
        m.s.alpha = -seed;
        m.s.out = dF[n];
        m.s.part = reinterpret_cast<float *>(b);
        b += rnd256(sgr_part_bytes(md.plan, rank));
        for (int o = 0; o < N - 1; ++o) {
            m.other[o] = md.idx[o];
            m.fac[o] = F[(n + 1 + o) % N];
        }
        m.fiber = md.fiber ? 1 : 0;
        if (m.fiber) {
            // the fiber mode (mode 1 for mode 0, else mode 0) first: the
            // product over the other rows does not depend on their order
            const int fm = n == 0 ? 1 : 0;
            const int of = (fm - n - 1 + N) % N;
            std::swap(m.other[0], m.other[of]);
            std::swap(m.fac[0], m.fac[of]);
        }
        m.own = F[n];
        m.perm = md.perm;
        m.resid = dX;
        m.seed = seed;
    }
    f.loss_part = reinterpret_cast<double *>(b);
    CpnLauncher<N> fn{f, loss, st};
    return dispatch_width(width_plan(rank, vec), fn);
}

}  // namespace nsd

using namespace nsd;

extern "C" {

nsd_status nsd_cpn_workspace_size(const nsd_coon *X, int32_t rank, size_t *bytes) {
    NSD_REQUIRE(bytes != nullptr, "bytes is NULL");
    NSD_REQUIRE(rank >= 1, "rank = %d < 1", rank);
    NSD_TRY(check_coon(X));
    *bytes = cpn_ws_bytes(X, rank);
    return NSD_OK;
}

nsd_status nsd_loss_cpn(const nsd_coon *X, const float *const *F, int32_t rank, float seed,
                        double *loss, float *dX, float *const *dF, void *ws, size_t ws_bytes,
                        void *stream) {
    NSD_TRY(check_coon(X));
    NSD_REQUIRE(rank >= 1, "rank = %d < 1", rank);
    NSD_REQUIRE(loss != nullptr && F != nullptr && dF != nullptr, "loss/F/dF is NULL");
    const int N = X->order;
    bool vec = rank % 4 == 0;
    for (int n = 0; n < N; ++n) {
        NSD_REQUIRE(X->dims[n] == 0 || dF[n] != nullptr, "dF%d is NULL", n + 1);
        NSD_REQUIRE(X->nnz == 0 || F[n] != nullptr, "F%d is NULL", n + 1);
        vec = vec && aligned16(F[n]) && aligned16(dF[n]);
    }
    NSD_REQUIRE(X->nnz == 0 || dX != nullptr, "dX is NULL");
    const size_t need = cpn_ws_bytes(X, rank);
    if (ws == nullptr || ws_bytes < need)
        return fail(NSD_ERR_WORKSPACE, "workspace %zu bytes at %p, need %zu", ws_bytes, ws, need);
    char *b = static_cast<char *>(ws);
    hipStream_t st = as_stream(stream);
    if (vec ? rank > 256 : rank > 64) return cpn_wide(X, F, rank, seed, loss, dX, dF, vec, b, st);
    switch (N) {
        case 3: return cpn_run<3>(X, F, rank, seed, loss, dX, dF, vec, b, st);
        case 4: return cpn_run<4>(X, F, rank, seed, loss, dX, dF, vec, b, st);
        case 5: return cpn_run<5>(X, F, rank, seed, loss, dX, dF, vec, b, st);
        default: return cpn_run<6>(X, F, rank, seed, loss, dX, dF, vec, b, st);
    }
}

}  // extern "C"
