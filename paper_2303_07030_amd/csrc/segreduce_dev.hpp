// Device building blocks shared by the gather-reduce, SDDMM, factorisation
// and CP kernels: the pipelined per-entry metadata, the walk of one work
// item, the long-segment combine, lane reductions and the lane-layout
// dispatch.  Included by several translation units; everything here is a
// template or inline.
#pragma once

#include <algorithm>

#include "nsd_internal.hpp"
#include "segreduce.hpp"

namespace nsd {

constexpr int kBlock = 256;
constexpr int kBlockWaves = kBlock / kWave;
constexpr int kHugeChunks = 64;  // matches the plan builder

// --------------------------------------------------------- entry metadata

// The value held by lane `src` of this lane's slot of G lanes (src uniform
// over the slot): a lane read into a scalar register for full-wave slots, a
// cross-lane shuffle otherwise.  Every lane of the slot must be active.
template <int G>
__device__ __forceinline__ int slot_bcast(int v, int src) {
    if constexpr (G == 64) return __builtin_amdgcn_readlane(v, src);
    else return __shfl(v, src, G);
}

template <int G>
__device__ __forceinline__ float slot_bcast(float v, int src) {
    return __int_as_float(slot_bcast<G>(__float_as_int(v), src));
}

// Feeds the entries [a0, b0) of one work item, in order, to
//   st.batch(p, r, c, pos, w, ps, ws)
// in batches of U entries p .. p + U - 1: segment r, gathered row c, weight
// position pos (wperm[q], or q) and weight w (1 without weights).  Entries
// past b0 are padding: the item's last segment and gathered row (valid
// addresses), position 0, weight 0.  ps / ws are the position and weight of
// entry g / (G / U) of the batch when G >= U (else those of the first).
//
// Slots of 8 or more lanes read the item in tiles of G entries: lane g
// loads the metadata of entry g of a tile, one coalesced load per field,
// and each batch takes its entries' fields from their lanes by broadcast.
// Narrow slots load every entry's metadata in every lane.  Either way the
// weight positions run one stage ahead of the weights they index, and the
// rest of the metadata one stage ahead of the batch that uses it.
template <int G, int U, class Slot>
__device__ __forceinline__ void walk_item(const SgrParams &a, int64_t a0, int64_t b0, int g,
                                          Slot &st) {
    const int last_r = a.segidx[b0 - 1], last_c = a.idx[b0 - 1];
    if constexpr (G >= 8) {
        static_assert(G % U == 0, "a tile holds whole batches");
        auto position = [&](int64_t t) -> int {
            const int64_t q = t + g;
            return q < b0 ? (a.wperm ? a.wperm[q] : (int)q) : 0;
        };
        auto rest = [&](int64_t t, int pos, int &r, int &c, float &w) {
            const int64_t q = t + g;
            r = q < b0 ? a.segidx[q] : last_r;
            c = q < b0 ? a.idx[q] : last_c;
            w = q < b0 ? (a.w ? a.w[pos] : 1.f) : 0.f;
        };
        int tr, tc, tpos, nr = 0, nc = 0, npos = 0, ppos = 0;
        float tw, nw = 0.f;
        tpos = position(a0);
        rest(a0, tpos, tr, tc, tw);
        if (a0 + G < b0) ppos = position(a0 + G);
        for (int64_t t = a0; t < b0; t += G) {
            if (t + G < b0) {
                npos = ppos;
                rest(t + G, npos, nr, nc, nw);
                if (t + 2 * G < b0) ppos = position(t + 2 * G);
            }
            for (int base = 0; base < G && t + base < b0; base += U) {
                int r[U], c[U], pos[U];
                float w[U];
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    r[u] = slot_bcast<G>(tr, base + u);
                    c[u] = slot_bcast<G>(tc, base + u);
                    pos[u] = slot_bcast<G>(tpos, base + u);
                    w[u] = slot_bcast<G>(tw, base + u);
                }
                const int src = base + g / (G / U);
                st.batch(t + base, r, c, pos, w, __shfl(tpos, src, G), __shfl(tw, src, G));
            }
            tr = nr;
            tc = nc;
            tpos = npos;
            tw = nw;
        }
    } else {
        auto positions = [&](int64_t p, int (&pos)[U]) {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int64_t q = p + u;
                pos[u] = q < b0 ? (a.wperm ? a.wperm[q] : (int)q) : 0;
            }
        };
        auto rest = [&](int64_t p, const int (&pos)[U], int (&r)[U], int (&c)[U], float (&w)[U]) {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int64_t q = p + u;
                r[u] = q < b0 ? a.segidx[q] : last_r;
                c[u] = q < b0 ? a.idx[q] : last_c;
                w[u] = q < b0 ? (a.w ? a.w[pos[u]] : 1.f) : 0.f;
            }
        };
        int r[U], c[U], pos[U], nr[U], nc[U], npos[U], ppos[U];
        float w[U], nw[U];
        positions(a0, pos);
        rest(a0, pos, r, c, w);
        positions(a0 + U, ppos);
        for (int64_t p = a0; p < b0; p += U) {
            if (p + U < b0) {
#pragma unroll
                for (int u = 0; u < U; ++u) npos[u] = ppos[u];
                rest(p + U, npos, nr, nc, nw);
                if (p + 2 * U < b0) positions(p + 2 * U, ppos);
            }
            int ps = pos[0];
            float ws = w[0];
            if constexpr (G > 1 && G >= U) {
                const int us = g / (G / U);
#pragma unroll
                for (int u = 1; u < U; ++u) {
                    if (us == u) {
                        ps = pos[u];
                        ws = w[u];
                    }
                }
            }
            st.batch(p, r, c, pos, w, ps, ws);
#pragma unroll
            for (int u = 0; u < U; ++u) {
                r[u] = nr[u];
                c[u] = nc[u];
                pos[u] = npos[u];
                w[u] = nw[u];
            }
        }
    }
}

// Chunk partials of a wave, added together before they are stored.  The
// chunk items of a long segment are consecutive and hold no other segment,
// so slots holding chunks of one segment are consecutive too.  Slots are
// taken in groups of chunk_group<G>() (consecutive slots of one wave); in a
// group, the first slot of every run of one segment adds the run's partials
// in slot order (lane shuffles, no barrier) and stores the sum as its own
// item's partial row.  A segment then has one partial row per group it
// spans: its first chunk's and those of the chunks at item indexes
// divisible by the group size, which the combine reads with chunk_stride =
// chunk_group<G>().  Partial rows are compact: item s writes row
// chunk_ord[s] (its position among the chunk items).  Every lane of the wave
// calls this (seg < 0: the slot holds no partial).
template <int G>
constexpr int chunk_group() {
    return kWave / G < 8 ? kWave / G : 8;
}

template <int VEC, int G>
__device__ __forceinline__ void store_chunk_partial(int seg, Vec<VEC> acc, float *part,
                                                    const int32_t *chunk_ord, int64_t s,
                                                    int64_t k, int col, bool on) {
    constexpr int CG = chunk_group<G>();
    if constexpr (CG == 1) {
        if (seg >= 0 && on) acc.store(part + (int64_t)chunk_ord[s] * k + col);
    } else {
        if (!__any(seg >= 0)) return;  // wave-uniform: no partial in this wave
        const int lane = threadIdx.x % kWave;
        const int q = (lane / G) % CG;  // slot within its group
        const int prev = __shfl(seg, q > 0 ? lane - G : lane);
        const bool leader = seg >= 0 && (q == 0 || prev != seg);
        const Vec<VEC> own = acc;  // every lane reads the others' own partials
        bool run = true;
#pragma unroll
        for (int d = 1; d < CG; ++d) {
            const int src = q + d < CG ? lane + d * G : lane;
            const int sseg = __shfl(seg, src);
            Vec<VEC> x;
#pragma unroll
            for (int e = 0; e < VEC; ++e) x.v[e] = __shfl(own.v[e], src);
            run = run && q + d < CG && sseg == seg;
            if (run) acc.add(x);
        }
        if (leader && on) acc.store(part + (int64_t)chunk_ord[s] * k + col);
    }
}

// One slot's gather-reduce over item s (entries [a0, b0)).  Complete
// segments are written as alpha * sum; a segment cut by the item's end or
// start goes to part[s].  `seg_done(segment, unscaled sum)` is called for
// every segment completed inside the item.
template <int VEC, int G, int U, class SegDone>
struct SgrSlot {
    const SgrParams &a;
    int64_t s, k;
    int col;
    bool on;
    int row;
    bool carry;  // the open segment started before this item (a later chunk)
    bool pend = false;  // acc is a chunk partial of segment `row`, not yet stored
    Vec<VEC> acc;
    SegDone &seg_done;

    __device__ __forceinline__ SgrSlot(const SgrParams &a_, int64_t s_, int col_, bool on_,
                                       int64_t a0, SegDone &sd)
        : a(a_), s(s_), k(a_.k), col(col_), on(on_), seg_done(sd) {
        row = a.segidx[a0];
        carry = a0 > 0 && a.segidx[a0 - 1] == row;
        acc.zero();
    }

    __device__ __forceinline__ void flush() {
        if (carry) {
            pend = true;  // a chunk item holds one segment: this is its end
        } else {
            seg_done(row, acc);
            if (on) {
                Vec<VEC> t = acc;
                t.scale(a.alpha);
                t.store(a.out + (int64_t)row * k + col);
            }
        }
    }

    __device__ __forceinline__ void batch(int64_t, const int (&r)[U], const int (&c)[U],
                                          const int (&)[U], const float (&w)[U], int, float) {
        Vec<VEC> xv[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (a.X && on) xv[u].load(a.X + (int64_t)c[u] * k + col);
            else xv[u].ones();
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (r[u] != row) {
                flush();
                row = r[u];
                carry = false;
                acc.zero();
            }
            acc.fma(w[u], xv[u]);
        }
    }

    __device__ __forceinline__ void finish(int64_t b0) {
        if (b0 == a.nnz || a.segidx[b0] != row) flush();
        else pend = true;  // a chunk of a long segment that goes on
    }
};

// Walks item s; returns the segment of the chunk partial left in `part_acc`
// (to be stored with store_chunk_partial), or -1.
template <int VEC, int G, int U, class SegDone>
__device__ __forceinline__ int sgr_walk(const SgrParams &a, int64_t s, int col, bool on,
                                        SegDone seg_done, Vec<VEC> &part_acc) {
    const int64_t a0 = a.plan.item_ptr[s];
    const int64_t b0 = a.plan.item_ptr[s + 1];
    SgrSlot<VEC, G, U, SegDone> st(a, s, col, on, a0, seg_done);
    walk_item<G, U>(a, a0, b0, (int)(threadIdx.x % G), st);
    st.finish(b0);
    part_acc = st.acc;
    return st.pend ? st.row : -1;
}

template <int VEC>
__device__ __forceinline__ void zero_segment(const SgrParams &a, int64_t e, int col, bool on) {
    if (e < a.plan.nempty && on) {
        Vec<VEC> z;
        z.zero();
        z.store(a.out + (int64_t)a.plan.empty_seg[e] * a.k + col);
    }
}

struct NoSegDone {
    template <int VEC>
    __device__ void operator()(int, const Vec<VEC> &) const {}
};

// ------------------------------------------------------------- loss total

// Strided partial sums of one thread over p[0, n): C independent loads
// issued before any is added, then the C chains added in a fixed pairwise
// order.  One block summing ~10^5 block partials with few chains is a chain
// of memory latencies; 16 chains take 32 more VGPRs, so kernels whose main
// work needs the registers use 4.
template <int C>
__device__ __forceinline__ double strided_sum(const double *p, int64_t n) {
    double s[C];
#pragma unroll
    for (int j = 0; j < C; ++j) s[j] = 0.0;
    int64_t i = threadIdx.x;
    for (; i + (C - 1) * kBlock < n; i += C * kBlock) {
        double x[C];
#pragma unroll
        for (int j = 0; j < C; ++j) x[j] = p[i + j * kBlock];
#pragma unroll
        for (int j = 0; j < C; ++j) s[j] += x[j];
    }
#pragma unroll
    for (int j = 0; j < C - 1; ++j)  // the ones left (static indexes)
        if (i + j * kBlock < n) s[j] += p[i + j * kBlock];
#pragma unroll
    for (int w = C / 2; w >= 1; w >>= 1)
#pragma unroll
        for (int j = 0; j < w; ++j) s[j] += s[j + w];
    return s[0];
}

// One whole block: the loss total of a job, in a fixed order (C: loads in
// flight per thread, see strided_sum).
template <int C>
__device__ __forceinline__ void loss_total_block(const LossJob &job) {
    __shared__ double sh[kBlock];
    sh[threadIdx.x] = strided_sum<C>(job.p1, job.n1) + strided_sum<C>(job.p2, job.n2);
    __syncthreads();
    for (int w = kBlock / 2; w >= 1; w >>= 1) {
        if ((int)threadIdx.x < w) sh[threadIdx.x] += sh[threadIdx.x + w];
        __syncthreads();
    }
    if (threadIdx.x == 0) *job.loss = sh[0];
}

// ----------------------------------------------------------- long segments

// out[seg] = alpha * sum of the segment's partial rows (see chunk_stride), in
// chunk order per row group, the groups then combined by a fixed butterfly.
// Of a pass's blocks, those below wave_blocks give one wave to each long
// segment of at most kHugeChunks partial rows; the blocks after them (when
// launched) give a whole block to each huge segment with more.  When
// seg_loss is given, beta * ||out[seg]||^2 is stored for every long segment.
// b is the block's index within the pass.
#ifdef NSD_FIX_DEPTH
constexpr int kFixDepth = NSD_FIX_DEPTH;
#else
constexpr int kFixDepth = 4;  // chunk partials in flight per lane (a power of two; measured)
#endif

template <int VEC, int G>
__device__ __forceinline__ void fix_block(const SgrParams &a, int b, int wave_blocks,
                                          double *seg_loss, double beta) {
    constexpr int RG = kWave / G;  // row groups per wave
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int q = lane / G, g = lane % G;
    const int64_t k = a.k;
    const int L = a.plan.item_len;
    __shared__ float red[kBlockWaves][G * VEC];
    const bool huge = b >= wave_blocks;
    int64_t i;
    int nsum, qq;  // number of groups sharing the chunks, this lane's group
    if (!huge) {
        i = (int64_t)b * kBlockWaves + wave;
        if (i >= a.plan.nlong) return;
        nsum = RG;
        qq = q;
    } else {
        i = a.plan.huge_idx[b - wave_blocks];
        nsum = RG * kBlockWaves;
        qq = wave * RG + q;
    }
    const int seg = a.plan.long_seg[i];
    const int64_t s0 = a.plan.long_first[i];
    const int64_t chunks = ((int64_t)a.segptr[seg + 1] - a.segptr[seg] + L - 1) / L;
    // the segment's partial rows: items s0, then s0 + fb + j * stride, whose
    // rows in the compact array follow the first chunk's (chunks are
    // consecutive items and consecutive in chunk_item)
    const int64_t stride = a.chunk_stride;
    const int64_t fb = stride - s0 % stride;
    const int64_t n = fb < chunks ? 1 + (chunks - fb + stride - 1) / stride : 1;
    const int64_t r0 = a.plan.chunk_ord[s0];
    auto prow = [&](int64_t t) { return r0 + (t == 0 ? 0 : fb + (t - 1) * stride); };
    // one wave per segment of at most kHugeChunks partial rows, else a block
    if (huge != (n > kHugeChunks)) return;
    double lsq = 0.0;
    for (int c0 = 0; c0 < a.k; c0 += G * VEC) {
        const int col = c0 + g * VEC;
        const bool on = col < a.k;
        // kFixDepth chunk partials in flight per lane, as many running sums
        Vec<VEC> acc[kFixDepth];
#pragma unroll
        for (int j = 0; j < kFixDepth; ++j) acc[j].zero();
        if (on) {
            int64_t t = qq;
            for (; t + (kFixDepth - 1) * nsum < n; t += kFixDepth * nsum) {
                Vec<VEC> x[kFixDepth];
#pragma unroll
                for (int j = 0; j < kFixDepth; ++j)
                    x[j].load(a.part + prow(t + j * nsum) * k + col);
#pragma unroll
                for (int j = 0; j < kFixDepth; ++j) acc[j].add(x[j]);
            }
#pragma unroll
            for (int j = 0; j < kFixDepth - 1; ++j) {  // the ones left
                if (t + j * nsum < n) {
                    Vec<VEC> x;
                    x.load(a.part + prow(t + j * nsum) * k + col);
                    acc[j].add(x);
                }
            }
        }
#pragma unroll
        for (int w = kFixDepth / 2; w >= 1; w >>= 1)
#pragma unroll
            for (int j = 0; j < w; ++j) acc[j].add(acc[j + w]);
#pragma unroll
        for (int m = G; m < kWave; m <<= 1)
#pragma unroll
            for (int e = 0; e < VEC; ++e) acc[0].v[e] += shfl_xor(acc[0].v[e], m);
        if (huge) {
            if (q == 0)
#pragma unroll
                for (int e = 0; e < VEC; ++e) red[wave][g * VEC + e] = acc[0].v[e];
            __syncthreads();
            if (wave == 0) {
#pragma unroll
                for (int e = 0; e < VEC; ++e)
                    acc[0].v[e] = (red[0][g * VEC + e] + red[1][g * VEC + e]) +
                                  (red[2][g * VEC + e] + red[3][g * VEC + e]);
            }
            __syncthreads();
        }
        if ((!huge || wave == 0) && q == 0 && on) {
            acc[0].scale(a.alpha);
            acc[0].store(a.out + (int64_t)seg * k + col);
#pragma unroll
            for (int e = 0; e < VEC; ++e) lsq += (double)acc[0].v[e] * acc[0].v[e];
        }
    }
    if (seg_loss) {
        // only the lanes of group 0 (of wave 0 for a huge segment) hold squares
#pragma unroll
        for (int m = 1; m < kWave; m <<= 1) lsq += __shfl_xor(lsq, m, kWave);
        if (lane == 0 && (!huge || wave == 0)) seg_loss[i] = beta * lsq;
    }
}

// Long segments of up to kMaxFixJobs passes, combined in one launch (each
// pass on its own block range), and the call's loss total.
constexpr int kMaxFixJobs = NSD_MAX_ORDER;

struct FixJob {
    SgrParams a;
    double *seg_loss = nullptr;
    double beta = 0.0;
    int wave_blocks = 0, blocks = 0;
};

struct FixJobs {
    FixJob job[kMaxFixJobs];
    int n = 0;
    LossJob loss;  // with a loss job, the grid's last block computes the
                   // call's loss total (its partials come from earlier launches)
};

static_assert(sizeof(FixJobs) <= 4096, "combine jobs fit the kernel argument limit");

// Loads in flight per thread for the loss total riding on the combine
// launch (its partials are one per block of a main pass: ~10^5 for a CP
// pass over 20M entries).
#ifdef NSD_FIX_SUM_CHAINS
constexpr int kFixSumChains = NSD_FIX_SUM_CHAINS;
#else
constexpr int kFixSumChains = 16;
#endif

template <int VEC, int G>
__global__ __launch_bounds__(kBlock) void sgr_fix_kernel(FixJobs f) {
    if (f.loss.loss && blockIdx.x == gridDim.x - 1) {
        loss_total_block<kFixSumChains>(f.loss);
        return;
    }
    int b = blockIdx.x;
    for (int t = 0; t < f.n; ++t) {
        const FixJob &j = f.job[t];
        if (b < j.blocks) {
            fix_block<VEC, G>(j.a, b, j.wave_blocks, j.seg_loss, j.beta);
            return;
        }
        b -= j.blocks;
    }
}

// Entries per batch (rows in flight per lane).  The defaults can be changed
// at build time (-DNSD_SGR_UNROLL=..., and likewise for the other kernel
// families) for tuning.  Where a batch's dot products are reduced with
// transpose_reduce the batch may not exceed the slot width G (G = 1 aside).
template <int G, int U>
constexpr int reduce_unroll() {
    return G == 1 ? U : (U < G ? U : G);
}

template <int G>
constexpr int sgr_unroll() {
#ifdef NSD_SGR_UNROLL
    return NSD_SGR_UNROLL;
#else
    // measured on MI355X: eight rows in flight per lane for 16-lane slots
    // (the SpMM row pass of k = 64, whose short items are latency-bound),
    // two for 32-lane slots, four for full-wave slots, eight for the narrow
    // slots of small widths
    return G >= 64 ? 4 : (G >= 32 ? 2 : 8);
#endif
}

template <int G>
constexpr int sddmm_unroll() {
#ifdef NSD_SDDMM_UNROLL
    return reduce_unroll<G, NSD_SDDMM_UNROLL>();
#else
    return reduce_unroll<G, 4>();
#endif
}

// Adds a pass's long segments to a combined launch.
inline void add_fix(FixJobs &f, const SgrParams &a, double *seg_loss = nullptr,
                    double beta = 0.0) {
    FixJob &j = f.job[f.n++];
    j.a = a;
    j.seg_loss = seg_loss;
    j.beta = beta;
    j.wave_blocks = (int)ceil_div(a.plan.nlong, kBlockWaves);
    // a segment of c chunks has at most 1 + ceil((c - 1) / chunk_stride)
    // partial rows; when the longest has no more than kHugeChunks, waves
    // take every segment and no block per huge segment is launched (such
    // blocks would each load their segment's bounds only to return)
    const int64_t c = a.plan.longest_chunks;
    const int64_t rows = c <= 1 ? c : 1 + (c - 1 + a.chunk_stride - 1) / a.chunk_stride;
    const bool blocks_needed = a.plan.nhuge > 0 && (c == 0 || rows > kHugeChunks);
    j.blocks = a.plan.nlong > 0 ? j.wave_blocks + (blocks_needed ? a.plan.nhuge : 0) : 0;
}

// Combines the long segments of every pass in f (those that have any) and
// runs the loss job (when given), all in one launch.
template <int VEC, int G>
inline nsd_status launch_fixes(const FixJobs &f, hipStream_t st) {
    int grid = 0;
    for (int t = 0; t < f.n; ++t) grid += f.job[t].blocks;
    if (grid == 0 && !f.loss.loss) return NSD_OK;
    probe_begin(NSD_KERNEL_SGR_FIX, st);
    sgr_fix_kernel<VEC, G><<<grid + (f.loss.loss ? 1 : 0), kBlock, 0, st>>>(f);
    probe_end(NSD_KERNEL_SGR_FIX, st);
    return check_launch("sgr_fix_kernel");
}

// One pass's long segments and the loss job, in one launch.
template <int VEC, int G>
inline nsd_status launch_fix(const SgrParams &a, double *seg_loss, double beta, hipStream_t st,
                             LossJob job = LossJob{}) {
    FixJobs f;
    add_fix(f, a, seg_loss, beta);
    f.loss = job;
    return launch_fixes<VEC, G>(f, st);
}

// Calls f.template operator()<VEC, G>() for the lane layout wp.
template <class F>
inline nsd_status dispatch_width(const WidthPlan &wp, F &f) {
    if (wp.vec == 4) {
        switch (wp.g) {
            case 1: return f.template operator()<4, 1>();
            case 2: return f.template operator()<4, 2>();
            case 4: return f.template operator()<4, 4>();
            case 8: return f.template operator()<4, 8>();
            case 16: return f.template operator()<4, 16>();
            case 32: return f.template operator()<4, 32>();
            default: return f.template operator()<4, 64>();
        }
    }
    switch (wp.g) {
        case 1: return f.template operator()<1, 1>();
        case 2: return f.template operator()<1, 2>();
        case 4: return f.template operator()<1, 4>();
        case 8: return f.template operator()<1, 8>();
        case 16: return f.template operator()<1, 16>();
        case 32: return f.template operator()<1, 32>();
        default: return f.template operator()<1, 64>();
    }
}

// Reduces U partial dot products across the G lanes of a slot with a
// transposing butterfly: at each step a lane keeps half of its values and
// receives the partner's matching half, so U values cost U - 1 exchanges
// plus log2(G / U) for the last one.  Lane g ends with the total of value
// number g / (G / U).
// Step of span M with C values still held per lane (the partner is the
// other half of the aligned 2M-lane group, lane_xor<M>).
template <int M, int C, int U>
__device__ __forceinline__ void transpose_step(float (&v)[U], int lane) {
    if constexpr (M >= 1) {
        if constexpr (C > 1) {
            const bool upper = (lane & M) != 0;
#pragma unroll
            for (int i = 0; i < C / 2; ++i) {
                const float send = upper ? v[i] : v[i + C / 2];
                const float keep = upper ? v[i + C / 2] : v[i];
                v[i] = keep + lane_xor<M>(send);
            }
            transpose_step<M / 2, C / 2, U>(v, lane);
        } else {
            v[0] += lane_xor<M>(v[0]);
            transpose_step<M / 2, 1, U>(v, lane);
        }
    }
}

template <int G, int U>
__device__ __forceinline__ float transpose_reduce(float (&v)[U], int lane) {
    transpose_step<G / 2, U, U>(v, lane);
    return v[0];
}

// After transpose_reduce (lane g holding the total of value g / (G / U)),
// every lane's copy of all U totals: with two values one lane move from the
// other half of the slot, otherwise U broadcasts.
template <int G, int U>
__device__ __forceinline__ void slot_totals(float tot, int lane, float (&out)[U]) {
    if constexpr (U == 2) {
        const float other = lane_xor<G / 2>(tot);
        const bool upper = (lane & (G / 2)) != 0;
        out[0] = upper ? other : tot;
        out[1] = upper ? tot : other;
    } else {
        constexpr int kRep = G / U;
#pragma unroll
        for (int u = 0; u < U; ++u) out[u] = __shfl(tot, u * kRep, G);
    }
}

// Block total of per-lane fp64 values, in a fixed order.
__device__ __forceinline__ double block_sum(double v) {
    __shared__ double wsum[kBlockWaves];
#pragma unroll
    for (int m = kWave / 2; m >= 1; m >>= 1) v += __shfl_xor(v, m, kWave);
    if (threadIdx.x % kWave == 0) wsum[threadIdx.x / kWave] = v;
    __syncthreads();
    const double t = (wsum[0] + wsum[1]) + (wsum[2] + wsum[3]);
    __syncthreads();
    return t;
}

}  // namespace nsd
