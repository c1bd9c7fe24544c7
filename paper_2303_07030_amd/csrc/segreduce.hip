// Segmented gather-reduce, sampled dense-dense products and the row pass of
// the SpMM gradient.
//
// Gather-reduce computes, for every segment s of a sorted sparse operand
// (a row of a CSR, or a column of its CSC),
//     out[s, :] = alpha * sum_{p in s} w_p * X[idx_p, :]
// which is SpMV / SpMM (segments = rows, idx = colind, w = val) and the
// transposed product A^T G (segments = columns, idx = rowind, w = val[perm]).
// It is the `sum(<j, a> in row) a * X(j)` of the matrix product in Logical
// SDQLite (Section 3) with the singleton "+=" of the paper's code generation
// (Section 5.5), arranged so that every output is written once, without
// atomics.
//
// Load balance comes from the operand's work plan (nsd_plan): every work item
// is either a run of whole short segments or one chunk of a long segment.  A
// slot of G lanes (VEC floats of a dense row each; VEC * G up to 256 columns
// per pass) walks its item in batches of U entries.  The entry metadata
// (segment, gathered row, weight) of the next batch is loaded while the
// current batch's dense rows are in flight, so one memory round trip is paid
// per batch.  A segment that ends inside the item is written directly; a
// chunk of a long segment leaves one partial sum, and a second kernel adds a
// long segment's chunk partials in chunk order, one wave per segment (one
// workgroup for huge segments).  Empty segments are zero-filled by extra
// blocks of the first launch.  Results are bitwise reproducible.
#include <algorithm>

#include "nsd_internal.hpp"
#include "segreduce.hpp"
#include "segreduce_dev.hpp"

namespace nsd {


template <int VEC, int G, int U>
__global__ __launch_bounds__(kBlock) void sgr_main_kernel(SgrParams a) {
    constexpr int kSlots = kBlock / G;
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
    if (s < a.plan.nitems) pseg = sgr_walk<VEC, G, U>(a, s, col, on, NoSegDone{}, pacc);
    store_chunk_partial<VEC, G>(pseg, pacc, a.part, a.plan.chunk_ord, s, a.k, col, on);
}

// Zero-fill of a whole output when there is nothing to reduce.
__global__ void fill_zero_kernel(float *out, int64_t n) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) out[i] = 0.f;
}

// One partial row per chunk item (compact, see store_chunk_partial).
size_t sgr_part_bytes(const nsd_plan &plan, int k) {
    return (size_t)std::max<int64_t>(plan.nchunks, 1) * (size_t)k * sizeof(float);
}

template <int VEC, int G>
static nsd_status launch_sgr_vg(SgrParams a, hipStream_t st) {
    constexpr int kSlots = kBlock / G;
    a.item_blocks = (int32_t)ceil_div(a.plan.nitems, kSlots);
    a.chunk_stride = chunk_group<G>();
    const int64_t empty_blocks = ceil_div(a.plan.nempty, kSlots);
    dim3 grid((unsigned)(a.item_blocks + empty_blocks), (unsigned)ceil_div(a.k, G * VEC));
    probe_begin(NSD_KERNEL_SGR_MAIN, st);
    sgr_main_kernel<VEC, G, sgr_unroll<G>()><<<grid, kBlock, 0, st>>>(a);
    probe_end(NSD_KERNEL_SGR_MAIN, st);
    NSD_TRY(check_launch("sgr_main_kernel"));
    return launch_fix<VEC, G>(a, nullptr, 0.0, st);
}

struct SgrLauncher {
    SgrParams a;
    hipStream_t st;
    template <int VEC, int G>
    nsd_status operator()() { return launch_sgr_vg<VEC, G>(a, st); }
};

nsd_status segreduce(SgrParams a, hipStream_t st) {
    const int64_t total = (int64_t)a.nseg * a.k;
    if (a.nnz == 0) {
        if (total > 0) fill_zero_kernel<<<ceil_div(total, 256), 256, 0, st>>>(a.out, total);
        return check_launch("fill_zero_kernel");
    }
    // float4 lanes need 16-byte aligned dense rows; otherwise use scalar lanes
    const WidthPlan wp = width_plan(a.k, aligned16(a.out) && (!a.X || aligned16(a.X)));
    SgrLauncher f{a, st};
    return dispatch_width(wp, f);
}

// ------------------------------------------------------------------ SDDMM

// SDDMM of entries [a0, b0) by one slot:
//   out[p] = alpha * <X[rowidx[p]], Y[colind[p]]>, lsum += w[p] * <...>.
template <int VEC, int G, int U>
__device__ __forceinline__ void sddmm_range(const SddmmParams &a, int64_t a0, int64_t b0,
                                            int lane, double &lsum) {
    const int g = lane % G;
    const int64_t k = a.k;
    const int last_r = a.rowidx[b0 - 1], last_c = a.colind[b0 - 1];
    int rr[U], cc[U], nr[U], nc[U];
    auto load = [&](int64_t p, int (&r)[U], int (&c)[U]) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const bool valid = p + u < b0;
            r[u] = valid ? a.rowidx[p + u] : last_r;
            c[u] = valid ? a.colind[p + u] : last_c;
        }
    };
    load(a0, rr, cc);
    for (int64_t p = a0; p < b0; p += U) {
        if (p + U < b0) load(p + U, nr, nc);
        float part[U];
#pragma unroll
        for (int u = 0; u < U; ++u) part[u] = 0.f;
        for (int c0 = 0; c0 < a.k; c0 += G * VEC) {
            const int col = c0 + g * VEC;
            if (col < a.k) {
                Vec<VEC> xv[U], yv[U];
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    if (a.X) xv[u].load(a.X + (int64_t)rr[u] * k + col);
                    else xv[u].ones();
                    yv[u].load(a.Y + (int64_t)cc[u] * k + col);
                }
#pragma unroll
                for (int u = 0; u < U; ++u) part[u] += xv[u].dot(yv[u]);
            }
        }
        if constexpr (G == 1) {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if (p + u < b0) {
                    a.out[a.operm ? a.operm[p + u] : p + u] = a.alpha * part[u];
                    if (a.w) lsum += (double)a.w[p + u] * (double)part[u];
                }
            }
        } else {
            const float tot = transpose_reduce<G, U>(part, lane);
            constexpr int kRep = G / U;
            const int64_t q = p + g / kRep;
            if (g % kRep == 0 && q < b0) {
                a.out[a.operm ? a.operm[q] : q] = a.alpha * tot;
                if (a.w) lsum += (double)a.w[q] * (double)tot;
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            rr[u] = nr[u];
            cc[u] = nc[u];
        }
    }
}

// Slots over equal entry ranges (nnz-split): no segment structure needed.
template <int VEC, int G, int U>
__global__ __launch_bounds__(kBlock) void sddmm_kernel(SddmmParams a) {
    constexpr int kSlots = kBlock / G;
    const int lane = threadIdx.x % kWave;
    const int64_t s = (int64_t)blockIdx.x * kSlots + threadIdx.x / G;
    double lsum = 0.0;
    if (s < a.nslots) {
        const int64_t a0 = s * a.L;
        sddmm_range<VEC, G, U>(a, a0, min(a0 + (int64_t)a.L, (int64_t)a.nnz), lane, lsum);
    }
    if (a.part) {
        const double t = block_sum(lsum);
        if (threadIdx.x == 0) a.part[blockIdx.x] = a.beta * t;
    }
}

int choose_slot_len(int64_t nnz, int slots_per_wave) {
    // aim for ~8192 waves (8 per SIMD on 256 CUs); 16 <= L <= 256
    const int64_t target = 8192LL * slots_per_wave;
    int L = 16;
    while (L < 256 && (int64_t)L * 2 * target <= nnz) L <<= 1;
    return L;
}

SddmmShape sddmm_shape(int64_t nnz, int k, bool vec_ok) {
    SddmmShape sh;
    sh.wp = width_plan(k, vec_ok);
    const int slots_per_block = kBlock / sh.wp.g;
    sh.L = choose_slot_len(nnz, kWave / sh.wp.g);
    sh.nslots = nnz > 0 ? ceil_div(nnz, sh.L) : 0;
    sh.nblocks = sh.nslots > 0 ? ceil_div(sh.nslots, slots_per_block) : 0;
    return sh;
}

bool sddmm_vec_ok(const SddmmParams &a) { return (!a.X || aligned16(a.X)) && aligned16(a.Y); }

struct SddmmLauncher {
    SddmmParams a;
    int64_t nb;
    hipStream_t st;
    template <int VEC, int G>
    nsd_status operator()() {
        probe_begin(NSD_KERNEL_SDDMM, st);
        sddmm_kernel<VEC, G, sddmm_unroll<G>()><<<(unsigned)nb, kBlock, 0, st>>>(a);
        probe_end(NSD_KERNEL_SDDMM, st);
        return check_launch("sddmm_kernel");
    }
};

nsd_status sddmm(SddmmParams a, hipStream_t st) {
    const SddmmShape sh = sddmm_shape(a.nnz, a.k, sddmm_vec_ok(a));
    a.L = sh.L;
    a.nslots = (int32_t)sh.nslots;
    if (sh.nblocks == 0) return NSD_OK;
    SddmmLauncher f{a, sh.nblocks, st};
    return dispatch_width(sh.wp, f);
}

// ------------------------------------------------------------ loss total

// One block: the loss total of part1[0, n1) and part2[0, n2).
__global__ __launch_bounds__(kBlock) void loss_finalize_kernel(const double *part1, int64_t n1,
                                                               const double *part2, int64_t n2,
                                                               double *loss) {
    LossJob job;
    job.p1 = part1;
    job.n1 = n1;
    job.p2 = part2;
    job.n2 = n2;
    job.loss = loss;
    loss_total_block<16>(job);
}

// Block partials of alpha * sum_i x_i * y_i (y NULL: ones) in fp64: block b
// sums elements b*kDotChunk .. in a fixed strided order.
constexpr int kDotItems = 8;
constexpr int64_t kDotChunk = (int64_t)kBlock * kDotItems;

__global__ __launch_bounds__(kBlock) void dot_kernel(int64_t n, const float *x, const float *y,
                                                     double alpha, int64_t per_block,
                                                     double *part) {
    double s = 0.0;
    const int64_t lo = (int64_t)blockIdx.x * per_block;
    const int64_t hi = min(n, lo + per_block);
    for (int64_t i = lo + threadIdx.x; i < hi; i += kBlock)
        s += y ? (double)x[i] * (double)y[i] : (double)x[i];
    const double t = block_sum(s);
    if (threadIdx.x == 0) part[blockIdx.x] = alpha * t;
}

int64_t dot_blocks(int64_t n) {
    return std::max<int64_t>(1, std::min<int64_t>(ceil_div(n, kDotChunk), 2048));
}

nsd_status dot(int64_t n, const float *x, const float *y, double alpha, bool accumulate,
               double *part, double *out, hipStream_t st) {
    const int64_t nb = dot_blocks(n);
    const int64_t per = ceil_div(std::max<int64_t>(n, 1), nb);
    dot_kernel<<<(unsigned)nb, kBlock, 0, st>>>(n, x, y, alpha, per, part);
    NSD_TRY(check_launch("dot_kernel"));
    // accumulate: the old *out is a second partial (read before the one write)
    loss_finalize_kernel<<<1, kBlock, 0, st>>>(part, nb, accumulate ? out : nullptr,
                                               accumulate ? 1 : 0, out);
    return check_launch("loss_finalize_kernel");
}

// y = alpha x + beta y (x NULL: ones; beta 0: y is not read).
__global__ __launch_bounds__(kBlock) void axpby_kernel(int64_t n, float alpha, const float *x,
                                                       float beta, float *y) {
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < n; i += stride) {
        const float ax = alpha * (x ? x[i] : 1.f);
        y[i] = beta == 0.f ? ax : ax + beta * y[i];
    }
}

nsd_status axpby(int64_t n, float alpha, const float *x, float beta, float *y, hipStream_t st) {
    if (n == 0) return NSD_OK;
    const int64_t nb = std::min<int64_t>(ceil_div(n, kBlock), 8192);
    axpby_kernel<<<(unsigned)nb, kBlock, 0, st>>>(n, alpha, x, beta, y);
    return check_launch("axpby_kernel");
}

// out[p] = alpha * [rowidx[p] == colind[p]] over the stored entries.
__global__ __launch_bounds__(kBlock) void diag_keys_kernel(int64_t n, const int32_t *rowidx,
                                                           const int32_t *colind, float alpha,
                                                           float *out) {
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    for (int64_t p = (int64_t)blockIdx.x * kBlock + threadIdx.x; p < n; p += stride)
        out[p] = rowidx[p] == colind[p] ? alpha : 0.f;
}

nsd_status diag_keys(int64_t n, const int32_t *rowidx, const int32_t *colind, float alpha,
                     float *out, hipStream_t st) {
    if (n == 0) return NSD_OK;
    const int64_t nb = std::min<int64_t>(ceil_div(n, kBlock), 8192);
    diag_keys_kernel<<<(unsigned)nb, kBlock, 0, st>>>(n, rowidx, colind, alpha, out);
    return check_launch("diag_keys_kernel");
}

nsd_status loss_finalize(const double *part, int64_t n, double *loss, hipStream_t st) {
    probe_begin(NSD_KERNEL_LOSS, st);
    loss_finalize_kernel<<<1, kBlock, 0, st>>>(part, n, nullptr, 0, loss);
    probe_end(NSD_KERNEL_LOSS, st);
    return check_launch("loss_finalize_kernel");
}

// ------------------------------------------ fused pass of the SpMM gradient

// Row pass of L = 1/2 ||A B||^2 over A's row plan, one slot per item: the C
// rows of the item (gather-reduce) and ||C_i||^2 of the rows completed in it
// into the block's loss partial; a long row's chunk leaves a partial instead.
// Blocks past the items zero the C rows of empty rows.
// Occupancy floor (waves per SIMD), a build-time tuning knob.
#ifdef NSD_FROB_WAVES
#define NSD_FROB_OCCUPANCY __attribute__((amdgpu_waves_per_eu(NSD_FROB_WAVES, 8)))
#else
#define NSD_FROB_OCCUPANCY
#endif

template <int VEC, int G, int U>
__global__ __launch_bounds__(kBlock) NSD_FROB_OCCUPANCY void frob_row_kernel(FrobParams f) {
    constexpr int kSlots = kBlock / G;
    const SgrParams &a = f.rows;
    const int g = threadIdx.x % G;
    const int col = g * VEC;  // k <= G * VEC on this path
    const bool on = col < a.k;
    double lsq = 0.0;
    if ((int)blockIdx.x >= a.item_blocks) {
        zero_segment<VEC>(a, (int64_t)(blockIdx.x - a.item_blocks) * kSlots + threadIdx.x / G, col,
                          on);
    } else {
        const int64_t s = (int64_t)blockIdx.x * kSlots + threadIdx.x / G;
        Vec<VEC> pacc;
        pacc.zero();
        int pseg = -1;
        if (s < a.plan.nitems) {
            pseg = sgr_walk<VEC, G, U>(a, s, col, on, [&](int, const Vec<VEC> &c) {
                if (on)
#pragma unroll
                    for (int e = 0; e < VEC; ++e) lsq += (double)c.v[e] * c.v[e];
            }, pacc);
        }
        store_chunk_partial<VEC, G>(pseg, pacc, a.part, a.plan.chunk_ord, s, a.k, col, on);
    }
    const double t = block_sum(lsq);
    if (threadIdx.x == 0) f.loss_part[blockIdx.x] = 0.5 * t;
}

// C = A B with the loss (row pass, long-row combine with their ||C_i||^2),
// then dB and dA in one linear dual pass over the columns (own row B_j,
// gathered row C_i) with the loss total in one extra block, then the
// long-column combine when there are long columns.
template <int VEC, int G>
static nsd_status launch_frob(FrobParams f, hipStream_t st) {
    constexpr int kSlots = kBlock / G;
    constexpr int U = sgr_unroll<G>();
    f.rows.item_blocks = (int32_t)ceil_div(f.rows.plan.nitems, kSlots);
    f.rows.chunk_stride = chunk_group<G>();
    const int row_blocks = f.rows.item_blocks + (int)ceil_div(f.rows.plan.nempty, kSlots);
    probe_begin(NSD_KERNEL_FROB_ROW, st);
    frob_row_kernel<VEC, G, U><<<row_blocks, kBlock, 0, st>>>(f);
    probe_end(NSD_KERNEL_FROB_ROW, st);
    NSD_TRY(check_launch("frob_row_kernel"));
    NSD_TRY((launch_fix<VEC, G>(f.rows, f.seg_loss, 0.5, st)));
    DualParams d;
    d.pass[0] = f.cols;
    d.npass = 1;
    // the loss total (row partials and long-row partials, complete before
    // the column pass starts) is one extra block of the column pass
    d.early.p1 = f.loss_part;
    d.early.n1 = row_blocks;
    d.early.p2 = f.seg_loss;
    d.early.n2 = f.rows.plan.nlong;
    d.early.loss = f.loss;
    return dual_fused(kDualLin, d, NSD_KERNEL_FROB_COL, LossJob{}, st);
}

int64_t frob_row_blocks(const nsd_plan &rows, int k) {
    const WidthPlan wp = width_plan(k, true);
    const int slots = kBlock / wp.g;
    return ceil_div(rows.nitems, slots) + ceil_div(rows.nempty, slots);
}

bool frob_fused_ok(int k, const void *B, const void *C, const void *dB) {
    return k <= 256 && k % 4 == 0 && aligned16(B) && aligned16(C) && aligned16(dB);
}

struct FrobLauncher {
    FrobParams f;
    hipStream_t st;
    template <int VEC, int G>
    nsd_status operator()() { return launch_frob<VEC, G>(f, st); }
};

nsd_status frob_fused(FrobParams f, hipStream_t st) {
    FrobLauncher fn{f, st};
    return dispatch_width(width_plan(f.rows.k, true), fn);
}

}  // namespace nsd
