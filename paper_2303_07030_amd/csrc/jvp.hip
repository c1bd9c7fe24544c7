// Forward-mode tangent of the matrix product, the paper's own mode of
// differentiation (Section 4.1: every value is carried with its tangent;
// Section 4.2: tensors of tangents at once).  For C = A B, with a tangent dA
// on A's stored keys and a dense tangent dB:
//     C(i,:)  = sum over stored (i,j) of A(i,j) B(j,:)
//     dC(i,:) = sum over stored (i,j) of dA(i,j) B(j,:) + A(i,j) dB(j,:)
// One pass over A's row plan computes both: per entry the rows B(j,:) and
// dB(j,:) are gathered once each and feed two running sums.  dA is a value
// array aligned 1:1 with A's storage order (its keys are A's).  Long rows
// leave two chunk partials, combined by the shared kernel.
#include <algorithm>

#include "nsd_internal.hpp"
#include "segreduce.hpp"
#include "segreduce_dev.hpp"

namespace nsd {

// Tangents carried by one pass over A (the batch of tangents of Section
// 4.2 is processed in groups of this many; each group reads A and the rows
// of B once for all of its tangents).
constexpr int kJvpGroup = 4;

template <int MB>
struct JvpParams {
    SgrParams c;                // C = A B: w = A's values, X = B, out = C, part
    SgrParams d[MB];            // per tangent: out = dC_t, part (chunk partials)
    const float *dw[MB] = {};   // dA_t [nnz], A's storage order (NULL: no dA)
    const float *dX[MB] = {};   // dB_t [ncols x k] (NULL: no dB)
    int mt = 0;                 // tangents of this launch (<= MB)
    bool primal = true;         // computes and stores C
    bool has_dw = false, has_dX = false;
};

template <int MB, int VEC, int G, int U>
struct JvpSlot {
    const JvpParams<MB> &f;
    int64_t s, k, b0;
    int col;
    bool on;
    int row;
    bool carry;
    bool pend = false;  // acc, dacc are chunk partials of segment `row`, not yet stored
    Vec<VEC> acc, dacc[MB];

    __device__ __forceinline__ JvpSlot(const JvpParams<MB> &f_, int64_t s_, int col_, bool on_,
                                       int64_t a0, int64_t b0_)
        : f(f_), s(s_), k(f_.c.k), b0(b0_), col(col_), on(on_) {
        row = f.c.segidx[a0];
        carry = a0 > 0 && f.c.segidx[a0 - 1] == row;
        zero_all();
    }

    __device__ __forceinline__ void zero_all() {
        acc.zero();
#pragma unroll
        for (int t = 0; t < MB; ++t) dacc[t].zero();
    }

    __device__ __forceinline__ void flush() {
        if (carry) {
            pend = true;  // a chunk item holds one segment: this is its end
        } else if (on) {
            if (f.primal) acc.store(f.c.out + (int64_t)row * k + col);
#pragma unroll
            for (int t = 0; t < MB; ++t)
                if (t < f.mt) dacc[t].store(f.d[t].out + (int64_t)row * k + col);
        }
    }

    // Entries [p, p + U): row r, column c, A's value w at storage position
    // pos (padding: weight 0; its tangent weights are read as 0 too).
    __device__ __forceinline__ void batch(int64_t p, const int (&r)[U], const int (&c)[U],
                                          const int (&pos)[U], const float (&w)[U], int, float) {
        float dw[MB][U];
#pragma unroll
        for (int t = 0; t < MB; ++t)
#pragma unroll
            for (int u = 0; u < U; ++u)
                dw[t][u] = f.has_dw && t < f.mt && p + u < b0 ? f.dw[t][pos[u]] : 0.f;
        Vec<VEC> xv[U], dxv[MB][U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (on) xv[u].load(f.c.X + (int64_t)c[u] * k + col);
            else xv[u].zero();
#pragma unroll
            for (int t = 0; t < MB; ++t) {
                if (on && f.has_dX && t < f.mt) dxv[t][u].load(f.dX[t] + (int64_t)c[u] * k + col);
                else dxv[t][u].zero();
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (r[u] != row) {
                flush();
                row = r[u];
                carry = false;
                zero_all();
            }
            acc.fma(w[u], xv[u]);
#pragma unroll
            for (int t = 0; t < MB; ++t) {
                dacc[t].fma(dw[t][u], xv[u]);
                dacc[t].fma(w[u], dxv[t][u]);
            }
        }
    }

    __device__ __forceinline__ void finish() {
        if (b0 == f.c.nnz || f.c.segidx[b0] != row) flush();
        else pend = true;  // a chunk of a long segment that goes on
    }
};

template <int MB, int VEC, int G, int U>
__global__ __launch_bounds__(kBlock) void jvp_kernel(JvpParams<MB> f) {
    constexpr int kSlots = kBlock / G;
    const int g = threadIdx.x % G;
    const int col = blockIdx.y * (G * VEC) + g * VEC;
    const bool on = col < f.c.k;
    if ((int)blockIdx.x >= f.c.item_blocks) {
        const int64_t e = (int64_t)(blockIdx.x - f.c.item_blocks) * kSlots + threadIdx.x / G;
        if (f.primal) zero_segment<VEC>(f.c, e, col, on);
#pragma unroll
        for (int t = 0; t < MB; ++t)
            if (t < f.mt) zero_segment<VEC>(f.d[t], e, col, on);
        return;
    }
    const int64_t s = (int64_t)blockIdx.x * kSlots + threadIdx.x / G;
    Vec<VEC> pc, pd[MB];
    pc.zero();
#pragma unroll
    for (int t = 0; t < MB; ++t) pd[t].zero();
    int pseg = -1;
    if (s < f.c.plan.nitems) {
        const int64_t a0 = f.c.plan.item_ptr[s], b0 = f.c.plan.item_ptr[s + 1];
        JvpSlot<MB, VEC, G, U> st(f, s, col, on, a0, b0);
        walk_item<G, U>(f.c, a0, b0, g, st);
        st.finish();
        if (st.pend) {
            pseg = st.row;
            pc = st.acc;
#pragma unroll
            for (int t = 0; t < MB; ++t) pd[t] = st.dacc[t];
        }
    }
    if (f.primal)
        store_chunk_partial<VEC, G>(pseg, pc, f.c.part, f.c.plan.chunk_ord, s, f.c.k, col, on);
#pragma unroll
    for (int t = 0; t < MB; ++t)
        if (t < f.mt)
            store_chunk_partial<VEC, G>(pseg, pd[t], f.d[t].part, f.c.plan.chunk_ord, s, f.c.k,
                                        col, on);
}

// Entries per batch (two rows are gathered per entry and tangent): four
// for one tangent, measured on MI355X for the 16-lane slots of k = 64; two
// for a group, whose slots hold a row of registers per tangent.
template <int MB, int G>
constexpr int jvp_unroll() {
#ifdef NSD_JVP_UNROLL
    return NSD_JVP_UNROLL;
#else
    return MB == 1 ? 4 : 2;
#endif
}

template <int MB, int VEC, int G>
static nsd_status launch_jvp(JvpParams<MB> f, hipStream_t st) {
    constexpr int kSlots = kBlock / G;
    f.c.item_blocks = (int32_t)ceil_div(f.c.plan.nitems, kSlots);
    f.c.chunk_stride = chunk_group<G>();
    for (int t = 0; t < MB; ++t) f.d[t].chunk_stride = f.c.chunk_stride;
    const int64_t empty_blocks = ceil_div(f.c.plan.nempty, kSlots);
    dim3 grid((unsigned)(f.c.item_blocks + empty_blocks), (unsigned)ceil_div(f.c.k, G * VEC));
    probe_begin(NSD_KERNEL_JVP, st);
    jvp_kernel<MB, VEC, G, jvp_unroll<MB, G>()><<<grid, kBlock, 0, st>>>(f);
    probe_end(NSD_KERNEL_JVP, st);
    NSD_TRY(check_launch("jvp_kernel"));
    FixJobs fx;
    if (f.primal) add_fix(fx, f.c);
    for (int t = 0; t < f.mt; ++t) add_fix(fx, f.d[t]);
    return launch_fixes<VEC, G>(fx, st);
}

template <int MB>
struct JvpLauncher {
    JvpParams<MB> f;
    hipStream_t st;
    template <int VEC, int G>
    nsd_status operator()() { return launch_jvp<MB, VEC, G>(f, st); }
};

static_assert(kJvpGroup + 1 <= kMaxFixJobs, "a group's combine jobs fit one launch");

// Bytes of one output's chunk partials, rounded to 256.
static size_t jvp_part_bytes(const nsd_plan &plan, int32_t k) {
    return (sgr_part_bytes(plan, k) + 255) & ~size_t(255);
}

static nsd_status check_jvp_csr(const nsd_csr *A, int32_t k) {
    NSD_REQUIRE(A != nullptr, "CSR descriptor is NULL");
    NSD_REQUIRE(A->nrows >= 0 && A->ncols >= 0 && A->nnz >= 0, "negative CSR size");
    NSD_REQUIRE(k >= 1, "k = %d < 1", k);
    if (A->nnz > 0) {
        NSD_REQUIRE(A->rowptr && A->rowidx && A->colind && A->val, "CSR array is NULL");
        NSD_REQUIRE(A->plan.item_ptr && A->plan.nitems >= 1,
                    "row plan is not built (nsd_plan_build)");
    }
    return NSD_OK;
}

static SgrParams jvp_rows(const nsd_csr *A, const float *B, int32_t k, float *out, float *part) {
    SgrParams c;
    c.nseg = A->nrows;
    c.nnz = A->nnz;
    c.k = k;
    c.plan = A->plan;
    c.segptr = A->rowptr;
    c.segidx = A->rowidx;
    c.idx = A->colind;
    c.w = A->val;
    c.X = B;
    c.alpha = 1.f;
    c.out = out;
    c.part = part;
    return c;
}

}  // namespace nsd


using namespace nsd;

extern "C" {

nsd_status nsd_spmm_jvp(const nsd_csr *A, const float *dAval, const float *B, const float *dB,
                        int32_t k, float *C, float *dC, void *ws, size_t ws_bytes,
                        void *stream) {
    NSD_TRY(check_jvp_csr(A, k));
    NSD_REQUIRE(A->nrows == 0 || (C && dC), "C/dC is NULL");
    if (A->nnz > 0) NSD_REQUIRE(dAval && B && dB, "dA/B/dB is NULL");
    hipStream_t st = as_stream(stream);
    const size_t half = jvp_part_bytes(A->plan, k);
    if (ws == nullptr || ws_bytes < 2 * half)
        return fail(NSD_ERR_WORKSPACE, "workspace %zu bytes at %p, need %zu", ws_bytes, ws,
                    2 * half);
    JvpParams<1> f;
    f.c = jvp_rows(A, B, k, C, static_cast<float *>(ws));
    f.d[0] = f.c;
    f.d[0].out = dC;
    f.d[0].part = reinterpret_cast<float *>(static_cast<char *>(ws) + half);
    f.dw[0] = dAval;
    f.dX[0] = dB;
    f.mt = 1;
    f.has_dw = f.has_dX = true;
    if (A->nnz == 0) {
        // empty sums: both outputs are zero
        NSD_TRY(segreduce(f.c, st));
        return segreduce(f.d[0], st);
    }
    const bool vec = k % 4 == 0 && aligned16(B) && aligned16(dB) && aligned16(C) && aligned16(dC);
    JvpLauncher<1> fn{f, st};
    return dispatch_width(width_plan(k, vec), fn);
}

nsd_status nsd_spmm_jvp_batch_workspace_size(const nsd_csr *A, int32_t k, size_t *bytes) {
    NSD_REQUIRE(bytes != nullptr, "bytes is NULL");
    NSD_TRY(check_jvp_csr(A, k));
    *bytes = (size_t)(kJvpGroup + 1) * jvp_part_bytes(A->plan, k);
    return NSD_OK;
}

nsd_status nsd_spmm_jvp_batch(const nsd_csr *A, int32_t m, const float *dAval, const float *B,
                              const float *dB, int32_t k, float *C, float *dC, void *ws,
                              size_t ws_bytes, void *stream) {
    NSD_TRY(check_jvp_csr(A, k));
    NSD_REQUIRE(m >= 0, "m = %d < 0", m);
    NSD_REQUIRE(A->nrows == 0 || m == 0 || dC != nullptr, "dC is NULL");
    if (A->nnz > 0) NSD_REQUIRE(B != nullptr, "B is NULL");
    hipStream_t st = as_stream(stream);
    const size_t one = jvp_part_bytes(A->plan, k);
    const size_t need = (size_t)(kJvpGroup + 1) * one;
    if (ws == nullptr || ws_bytes < need)
        return fail(NSD_ERR_WORKSPACE, "workspace %zu bytes at %p, need %zu", ws_bytes, ws,
                    need);
    char *w = static_cast<char *>(ws);
    const int64_t nnz = A->nnz, xstride = (int64_t)A->ncols * k, ostride = (int64_t)A->nrows * k;
    const bool vec0 = k % 4 == 0 && aligned16(B) && (dB == nullptr || aligned16(dB)) &&
                      (C == nullptr || aligned16(C)) && (dC == nullptr || aligned16(dC));
    // groups of tangents, C with the first (or alone when m == 0)
    for (int32_t t0 = 0; t0 < m || (t0 == 0 && C != nullptr); t0 += kJvpGroup) {
        JvpParams<kJvpGroup> f;
        f.c = jvp_rows(A, B, k, C, reinterpret_cast<float *>(w));
        f.primal = t0 == 0 && C != nullptr;
        f.mt = std::min<int32_t>(kJvpGroup, std::max<int32_t>(m - t0, 0));
        f.has_dw = dAval != nullptr;
        f.has_dX = dB != nullptr;
        for (int t = 0; t < f.mt; ++t) {
            f.d[t] = f.c;
            f.d[t].out = dC + (t0 + t) * ostride;
            f.d[t].part = reinterpret_cast<float *>(w + (size_t)(t + 1) * one);
            f.dw[t] = dAval ? dAval + (t0 + t) * nnz : nullptr;
            f.dX[t] = dB ? dB + (t0 + t) * xstride : nullptr;
        }
        if (A->nnz == 0) {
            if (f.primal) NSD_TRY(segreduce(f.c, st));
            for (int t = 0; t < f.mt; ++t) NSD_TRY(segreduce(f.d[t], st));
            continue;
        }
        JvpLauncher<kJvpGroup> fn{f, st};
        NSD_TRY(dispatch_width(width_plan(k, vec0), fn));
    }
    return NSD_OK;
}

}  // extern "C"
