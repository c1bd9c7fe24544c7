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

struct JvpParams {
    SgrParams c;             // C = A B: w = A's values, X = B, out = C, part
    SgrParams d;             // the tangent's outputs only: out = dC, part (chunk partials)
    const float *dw = nullptr;  // dA [nnz], A's storage order
    const float *dX = nullptr;  // dB [ncols x k]
};

template <int VEC, int G, int U>
struct JvpSlot {
    const JvpParams &f;
    int64_t s, k, b0;
    int col;
    bool on;
    int row;
    bool carry;
    bool pend = false;  // acc, dacc are chunk partials of segment `row`, not yet stored
    Vec<VEC> acc, dacc;

    __device__ __forceinline__ JvpSlot(const JvpParams &f_, int64_t s_, int col_, bool on_,
                                       int64_t a0, int64_t b0_)
        : f(f_), s(s_), k(f_.c.k), b0(b0_), col(col_), on(on_) {
        row = f.c.segidx[a0];
        carry = a0 > 0 && f.c.segidx[a0 - 1] == row;
        acc.zero();
        dacc.zero();
    }

    __device__ __forceinline__ void flush() {
        if (carry) {
            pend = true;  // a chunk item holds one segment: this is its end
        } else if (on) {
            acc.store(f.c.out + (int64_t)row * k + col);
            dacc.store(f.d.out + (int64_t)row * k + col);
        }
    }

    // Entries [p, p + U): row r, column c, A's value w at storage position
    // pos (padding: weight 0; its tangent weight is read as 0 too).
    __device__ __forceinline__ void batch(int64_t p, const int (&r)[U], const int (&c)[U],
                                          const int (&pos)[U], const float (&w)[U], int, float) {
        float dw[U];
#pragma unroll
        for (int u = 0; u < U; ++u) dw[u] = p + u < b0 ? f.dw[pos[u]] : 0.f;
        Vec<VEC> xv[U], dxv[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (on) {
                xv[u].load(f.c.X + (int64_t)c[u] * k + col);
                dxv[u].load(f.dX + (int64_t)c[u] * k + col);
            } else {
                xv[u].zero();
                dxv[u].zero();
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (r[u] != row) {
                flush();
                row = r[u];
                carry = false;
                acc.zero();
                dacc.zero();
            }
            acc.fma(w[u], xv[u]);
            dacc.fma(dw[u], xv[u]);
            dacc.fma(w[u], dxv[u]);
        }
    }

    __device__ __forceinline__ void finish() {
        if (b0 == f.c.nnz || f.c.segidx[b0] != row) flush();
        else pend = true;  // a chunk of a long segment that goes on
    }
};

template <int VEC, int G, int U>
__global__ __launch_bounds__(kBlock) void jvp_kernel(JvpParams f) {
    constexpr int kSlots = kBlock / G;
    const int g = threadIdx.x % G;
    const int col = blockIdx.y * (G * VEC) + g * VEC;
    const bool on = col < f.c.k;
    if ((int)blockIdx.x >= f.c.item_blocks) {
        const int64_t e = (int64_t)(blockIdx.x - f.c.item_blocks) * kSlots + threadIdx.x / G;
        zero_segment<VEC>(f.c, e, col, on);
        zero_segment<VEC>(f.d, e, col, on);
        return;
    }
    const int64_t s = (int64_t)blockIdx.x * kSlots + threadIdx.x / G;
    Vec<VEC> pc, pd;
    pc.zero();
    pd.zero();
    int pseg = -1;
    if (s < f.c.plan.nitems) {
        const int64_t a0 = f.c.plan.item_ptr[s], b0 = f.c.plan.item_ptr[s + 1];
        JvpSlot<VEC, G, U> st(f, s, col, on, a0, b0);
        walk_item<G, U>(f.c, a0, b0, g, st);
        st.finish();
        if (st.pend) {
            pseg = st.row;
            pc = st.acc;
            pd = st.dacc;
        }
    }
    store_chunk_partial<VEC, G>(pseg, pc, f.c.part, f.c.plan.chunk_ord, s, f.c.k, col, on);
    store_chunk_partial<VEC, G>(pseg, pd, f.d.part, f.c.plan.chunk_ord, s, f.c.k, col, on);
}

// Entries per batch (two rows are gathered per entry): four, measured on
// MI355X for the 16-lane slots of k = 64.
template <int G>
constexpr int jvp_unroll() {
#ifdef NSD_JVP_UNROLL
    return NSD_JVP_UNROLL;
#else
    return 4;
#endif
}

template <int VEC, int G>
static nsd_status launch_jvp(JvpParams f, hipStream_t st) {
    constexpr int kSlots = kBlock / G;
    f.c.item_blocks = (int32_t)ceil_div(f.c.plan.nitems, kSlots);
    f.c.chunk_stride = f.d.chunk_stride = chunk_group<G>();
    const int64_t empty_blocks = ceil_div(f.c.plan.nempty, kSlots);
    dim3 grid((unsigned)(f.c.item_blocks + empty_blocks), (unsigned)ceil_div(f.c.k, G * VEC));
    probe_begin(NSD_KERNEL_JVP, st);
    jvp_kernel<VEC, G, jvp_unroll<G>()><<<grid, kBlock, 0, st>>>(f);
    probe_end(NSD_KERNEL_JVP, st);
    NSD_TRY(check_launch("jvp_kernel"));
    FixJobs fx;
    add_fix(fx, f.c);
    add_fix(fx, f.d);
    return launch_fixes<VEC, G>(fx, st);
}

struct JvpLauncher {
    JvpParams f;
    hipStream_t st;
    template <int VEC, int G>
    nsd_status operator()() { return launch_jvp<VEC, G>(f, st); }
};

}  // namespace nsd

using namespace nsd;

extern "C" {

nsd_status nsd_spmm_jvp(const nsd_csr *A, const float *dAval, const float *B, const float *dB,
                        int32_t k, float *C, float *dC, void *ws, size_t ws_bytes,
                        void *stream) {
    NSD_REQUIRE(A != nullptr, "CSR descriptor is NULL");
    NSD_REQUIRE(A->nrows >= 0 && A->ncols >= 0 && A->nnz >= 0, "negative CSR size");
    NSD_REQUIRE(k >= 1, "k = %d < 1", k);
    NSD_REQUIRE(A->nrows == 0 || (C && dC), "C/dC is NULL");
    if (A->nnz > 0) {
        NSD_REQUIRE(A->rowptr && A->rowidx && A->colind && A->val, "CSR array is NULL");
        NSD_REQUIRE(dAval && B && dB, "dA/B/dB is NULL");
        NSD_REQUIRE(A->plan.item_ptr && A->plan.nitems >= 1,
                    "row plan is not built (nsd_plan_build)");
    }
    hipStream_t st = as_stream(stream);
    const size_t half = (sgr_part_bytes(A->plan, k) + 255) & ~size_t(255);
    if (ws == nullptr || ws_bytes < 2 * half)
        return fail(NSD_ERR_WORKSPACE, "workspace %zu bytes at %p, need %zu", ws_bytes, ws,
                    2 * half);
    JvpParams f;
    f.c.nseg = A->nrows;
    f.c.nnz = A->nnz;
    f.c.k = k;
    f.c.plan = A->plan;
    f.c.segptr = A->rowptr;
    f.c.segidx = A->rowidx;
    f.c.idx = A->colind;
    f.c.w = A->val;
    f.c.X = B;
    f.c.alpha = 1.f;
    f.c.out = C;
    f.c.part = static_cast<float *>(ws);
    f.d = f.c;
    f.d.out = dC;
    f.d.part = reinterpret_cast<float *>(static_cast<char *>(ws) + half);
    f.dw = dAval;
    f.dX = dB;
    if (A->nnz == 0) {
        // empty sums: both outputs are zero
        NSD_TRY(segreduce(f.c, st));
        return segreduce(f.d, st);
    }
    const bool vec = k % 4 == 0 && aligned16(B) && aligned16(dB) && aligned16(C) && aligned16(dC);
    JvpLauncher fn{f, st};
    return dispatch_width(width_plan(k, vec), fn);
}

}  // extern "C"
