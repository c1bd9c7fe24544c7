// Jacobian of the BATAX kernel f(j) = sum_{i,k} beta A(i,j) A(i,k) x(k) with
// respect to x:  J = beta A^T A, a sparse matrix whose pattern is not an
// input's (Example 5; the matrix-kernel benchmarks of Section 7).
//
// The paper's differentiated, normalised program inserts, for every stored
// row r of A, the outer product r x r into the result dictionary.  Here that
// is expand / sort / reduce:
//   1. every ordered pair (p, q) of stored entries of one row becomes a term
//      (j, k, beta * a_p * a_q) with j = col(p), k = col(q); rows are laid
//      out in order, pairs row-major inside a row;
//   2. the terms are sorted stably by k, then stably by j (two radix sorts),
//      so a run of equal (j, k) keeps its terms in row order;
//   3. runs become the keys of J (run heads, a scan); J's row pointers come
//      from the runs' j, its columns from their k;
//   4. the values are the run sums, one thread per run adding its terms in
//      row order in fp64 and rounding once: no float atomics, bitwise
//      reproducible.  (A run is as long as the number of rows two columns
//      share, at most a column's length; a pathologically dense column makes
//      its diagonal run a serial tail, which the fixed order accepts.)
// Keys are structural: a pair whose product is 0 keeps its key, as the
// dictionary insert of the paper's program does.
#include <algorithm>

#include "nsd_internal.hpp"

namespace nsd {

constexpr int kBataxThreads = 256;
constexpr int64_t kBataxMaxPairs = 1LL << 30;  // positions stay in int32

static int64_t bgrid(int64_t n) { return ceil_div(n > 0 ? n : 1, kBataxThreads); }

__global__ void row_pairs_kernel(int32_t nrows, const int32_t *rowptr, int32_t *sq) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= nrows) return;
    const int32_t len = rowptr[i + 1] - rowptr[i];
    sq[i] = len * len;
}

__global__ void pairs_total_kernel(int32_t nrows, const int32_t *rowptr,
                                   unsigned long long *total) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    unsigned long long v = 0;
    if (i < nrows) {
        const unsigned long long len = (unsigned long long)(rowptr[i + 1] - rowptr[i]);
        v = len * len;
    }
    // integer sums are exact in any order
#pragma unroll
    for (int m = kWave / 2; m >= 1; m >>= 1) v += __shfl_xor(v, m, kWave);
    if ((threadIdx.x & (kWave - 1)) == 0 && v) atomicAdd(total, v);
}

// Term t of row i: the pair (p, q) = (u / len, u % len) of the row's
// entries, u = t - off[i]; the row is found by binary search over off.
__global__ void expand_pairs_kernel(int64_t npairs, int32_t nrows, const int32_t *off,
                                    const int32_t *rowptr, const int32_t *colind,
                                    const float *val, float beta, int32_t *key_j,
                                    int32_t *key_k, float *term) {
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= npairs) return;
    int32_t lo = 0, hi = nrows - 1;  // last row with off[row] <= t (rows of length 0 share off)
    while (lo < hi) {
        const int32_t mid = lo + (hi - lo + 1) / 2;
        if (off[mid] <= t) lo = mid;
        else hi = mid - 1;
    }
    const int32_t b = rowptr[lo];
    const int32_t len = rowptr[lo + 1] - b;
    const int32_t u = (int32_t)(t - off[lo]);
    const int32_t p = b + u / len, q = b + u % len;
    key_j[t] = colind[p];
    key_k[t] = colind[q];
    term[t] = (beta * val[p]) * val[q];
}

__global__ void gather_keys_kernel(int64_t n, const int32_t *perm, const int32_t *src,
                                   int32_t *dst) {
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t < n) dst[t] = src[perm[t]];
}

__global__ void pair_heads_kernel(int64_t n, const int32_t *js, const int32_t *ks, int32_t *head) {
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= n) return;
    head[t] = (t == 0 || js[t] != js[t - 1] || ks[t] != ks[t - 1]) ? 1 : 0;
}

// run[t] = index of the run holding sorted term t; heads name J's keys.
__global__ void runs_kernel(int64_t n, const int32_t *head, const int32_t *pos,
                            const int32_t *js, const int32_t *ks, int32_t *run, int32_t *run_j,
                            int32_t *jcolind) {
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= n) return;
    run[t] = pos[t] + head[t] - 1;
    if (head[t]) {
        run_j[pos[t]] = js[t];
        jcolind[pos[t]] = ks[t];
    }
}

// jval[r] = sum of the terms of run r (sorted positions runptr[r] ..
// runptr[r+1], terms reached through perm), in order, in fp64.
__global__ void run_sums_kernel(int32_t nruns, const int32_t *runptr, const int32_t *perm,
                                const float *term, float *jval) {
    const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (r >= nruns) return;
    double s = 0.0;
    for (int32_t t = runptr[r]; t < runptr[r + 1]; ++t) s += (double)term[perm[t]];
    jval[r] = (float)s;
}

// Workspace layout shared by the size query and the call.
struct BataxWs {
    int32_t *sq, *off, *tot;
    int32_t *key_j, *key_k, *kperm, *jg, *js, *perm2, *ks, *head, *pos, *run, *runptr, *run_j;
    float *term;
    void *sort_ws, *scan_ws;
    size_t sort_bytes, scan_bytes;
};

static nsd_status batax_carve(void *ws, int32_t nrows, int32_t n, int64_t P, BataxWs *w,
                              size_t *total) {
    Carver c(ws);
    w->sq = c.take<int32_t>(std::max<int64_t>(nrows, 1));
    w->off = c.take<int32_t>(std::max<int64_t>(nrows, 1));
    w->tot = c.take<int32_t>(64);
    const int64_t Q = std::max<int64_t>(P, 1);
    w->key_j = c.take<int32_t>(Q);
    w->key_k = c.take<int32_t>(Q);
    w->term = c.take<float>(Q);
    w->kperm = c.take<int32_t>(Q);
    w->jg = c.take<int32_t>(Q);
    w->js = c.take<int32_t>(Q);
    w->perm2 = c.take<int32_t>(Q);
    w->ks = c.take<int32_t>(Q);
    w->head = c.take<int32_t>(Q);
    w->pos = c.take<int32_t>(Q);
    w->run = c.take<int32_t>(Q);
    w->runptr = c.take<int32_t>(Q + 1);
    w->run_j = c.take<int32_t>(Q);
    w->sort_bytes = sort_ws_bytes(Q, std::max(n, 1));
    w->scan_bytes = scan_ws_bytes(std::max<int64_t>(Q, nrows));
    // the sort and scan scratch are used one after another
    char *s = c.take<char>((int64_t)std::max(w->sort_bytes, w->scan_bytes));
    w->sort_ws = w->scan_ws = s;
    *total = c.bytes();
    return NSD_OK;
}

static nsd_status check_batax_csr(const nsd_csr *A) {
    NSD_REQUIRE(A != nullptr, "CSR descriptor is NULL");
    NSD_REQUIRE(A->nrows >= 0 && A->ncols >= 0 && A->nnz >= 0, "negative CSR size");
    NSD_REQUIRE(A->rowptr != nullptr, "CSR rowptr is NULL");
    if (A->nnz > 0) {
        NSD_REQUIRE(A->nrows > 0 && A->ncols > 0, "nnz > 0 in an empty shape");
        NSD_REQUIRE(A->colind && A->val, "CSR colind/val is NULL");
    }
    return NSD_OK;
}

}  // namespace nsd

using namespace nsd;

extern "C" {

nsd_status nsd_batax_pairs(const nsd_csr *A, int64_t *npairs, void *ws, size_t ws_bytes,
                           void *stream) {
    NSD_TRY(check_batax_csr(A));
    NSD_REQUIRE(npairs != nullptr, "npairs is NULL");
    NSD_REQUIRE(ws != nullptr && ws_bytes >= 256, "workspace of at least 256 bytes needed");
    hipStream_t st = as_stream(stream);
    auto *total = static_cast<unsigned long long *>(ws);
    NSD_HIP(hipMemsetAsync(total, 0, sizeof(unsigned long long), st));
    if (A->nrows > 0) {
        pairs_total_kernel<<<bgrid(A->nrows), kBataxThreads, 0, st>>>(A->nrows, A->rowptr, total);
        NSD_TRY(check_launch("pairs_total_kernel"));
    }
    unsigned long long h = 0;
    NSD_HIP(hipMemcpyAsync(&h, total, sizeof(h), hipMemcpyDeviceToHost, st));
    NSD_HIP(hipStreamSynchronize(st));
    *npairs = (int64_t)h;
    return NSD_OK;
}

nsd_status nsd_batax_workspace_size(const nsd_csr *A, int64_t npairs, size_t *bytes) {
    NSD_TRY(check_batax_csr(A));
    NSD_REQUIRE(bytes != nullptr, "bytes is NULL");
    NSD_REQUIRE(npairs >= 0, "negative pair count");
    if (npairs >= kBataxMaxPairs)
        return fail(NSD_ERR_TOO_LARGE, "%lld row pairs (at most 2^30)", (long long)npairs);
    BataxWs w;
    return batax_carve(nullptr, A->nrows, A->ncols, npairs, &w, bytes);
}

nsd_status nsd_batax_jacobian(const nsd_csr *A, float beta, int64_t npairs, int32_t *jrowptr,
                              int32_t *jcolind, float *jval, int32_t *nnz_out, void *ws,
                              size_t ws_bytes, void *stream) {
    NSD_TRY(check_batax_csr(A));
    NSD_REQUIRE(jrowptr != nullptr && nnz_out != nullptr, "jrowptr/nnz_out is NULL");
    NSD_REQUIRE(npairs >= 0, "negative pair count");
    if (npairs >= kBataxMaxPairs)
        return fail(NSD_ERR_TOO_LARGE, "%lld row pairs (at most 2^30)", (long long)npairs);
    NSD_REQUIRE(npairs == 0 || (jcolind && jval), "jcolind/jval is NULL");
    size_t need = 0;
    BataxWs w;
    NSD_TRY(batax_carve(nullptr, A->nrows, A->ncols, npairs, &w, &need));
    if (ws == nullptr || ws_bytes < need)
        return fail(NSD_ERR_WORKSPACE, "workspace %zu bytes at %p, need %zu", ws_bytes, ws, need);
    NSD_TRY(batax_carve(ws, A->nrows, A->ncols, npairs, &w, &need));
    hipStream_t st = as_stream(stream);
    const int32_t m = A->nrows, n = A->ncols;
    const int64_t P = npairs;
    if (P == 0) {
        NSD_TRY(segptr_from_sorted(0, n, nullptr, jrowptr, st));
        NSD_HIP(hipStreamSynchronize(st));
        *nnz_out = 0;
        return NSD_OK;
    }
    // 1. term offsets per row and the terms
    row_pairs_kernel<<<bgrid(m), kBataxThreads, 0, st>>>(m, A->rowptr, w.sq);
    NSD_TRY(check_launch("row_pairs_kernel"));
    NSD_TRY(scan_exclusive(w.sq, w.off, m, w.tot, w.scan_ws, st));
    int32_t hp = 0;
    NSD_HIP(hipMemcpyAsync(&hp, w.tot, sizeof(hp), hipMemcpyDeviceToHost, st));
    NSD_HIP(hipStreamSynchronize(st));
    if ((int64_t)hp != P)
        return fail(NSD_ERR_INVALID_ARG, "npairs = %lld, but A's rows give %d pairs",
                    (long long)P, hp);
    expand_pairs_kernel<<<bgrid(P), kBataxThreads, 0, st>>>(P, m, w.off, A->rowptr, A->colind,
                                                            A->val, beta, w.key_j, w.key_k,
                                                            w.term);
    NSD_TRY(check_launch("expand_pairs_kernel"));
    // 2. stable sort by k, then stably by j: (j, k) order, runs in row order
    NSD_TRY(radix_sort_pairs(P, n, w.key_k, nullptr, w.ks, w.kperm, w.sort_ws, st));
    gather_keys_kernel<<<bgrid(P), kBataxThreads, 0, st>>>(P, w.kperm, w.key_j, w.jg);
    NSD_TRY(check_launch("gather_keys_kernel"));
    NSD_TRY(radix_sort_pairs(P, n, w.jg, w.kperm, w.js, w.perm2, w.sort_ws, st));
    gather_keys_kernel<<<bgrid(P), kBataxThreads, 0, st>>>(P, w.perm2, w.key_k, w.ks);
    NSD_TRY(check_launch("gather_keys_kernel"));
    // 3. runs -> keys of J
    pair_heads_kernel<<<bgrid(P), kBataxThreads, 0, st>>>(P, w.js, w.ks, w.head);
    NSD_TRY(check_launch("pair_heads_kernel"));
    NSD_TRY(scan_exclusive(w.head, w.pos, P, w.tot + 1, w.scan_ws, st));
    runs_kernel<<<bgrid(P), kBataxThreads, 0, st>>>(P, w.head, w.pos, w.js, w.ks, w.run, w.run_j,
                                                    jcolind);
    NSD_TRY(check_launch("runs_kernel"));
    int32_t nk = 0;
    NSD_HIP(hipMemcpyAsync(&nk, w.tot + 1, sizeof(nk), hipMemcpyDeviceToHost, st));
    NSD_HIP(hipStreamSynchronize(st));
    NSD_TRY(segptr_from_sorted(P, nk, w.run, w.runptr, st));
    NSD_TRY(segptr_from_sorted(nk, n, w.run_j, jrowptr, st));
    // 4. run sums (terms reached through perm2)
    run_sums_kernel<<<bgrid(nk), kBataxThreads, 0, st>>>(nk, w.runptr, w.perm2, w.term, jval);
    NSD_TRY(check_launch("run_sums_kernel"));
    NSD_HIP(hipStreamSynchronize(st));
    *nnz_out = nk;
    return NSD_OK;
}

}  // extern "C"
