/*
 * nsd_oracle.c -- fp64 reference for the sparse-gradient path.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the CPU
 * baseline of the benchmark load this file; the library never does.  It
 * shares no code, header, table or helper with the HIP implementation.
 *
 * A sparse operand is a dictionary of keys (DOK): an open-addressing hash
 * from a packed coordinate to a double.  It follows the semi-ring dictionary
 * of the paper (Section 2.2, "Semi-ring Dictionaries", and the SDQL lookup /
 * singleton / sum constructs):
 *   - looking up a key that is not stored yields 0 (the additive identity);
 *   - inserting a key that is already stored adds to its value, the "+="
 *     that the paper's code generation uses for a singleton inside a sum
 *     (Section 5.5, destination-passing style and C++ generation);
 *   - every reduction iterates only the stored keys, the way `sum(<k,v> in d)`
 *     does, so the work is proportional to the number of stored keys.
 *
 * Gradients are the reverse-mode gradients of each loss written out by hand.
 * By the correctness theorem of tensorized forward-mode AD (Section 6.4) the
 * paper's `gradient e x` computes the same values; w.r.t. a sparse operand it
 * is keyed by the operand's stored keys because `onehot` iterates only those
 * keys (Section 4.3, the gradient API figure).
 *
 * Every floating-point output has a companion "mag": the same expression
 * evaluated on the absolute values of every input term (a subtraction becomes
 * an addition).  |fl(y) - y| <= c * u * mag(y) bounds the rounding error of any
 * summation order, which is what the parity tolerance is measured against.
 *
 * Dense operands are row-major double arrays (the dense row-major storage of
 * Section 5.3: element (i, j) of an r x c matrix sits at i * c + j).
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <math.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/*
 * Threads.  The loss scans sum fixed chunks of the hash table in chunk order;
 * the gradient loops split their OUTPUTS by owner (output index modulo the
 * thread count): every thread scans all stored keys and accumulates only into
 * the outputs it owns.  Each output therefore receives its terms in the same
 * slot order whatever the thread count, and the results are bitwise those of
 * one thread.
 */
void orc_set_threads(int n)
{
#ifdef _OPENMP
    omp_set_num_threads(n > 0 ? n : 1);
#else
    (void)n;
#endif
}

int orc_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* number of threads of the enclosing parallel region and this one's index */
static int orc_nthr(void)
{
#ifdef _OPENMP
    return omp_get_num_threads();
#else
    return 1;
#endif
}

static int orc_tid(void)
{
#ifdef _OPENMP
    return omp_get_thread_num();
#else
    return 0;
#endif
}

/* ------------------------------------------------------------------ DOK */

typedef struct orc_dok {
    int64_t cap;     /* number of slots, a power of two */
    int64_t n;       /* number of stored keys */
    int64_t *key;    /* packed coordinate, -1 marks an empty slot */
    double *val;     /* value stored under the key */
    int64_t *first;  /* index of the insertion that created the key */
    int32_t order;   /* 2 (matrix) to ORC_MAX_ORDER */
    int64_t dims[6];
} orc_dok;

#define ORC_MAX_ORDER 6

static uint64_t orc_hash(uint64_t x)
{   /* splitmix64 finaliser */
    x ^= x >> 30; x *= 0xbf58476d1ce4e5b9ULL;
    x ^= x >> 27; x *= 0x94d049bb133111ebULL;
    x ^= x >> 31;
    return x;
}

static int64_t dok_slot(const orc_dok *d, int64_t k)
{
    int64_t mask = d->cap - 1;
    int64_t s = (int64_t)(orc_hash((uint64_t)k) & (uint64_t)mask);
    while (d->key[s] != -1 && d->key[s] != k)
        s = (s + 1) & mask;
    return s;
}

static orc_dok *dok_new(int32_t order, const int64_t *dims, int64_t expected)
{
    orc_dok *d = (orc_dok *)calloc(1, sizeof(orc_dok));
    int64_t cap = 16;
    while (cap < 2 * expected + 16) cap <<= 1;
    d->cap = cap;
    d->order = order;
    for (int i = 0; i < ORC_MAX_ORDER; ++i) d->dims[i] = i < order ? dims[i] : 1;
    d->key = (int64_t *)malloc(sizeof(int64_t) * cap);
    d->val = (double *)malloc(sizeof(double) * cap);
    d->first = (int64_t *)malloc(sizeof(int64_t) * cap);
    memset(d->key, 0xff, sizeof(int64_t) * cap);
    return d;
}

/* semi-ring insert: a new key takes the value, a stored key adds it */
static void dok_add(orc_dok *d, int64_t k, double v, int64_t tag)
{
    int64_t s = dok_slot(d, k);
    if (d->key[s] == -1) {
        d->key[s] = k; d->val[s] = v; d->first[s] = tag; d->n++;
    } else {
        d->val[s] += v;
    }
}

/* lookup: an absent key reads as 0 */
static double dok_get(const orc_dok *d, int64_t k, int *present)
{
    int64_t s = dok_slot(d, k);
    if (present) *present = d->key[s] == k;
    return d->key[s] == k ? d->val[s] : 0.0;
}

static void unpack2(const orc_dok *d, int64_t k, int64_t *i, int64_t *j)
{
    *i = k / d->dims[1]; *j = k % d->dims[1];
}

static void unpack3(const orc_dok *d, int64_t k, int64_t *i, int64_t *j, int64_t *l)
{
    *i = k / (d->dims[1] * d->dims[2]);
    *j = (k / d->dims[2]) % d->dims[1];
    *l = k % d->dims[2];
}

static void unpackn(const orc_dok *d, int64_t k, int64_t *c);

orc_dok *orc_dok_build2(int64_t nr, int64_t nc, int64_t nnz, const int32_t *row,
                        const int32_t *col, const float *val)
{
    int64_t dims[3] = {nr, nc, 1};
    orc_dok *d = dok_new(2, dims, nnz);
    for (int64_t p = 0; p < nnz; ++p)
        dok_add(d, (int64_t)row[p] * nc + col[p], val ? (double)val[p] : 1.0, p);
    return d;
}

orc_dok *orc_dok_build3(int64_t d0, int64_t d1, int64_t d2, int64_t nnz,
                        const int32_t *i, const int32_t *j, const int32_t *l,
                        const float *val)
{
    int64_t dims[3] = {d0, d1, d2};
    orc_dok *d = dok_new(3, dims, nnz);
    for (int64_t p = 0; p < nnz; ++p)
        dok_add(d, ((int64_t)i[p] * d1 + j[p]) * d2 + l[p], (double)val[p], p);
    return d;
}

void orc_dok_free(orc_dok *d)
{
    if (!d) return;
    free(d->key); free(d->val); free(d->first); free(d);
}

int64_t orc_dok_nkeys(const orc_dok *d) { return d->n; }

/* value stored under each queried coordinate (0 if absent) */
void orc_dok_lookup2(const orc_dok *d, int64_t nq, const int32_t *qi, const int32_t *qj,
                     double *out, int8_t *present)
{
    for (int64_t q = 0; q < nq; ++q) {
        int pr;
        out[q] = dok_get(d, (int64_t)qi[q] * d->dims[1] + qj[q], &pr);
        if (present) present[q] = (int8_t)pr;
    }
}

/* ---------------------------------------------------------- sorted emission */

typedef struct { int64_t key; int64_t tag; } kt_pair;

static int cmp_kt(const void *a, const void *b)
{
    const kt_pair *x = (const kt_pair *)a, *y = (const kt_pair *)b;
    if (x->key != y->key) return x->key < y->key ? -1 : 1;
    if (x->tag != y->tag) return x->tag < y->tag ? -1 : 1;
    return 0;
}

/*
 * COO -> CSR: the stored keys of a matrix DOK in (row, col) order.
 * The matrix CSR storage of Section 5.3 keeps unique keys; duplicates in the
 * input were already summed by the semi-ring insert.  For every output slot
 * `first` is the input position of the first occurrence of that key.
 * rowptr has nr+1 entries; colind / val / first have n entries.
 */
int64_t orc_coo_to_csr(const orc_dok *d, int32_t *rowptr, int32_t *colind, double *val,
                       int64_t *first)
{
    int64_t n = d->n, m = 0;
    kt_pair *kp = (kt_pair *)malloc(sizeof(kt_pair) * (n ? n : 1));
    for (int64_t s = 0; s < d->cap; ++s)
        if (d->key[s] != -1) { kp[m].key = d->key[s]; kp[m].tag = s; ++m; }
    qsort(kp, (size_t)n, sizeof(kt_pair), cmp_kt);
    int64_t nr = d->dims[0];
    for (int64_t r = 0; r <= nr; ++r) rowptr[r] = 0;
    for (int64_t p = 0; p < n; ++p) {
        int64_t i, j;
        unpack2(d, kp[p].key, &i, &j);
        colind[p] = (int32_t)j;
        val[p] = d->val[kp[p].tag];
        first[p] = d->first[kp[p].tag];
        rowptr[i + 1]++;
    }
    for (int64_t r = 0; r < nr; ++r) rowptr[r + 1] += rowptr[r];
    free(kp);
    return n;
}

/*
 * Stable sort of positions 0..n-1 by an integer key in [0, nkeys):
 * perm[q] = position placed at q; sorted_key[q] = key[perm[q]];
 * segptr[c] = first q with key >= c (nkeys+1 entries).
 * With key = CSR column indices this is CSR -> CSC (the CSC storage the paper
 * says is expressed like CSR, Section 5.3); with key = one coordinate of a
 * 3-tensor it is that mode's index.  Stability (ties kept in position order)
 * is part of the definition: rows ascend inside each CSC column.
 */
void orc_stable_sort_by_key(int64_t n, const int32_t *key, int64_t nkeys,
                            int32_t *segptr, int32_t *sorted_key, int32_t *perm)
{
    kt_pair *kp = (kt_pair *)malloc(sizeof(kt_pair) * (n ? n : 1));
    for (int64_t p = 0; p < n; ++p) { kp[p].key = key[p]; kp[p].tag = p; }
    qsort(kp, (size_t)n, sizeof(kt_pair), cmp_kt);
    for (int64_t c = 0; c <= nkeys; ++c) segptr[c] = 0;
    for (int64_t q = 0; q < n; ++q) {
        perm[q] = (int32_t)kp[q].tag;
        sorted_key[q] = (int32_t)kp[q].key;
        segptr[kp[q].key + 1]++;
    }
    for (int64_t c = 0; c < nkeys; ++c) segptr[c + 1] += segptr[c];
    free(kp);
}

/* ------------------------------------------------------ selection helper */

/* map[id] = position of id in sel, or -1; sel == NULL selects every id */
static int64_t *select_map(int64_t n, int64_t nsel, const int32_t *sel)
{
    int64_t *map = (int64_t *)malloc(sizeof(int64_t) * (n ? n : 1));
    if (!sel) {
        for (int64_t x = 0; x < n; ++x) map[x] = x;
    } else {
        for (int64_t x = 0; x < n; ++x) map[x] = -1;
        for (int64_t s = 0; s < nsel; ++s) map[sel[s]] = s;
    }
    return map;
}

/* --------------------------------------------------- matrix products */

/*
 * SpMM / SpMV, from the matrix-matrix product in Logical SDQLite
 * (Section 3): C(i,:) = sum over stored (i, j, a) of a * B(j,:).
 * Only rows listed in sel are produced (sel == NULL: all nr rows), into
 * out[s*k ...].  B == NULL means an all-ones B.  Bmag, if given, replaces
 * |B| in the magnitude.
 */
void orc_spmm(const orc_dok *A, const double *B, const double *Bmag, int64_t k,
              int64_t nsel, const int32_t *sel, double *out, double *outmag)
{
    int64_t nr = A->dims[0];
    int64_t *map = select_map(nr, nsel, sel);
    int64_t rows = sel ? nsel : nr;
    memset(out, 0, sizeof(double) * rows * k);
    memset(outmag, 0, sizeof(double) * rows * k);
#pragma omp parallel
    {
    const int nt = orc_nthr(), me = orc_tid();
    for (int64_t s = 0; s < A->cap; ++s) {
        if (A->key[s] == -1) continue;
        int64_t i, j;
        unpack2(A, A->key[s], &i, &j);
        int64_t o = map[i];
        if (o < 0 || o % nt != me) continue;
        double a = A->val[s];
        for (int64_t c = 0; c < k; ++c) {
            double b = B ? B[j * k + c] : 1.0;
            double bm = Bmag ? Bmag[j * k + c] : fabs(b);
            out[o * k + c] += a * b;
            outmag[o * k + c] += fabs(a) * bm;
        }
    }
    }
    free(map);
}

/*
 * Transposed product, the gradient w.r.t. a dense right operand (the reverse
 * gradient that Sections 4.2-4.3 produce for the matrix product of Section 3):
 * out(j,:) = alpha * sum over stored (i, j, a) of a * G(i,:).
 * G == NULL means all ones (k must then be the output width, e.g. 1 for the
 * column sums of SMVM's gradient).  Only columns listed in sel are produced.
 */
void orc_spmm_t(const orc_dok *A, const double *G, const double *Gmag, int64_t k,
                double alpha, int64_t nsel, const int32_t *sel, double *out,
                double *outmag)
{
    int64_t nc = A->dims[1];
    int64_t *map = select_map(nc, nsel, sel);
    int64_t cols = sel ? nsel : nc;
    memset(out, 0, sizeof(double) * cols * k);
    memset(outmag, 0, sizeof(double) * cols * k);
#pragma omp parallel
    {
    const int nt = orc_nthr(), me = orc_tid();
    for (int64_t s = 0; s < A->cap; ++s) {
        if (A->key[s] == -1) continue;
        int64_t i, j;
        unpack2(A, A->key[s], &i, &j);
        int64_t o = map[j];
        if (o < 0 || o % nt != me) continue;
        double a = A->val[s];
        for (int64_t c = 0; c < k; ++c) {
            double g = G ? G[i * k + c] : 1.0;
            double gm = Gmag ? Gmag[i * k + c] : fabs(g);
            out[o * k + c] += alpha * a * g;
            outmag[o * k + c] += fabs(alpha * a) * gm;
        }
    }
    }
    free(map);
}

/*
 * SDDMM, the gradient w.r.t. the sparse operand (keyed by its stored keys,
 * since `onehot` iterates only those, Section 4.3): for every queried
 * coordinate (qi, qj) that is a stored key of A,
 *   out = alpha * sum_c X(qi, c) * Y(qj, c);
 * a coordinate that is not stored gets 0, because the one-hot seed of the
 * gradient API only ranges over stored keys.  X == NULL means ones.
 * Xmag / Ymag, if given, replace |X| / |Y| in the magnitude.
 */
void orc_sddmm(const orc_dok *A, const double *X, const double *Xmag, const double *Y,
               const double *Ymag, int64_t k, double alpha, int64_t nq,
               const int32_t *qi, const int32_t *qj, double *out, double *outmag)
{
#pragma omp parallel for schedule(static)
    for (int64_t q = 0; q < nq; ++q) {
        int pr;
        int64_t i = qi[q], j = qj[q];
        dok_get(A, i * A->dims[1] + j, &pr);
        double acc = 0.0, mag = 0.0;
        if (pr) {
            for (int64_t c = 0; c < k; ++c) {
                double x = X ? X[i * k + c] : 1.0;
                double xm = Xmag ? Xmag[i * k + c] : fabs(x);
                double y = Y[j * k + c];
                double ym = Ymag ? Ymag[j * k + c] : fabs(y);
                acc += x * y;
                mag += xm * ym;
            }
        }
        out[q] = alpha * acc;
        outmag[q] = fabs(alpha) * mag;
    }
}

/* ----------------------------------------------------------------- losses */

/* deterministic parallel scan over the stored keys: fixed chunks summed in
 * chunk order */
#define ORC_CHUNKS 256

static void chunk_bounds(int64_t cap, int c, int64_t *lo, int64_t *hi)
{
    *lo = cap * c / ORC_CHUNKS;
    *hi = cap * (c + 1) / ORC_CHUNKS;
}

/* sum(A . x) with x dense (the SMVM kernel of Section 7.1): L = sum over stored
 * (i, j, a) of a * x(j) */
void orc_loss_sum_spmv(const orc_dok *A, const double *x, double *loss, double *mag)
{
    double L = 0.0, M = 0.0;
    for (int64_t s = 0; s < A->cap; ++s) {
        if (A->key[s] == -1) continue;
        int64_t i, j;
        unpack2(A, A->key[s], &i, &j);
        L += A->val[s] * x[j];
        M += fabs(A->val[s] * x[j]);
    }
    *loss = L; *mag = M;
}

/* L = 1/2 * sum of C(i,c)^2 over a dense n x k array (a plain sum over a
 * dense array, Section 3); mag uses Cmag */
void orc_loss_half_sq(int64_t n, const double *C, const double *Cmag, double *loss,
                      double *mag)
{
    double L = 0.0, M = 0.0;
    for (int64_t e = 0; e < n; ++e) { L += C[e] * C[e]; M += Cmag[e] * Cmag[e]; }
    *loss = 0.5 * L; *mag = 0.5 * M;
}

/* bilinear form of the GNN layer (a sum over A's stored keys, Section 2.2):
 * L = sum over stored (i, j, a) of
 * a * <G(i,:), H(j,:)>  ( = sum of (A H) o G ) */
void orc_loss_bilinear(const orc_dok *A, const double *G, const double *H, int64_t k,
                       double *loss, double *mag)
{
    double part[ORC_CHUNKS], partm[ORC_CHUNKS];
#pragma omp parallel for schedule(dynamic, 1)
    for (int c = 0; c < ORC_CHUNKS; ++c) {
        int64_t lo, hi;
        chunk_bounds(A->cap, c, &lo, &hi);
        double L = 0.0, M = 0.0;
        for (int64_t s = lo; s < hi; ++s) {
            if (A->key[s] == -1) continue;
            int64_t i, j;
            unpack2(A, A->key[s], &i, &j);
            double a = A->val[s], dot = 0.0, dm = 0.0;
            for (int64_t f = 0; f < k; ++f) {
                dot += G[i * k + f] * H[j * k + f];
                dm += fabs(G[i * k + f] * H[j * k + f]);
            }
            L += a * dot;
            M += fabs(a) * dm;
        }
        part[c] = L; partm[c] = M;
    }
    double L = 0.0, M = 0.0;
    for (int c = 0; c < ORC_CHUNKS; ++c) { L += part[c]; M += partm[c]; }
    *loss = L; *mag = M;
}

/* ------------------------------------------- sparse matrix factorisation */

/* residual of one stored entry: r = a - <U(i,:), V(j,:)>, with its magnitude */
static double mf_resid(const double *U, const double *V, int64_t k, int64_t i, int64_t j,
                       double a, double *rmag)
{
    double dot = 0.0, dm = 0.0;
    for (int64_t c = 0; c < k; ++c) {
        dot += U[i * k + c] * V[j * k + c];
        dm += fabs(U[i * k + c] * V[j * k + c]);
    }
    *rmag = fabs(a) + dm;
    return a - dot;
}

/* L = sum over stored (i, j, a) of (a - <U_i, V_j>)^2 (a sum over the stored
 * keys, Section 2.2) */
void orc_mf_loss(const orc_dok *A, const double *U, const double *V, int64_t k,
                 double *loss, double *mag)
{
    double part[ORC_CHUNKS], partm[ORC_CHUNKS];
#pragma omp parallel for schedule(dynamic, 1)
    for (int c = 0; c < ORC_CHUNKS; ++c) {
        int64_t lo, hi;
        chunk_bounds(A->cap, c, &lo, &hi);
        double L = 0.0, M = 0.0;
        for (int64_t s = lo; s < hi; ++s) {
            if (A->key[s] == -1) continue;
            int64_t i, j;
            unpack2(A, A->key[s], &i, &j);
            double rm, r = mf_resid(U, V, k, i, j, A->val[s], &rm);
            L += r * r;
            M += rm * rm;
        }
        part[c] = L; partm[c] = M;
    }
    double L = 0.0, M = 0.0;
    for (int c = 0; c < ORC_CHUNKS; ++c) { L += part[c]; M += partm[c]; }
    *loss = L; *mag = M;
}

/* residual at queried coordinates (0 where not stored: the lookup of an
 * absent key, Section 2.2) */
void orc_mf_resid(const orc_dok *A, const double *U, const double *V, int64_t k,
                  int64_t nq, const int32_t *qi, const int32_t *qj, double *r,
                  double *rmag)
{
    for (int64_t q = 0; q < nq; ++q) {
        int pr;
        double a = dok_get(A, (int64_t)qi[q] * A->dims[1] + qj[q], &pr);
        if (!pr) { r[q] = 0.0; rmag[q] = 0.0; continue; }
        r[q] = mf_resid(U, V, k, qi[q], qj[q], a, &rmag[q]);
    }
}

/*
 * Reverse gradients of the factorisation loss (Sections 4.2-4.3):
 * mode 0: dU(i,:) = -2 * sum over stored (i, j) of r_ij * V(j,:)
 * mode 1: dV(j,:) = -2 * sum over stored (i, j) of r_ij * U(i,:)
 * for the selected rows of dU (mode 0) or of dV (mode 1).
 */
void orc_mf_grad(const orc_dok *A, const double *U, const double *V, int64_t k, int mode,
                 int64_t nsel, const int32_t *sel, double *out, double *outmag)
{
    int64_t n = A->dims[mode];
    int64_t *map = select_map(n, nsel, sel);
    int64_t rows = sel ? nsel : n;
    memset(out, 0, sizeof(double) * rows * k);
    memset(outmag, 0, sizeof(double) * rows * k);
#pragma omp parallel
    {
    const int nt = orc_nthr(), me = orc_tid();
    for (int64_t s = 0; s < A->cap; ++s) {
        if (A->key[s] == -1) continue;
        int64_t i, j;
        unpack2(A, A->key[s], &i, &j);
        int64_t o = map[mode == 0 ? i : j];
        if (o < 0 || o % nt != me) continue;
        double rm, r = mf_resid(U, V, k, i, j, A->val[s], &rm);
        const double *other = mode == 0 ? V + j * k : U + i * k;
        for (int64_t c = 0; c < k; ++c) {
            out[o * k + c] += -2.0 * r * other[c];
            outmag[o * k + c] += 2.0 * rm * fabs(other[c]);
        }
    }
    }
    free(map);
}

/* --------------------------------------------------------- CP decomposition */

/* model value m = sum_r F1(i,r) F2(j,r) F3(l,r) and residual R = x - m */
static double cp_resid(const double *F1, const double *F2, const double *F3, int64_t R,
                       int64_t i, int64_t j, int64_t l, double x, double *rmag)
{
    double m = 0.0, mm = 0.0;
    for (int64_t r = 0; r < R; ++r) {
        double t = F1[i * R + r] * F2[j * R + r] * F3[l * R + r];
        m += t;
        mm += fabs(t);
    }
    *rmag = fabs(x) + mm;
    return x - m;
}

/* L = 1/2 * sum over stored (i, j, l, x) of (x - m_ijl)^2 (a sum over the
 * stored keys of an order-3 tensor, Sections 2.2 and 3) */
void orc_cp_loss(const orc_dok *X, const double *F1, const double *F2, const double *F3,
                 int64_t R, double *loss, double *mag)
{
    double part[ORC_CHUNKS], partm[ORC_CHUNKS];
#pragma omp parallel for schedule(dynamic, 1)
    for (int c = 0; c < ORC_CHUNKS; ++c) {
        int64_t lo, hi;
        chunk_bounds(X->cap, c, &lo, &hi);
        double L = 0.0, M = 0.0;
        for (int64_t s = lo; s < hi; ++s) {
            if (X->key[s] == -1) continue;
            int64_t i, j, l;
            unpack3(X, X->key[s], &i, &j, &l);
            double rm, r = cp_resid(F1, F2, F3, R, i, j, l, X->val[s], &rm);
            L += r * r;
            M += rm * rm;
        }
        part[c] = L; partm[c] = M;
    }
    double L = 0.0, M = 0.0;
    for (int c = 0; c < ORC_CHUNKS; ++c) { L += part[c]; M += partm[c]; }
    *loss = 0.5 * L; *mag = 0.5 * M;
}

/* residual (the gradient w.r.t. the stored values, keyed by X's keys,
 * Section 4.3) at queried coordinates */
void orc_cp_resid(const orc_dok *X, const double *F1, const double *F2, const double *F3,
                  int64_t R, int64_t nq, const int32_t *qi, const int32_t *qj,
                  const int32_t *ql, double *res, double *resmag)
{
    for (int64_t q = 0; q < nq; ++q) {
        int pr;
        int64_t key = ((int64_t)qi[q] * X->dims[1] + qj[q]) * X->dims[2] + ql[q];
        double x = dok_get(X, key, &pr);
        if (!pr) { res[q] = 0.0; resmag[q] = 0.0; continue; }
        res[q] = cp_resid(F1, F2, F3, R, qi[q], qj[q], ql[q], x, &resmag[q]);
    }
}

/*
 * Factor gradients, the negated MTTKRPs of the residual (reverse gradients
 * of the CP loss, Sections 4.2-4.3):
 *   mode 0: dF1(i,:) = -sum over stored (i, j, l) of R_ijl * (F2(j,:) o F3(l,:))
 *   mode 1: dF2(j,:) = -sum ... R_ijl * (F1(i,:) o F3(l,:))
 *   mode 2: dF3(l,:) = -sum ... R_ijl * (F1(i,:) o F2(j,:))
 */
void orc_cp_grad(const orc_dok *X, const double *F1, const double *F2, const double *F3,
                 int64_t R, int mode, int64_t nsel, const int32_t *sel, double *out,
                 double *outmag)
{
    int64_t n = X->dims[mode];
    int64_t *map = select_map(n, nsel, sel);
    int64_t rows = sel ? nsel : n;
    memset(out, 0, sizeof(double) * rows * R);
    memset(outmag, 0, sizeof(double) * rows * R);
#pragma omp parallel
    {
    const int nt = orc_nthr(), me = orc_tid();
    for (int64_t s = 0; s < X->cap; ++s) {
        if (X->key[s] == -1) continue;
        int64_t c[3];
        unpack3(X, X->key[s], &c[0], &c[1], &c[2]);
        int64_t o = map[c[mode]];
        if (o < 0 || o % nt != me) continue;
        double rm, r = cp_resid(F1, F2, F3, R, c[0], c[1], c[2], X->val[s], &rm);
        const double *Fs[3] = {F1, F2, F3};
        const double *P = Fs[(mode + 1) % 3] + c[(mode + 1) % 3] * R;
        const double *Q = Fs[(mode + 2) % 3] + c[(mode + 2) % 3] * R;
        for (int64_t t = 0; t < R; ++t) {
            out[o * R + t] += -r * P[t] * Q[t];
            outmag[o * R + t] += rm * fabs(P[t] * Q[t]);
        }
    }
    }
    free(map);
}

/* ------------------------------------------ tensor-times-vector (mode 3) */

/*
 * Y(i, j) = sum over stored (i, j, l, x) of x * v(l): a sum over the stored
 * keys with a singleton {(i, j) -> x * v(l)} accumulated by "+=".  The result
 * is itself a DOK whose keys are the projection of X's keys onto (i, j).
 * Emitted in (i, j) order; returns the number of output keys.
 */
int64_t orc_ttv(const orc_dok *X, const double *v, int32_t *yi, int32_t *yj, double *y,
                double *ymag)
{
    int64_t dims[3] = {X->dims[0], X->dims[1], 1};
    orc_dok *Y = dok_new(2, dims, X->n);
    orc_dok *Ym = dok_new(2, dims, X->n);
    for (int64_t s = 0; s < X->cap; ++s) {
        if (X->key[s] == -1) continue;
        int64_t i, j, l;
        unpack3(X, X->key[s], &i, &j, &l);
        dok_add(Y, i * dims[1] + j, X->val[s] * v[l], 0);
        dok_add(Ym, i * dims[1] + j, fabs(X->val[s] * v[l]), 0);
    }
    int64_t n = Y->n, m = 0;
    kt_pair *kp = (kt_pair *)malloc(sizeof(kt_pair) * (n ? n : 1));
    for (int64_t s = 0; s < Y->cap; ++s)
        if (Y->key[s] != -1) { kp[m].key = Y->key[s]; kp[m].tag = s; ++m; }
    qsort(kp, (size_t)n, sizeof(kt_pair), cmp_kt);
    for (int64_t q = 0; q < n; ++q) {
        int64_t i, j;
        unpack2(Y, kp[q].key, &i, &j);
        yi[q] = (int32_t)i; yj[q] = (int32_t)j;
        y[q] = Y->val[kp[q].tag];
        ymag[q] = dok_get(Ym, kp[q].key, NULL);
    }
    free(kp);
    orc_dok_free(Y); orc_dok_free(Ym);
    return n;
}

/*
 * Vector-Jacobian product (Sections 4.2-4.3) of Y = X x_3 v given the
 * upstream gY (a DOK on Y's
 * keys, read by lookup so absent keys count as 0):
 *   dX at queried (i, j, l) that are stored: gY(i, j) * v(l)
 *   dv(l) = sum over stored (i, j, l, x) of x * gY(i, j)
 */
void orc_ttv_vjp(const orc_dok *X, const double *v, const orc_dok *gY, int64_t nq,
                 const int32_t *qi, const int32_t *qj, const int32_t *ql, double *dX,
                 double *dXmag, double *dv, double *dvmag)
{
    int64_t ncj = X->dims[1];
    for (int64_t q = 0; q < nq; ++q) {
        int pr;
        int64_t key = ((int64_t)qi[q] * X->dims[1] + qj[q]) * X->dims[2] + ql[q];
        dok_get(X, key, &pr);
        double g = pr ? dok_get(gY, (int64_t)qi[q] * ncj + qj[q], NULL) : 0.0;
        dX[q] = g * v[ql[q]];
        dXmag[q] = fabs(dX[q]);
    }
    memset(dv, 0, sizeof(double) * X->dims[2]);
    memset(dvmag, 0, sizeof(double) * X->dims[2]);
    for (int64_t s = 0; s < X->cap; ++s) {
        if (X->key[s] == -1) continue;
        int64_t i, j, l;
        unpack3(X, X->key[s], &i, &j, &l);
        double g = dok_get(gY, i * ncj + j, NULL);
        dv[l] += X->val[s] * g;
        dvmag[l] += fabs(X->val[s] * g);
    }
}

/*
 * Tensor-times-matrix along the third mode, the matrix form of TTV:
 *   Y(i, j, r) = sum over stored (i, j, l) of X_ijl * U(l, r)
 * on the projected keys {(i, j)}: a sum over X's keys inserting the row
 * {(i, j) -> X_ijl U(l, :)} with "+=" (Section 3, Section 5.5).  U is row-major
 * [dims[2] x R]; the keys come out sorted by (i, j), y row-major [ny x R]
 * with mag on |terms|.  Returns ny.
 */
static orc_dok *ttm_keys(const orc_dok *X, int32_t *yi, int32_t *yj, int64_t *ny)
{
    int64_t dims[3] = {X->dims[0], X->dims[1], 1};
    orc_dok *K = dok_new(2, dims, X->n);
    for (int64_t s = 0; s < X->cap; ++s) {
        if (X->key[s] == -1) continue;
        int64_t i, j, l;
        unpack3(X, X->key[s], &i, &j, &l);
        dok_add(K, i * dims[1] + j, 1.0, 0);
    }
    int64_t n = K->n, m = 0;
    kt_pair *kp = (kt_pair *)malloc(sizeof(kt_pair) * (n ? n : 1));
    for (int64_t s = 0; s < K->cap; ++s)
        if (K->key[s] != -1) { kp[m].key = K->key[s]; kp[m].tag = s; ++m; }
    qsort(kp, (size_t)n, sizeof(kt_pair), cmp_kt);
    for (int64_t q = 0; q < n; ++q) {  /* the value of key q becomes its row number */
        int64_t i, j;
        unpack2(K, kp[q].key, &i, &j);
        if (yi) { yi[q] = (int32_t)i; yj[q] = (int32_t)j; }
        K->val[kp[q].tag] = (double)q;
    }
    free(kp);
    *ny = n;
    return K;
}

int64_t orc_ttm(const orc_dok *X, const double *U, int32_t R, int32_t *yi, int32_t *yj, double *y,
                double *ymag)
{
    int64_t ny;
    orc_dok *K = ttm_keys(X, yi, yj, &ny);
    memset(y, 0, sizeof(double) * ny * R);
    memset(ymag, 0, sizeof(double) * ny * R);
    for (int64_t s = 0; s < X->cap; ++s) {
        if (X->key[s] == -1) continue;
        int64_t i, j, l;
        unpack3(X, X->key[s], &i, &j, &l);
        int64_t q = (int64_t)dok_get(K, i * X->dims[1] + j, NULL);
        for (int32_t r = 0; r < R; ++r) {
            double t = X->val[s] * U[l * R + r];
            y[q * R + r] += t;
            ymag[q * R + r] += fabs(t);
        }
    }
    orc_dok_free(K);
    return ny;
}

/*
 * Vector-Jacobian product (Sections 4.2-4.3) of Y = X x_3 U given the
 * upstream gY row-major
 * [ny x R] on Y's keys in (i, j) order:
 *   dX at queried (i, j, l) that are stored: sum_r gY(i, j, r) U(l, r)
 *   dU(l, r) = sum over stored (i, j, l, x) of x * gY(i, j, r)
 */
void orc_ttm_vjp(const orc_dok *X, const double *U, int32_t R, const double *gY, int64_t nq,
                 const int32_t *qi, const int32_t *qj, const int32_t *ql, double *dX,
                 double *dXmag, double *dU, double *dUmag)
{
    int64_t ny;
    orc_dok *K = ttm_keys(X, NULL, NULL, &ny);
    for (int64_t q = 0; q < nq; ++q) {
        int pr;
        int64_t key = ((int64_t)qi[q] * X->dims[1] + qj[q]) * X->dims[2] + ql[q];
        dok_get(X, key, &pr);
        double d = 0.0, m = 0.0;
        if (pr) {
            int64_t row = (int64_t)dok_get(K, (int64_t)qi[q] * X->dims[1] + qj[q], NULL);
            for (int32_t r = 0; r < R; ++r) {
                double t = gY[row * R + r] * U[(int64_t)ql[q] * R + r];
                d += t;
                m += fabs(t);
            }
        }
        dX[q] = d;
        dXmag[q] = m;
    }
    memset(dU, 0, sizeof(double) * X->dims[2] * R);
    memset(dUmag, 0, sizeof(double) * X->dims[2] * R);
    for (int64_t s = 0; s < X->cap; ++s) {
        if (X->key[s] == -1) continue;
        int64_t i, j, l;
        unpack3(X, X->key[s], &i, &j, &l);
        int64_t row = (int64_t)dok_get(K, i * X->dims[1] + j, NULL);
        for (int32_t r = 0; r < R; ++r) {
            double t = X->val[s] * gY[row * R + r];
            dU[l * R + r] += t;
            dUmag[l * R + r] += fabs(t);
        }
    }
    orc_dok_free(K);
}

/* ------------------------------- tensor-times-matrix along any mode */

/*
 * Mode-n product of an order-N sparse tensor (3 <= N <= 6) with a matrix,
 * kept sparse on the projected keys (the n-mode product of Section 3's
 * tensor algebra; TTV is its R = 1 case):
 *   Y(c_{-n}, r) = sum over stored keys c with those other coordinates of
 *                  X(c) * U(c_n, r)
 * where c_{-n} is the key with coordinate n dropped.  The result is a DOK of
 * order N - 1 whose keys are the projections of X's keys, built by a sum over
 * X's keys inserting the row {c_{-n} -> X(c) U(c_n, :)} with "+=" (Section 3,
 * Section 5.5).  Keys come out in lexicographic order (mode 0 first) as
 * N - 1 coordinate arrays ykey[o] (the modes other than n in increasing
 * order), y row-major [ny x R] with its mag.  Returns ny.
 */
static void proj_dims(const orc_dok *X, int mode, int64_t *pd)
{
    int o = 0;
    for (int m = 0; m < X->order; ++m)
        if (m != mode) pd[o++] = X->dims[m];
}

static int64_t proj_pack(const orc_dok *X, int mode, const int64_t *c)
{
    int64_t key = 0;
    for (int m = 0; m < X->order; ++m)
        if (m != mode) key = key * X->dims[m] + c[m];
    return key;
}

/* the projected keys of X, each DOK value set to the key's row number in
 * lexicographic order; their coordinates written to ykey (when given) */
static orc_dok *proj_keys(const orc_dok *X, int mode, int32_t *const *ykey, int64_t *ny)
{
    int64_t pd[ORC_MAX_ORDER], c[ORC_MAX_ORDER];
    proj_dims(X, mode, pd);
    orc_dok *K = dok_new(X->order - 1, pd, X->n);
    for (int64_t s = 0; s < X->cap; ++s) {
        if (X->key[s] == -1) continue;
        unpackn(X, X->key[s], c);
        dok_add(K, proj_pack(X, mode, c), 1.0, 0);
    }
    int64_t n = K->n, m = 0;
    kt_pair *kp = (kt_pair *)malloc(sizeof(kt_pair) * (n ? n : 1));
    for (int64_t s = 0; s < K->cap; ++s)
        if (K->key[s] != -1) { kp[m].key = K->key[s]; kp[m].tag = s; ++m; }
    qsort(kp, (size_t)n, sizeof(kt_pair), cmp_kt);
    for (int64_t q = 0; q < n; ++q) {
        if (ykey) {
            int64_t pc[ORC_MAX_ORDER];
            unpackn(K, kp[q].key, pc);
            for (int o = 0; o < K->order; ++o) ykey[o][q] = (int32_t)pc[o];
        }
        K->val[kp[q].tag] = (double)q;
    }
    free(kp);
    *ny = n;
    return K;
}

int64_t orc_ttmn(const orc_dok *X, int32_t mode, const double *U, int32_t R,
                 int32_t *const *ykey, double *y, double *ymag)
{
    int64_t ny, c[ORC_MAX_ORDER];
    orc_dok *K = proj_keys(X, mode, ykey, &ny);
    memset(y, 0, sizeof(double) * ny * R);
    memset(ymag, 0, sizeof(double) * ny * R);
    for (int64_t s = 0; s < X->cap; ++s) {
        if (X->key[s] == -1) continue;
        unpackn(X, X->key[s], c);
        int64_t q = (int64_t)dok_get(K, proj_pack(X, mode, c), NULL);
        for (int32_t r = 0; r < R; ++r) {
            double t = X->val[s] * U[c[mode] * R + r];
            y[q * R + r] += t;
            ymag[q * R + r] += fabs(t);
        }
    }
    orc_dok_free(K);
    return ny;
}

/*
 * Vector-Jacobian product (Sections 4.2-4.3) of the mode-n product for the
 * upstream gY row-major [ny x R] on Y's keys in lexicographic order:
 *   dX at the queried keys that are stored: sum_r gY(c_{-n}, r) U(c_n, r)
 *   dU(l, r) = sum over stored keys c with c_n = l of X(c) gY(c_{-n}, r)
 * q[m][p] is coordinate m of query p.
 */
void orc_ttmn_vjp(const orc_dok *X, int32_t mode, const double *U, int32_t R, const double *gY,
                  int64_t nq, const int32_t *const *q, double *dX, double *dXmag, double *dU,
                  double *dUmag)
{
    int64_t ny, c[ORC_MAX_ORDER];
    orc_dok *K = proj_keys(X, mode, NULL, &ny);
    for (int64_t p = 0; p < nq; ++p) {
        int64_t key = 0;
        for (int m = 0; m < X->order; ++m) {
            c[m] = q[m][p];
            key = key * X->dims[m] + c[m];
        }
        int pr;
        dok_get(X, key, &pr);
        double d = 0.0, mg = 0.0;
        if (pr) {
            int64_t row = (int64_t)dok_get(K, proj_pack(X, mode, c), NULL);
            for (int32_t r = 0; r < R; ++r) {
                double t = gY[row * R + r] * U[c[mode] * R + r];
                d += t;
                mg += fabs(t);
            }
        }
        dX[p] = d;
        dXmag[p] = mg;
    }
    int64_t nl = X->dims[mode];
    memset(dU, 0, sizeof(double) * nl * R);
    memset(dUmag, 0, sizeof(double) * nl * R);
    for (int64_t s = 0; s < X->cap; ++s) {
        if (X->key[s] == -1) continue;
        unpackn(X, X->key[s], c);
        int64_t row = (int64_t)dok_get(K, proj_pack(X, mode, c), NULL);
        for (int32_t r = 0; r < R; ++r) {
            double t = X->val[s] * gY[row * R + r];
            dU[c[mode] * R + r] += t;
            dUmag[c[mode] * R + r] += fabs(t);
        }
    }
    orc_dok_free(K);
}

/* ---------------------------------------------------- BATAX Jacobian */

/*
 * Jacobian of the BATAX kernel f(j) = sum_{i,k} beta A(i,j) A(i,k) x(k) with
 * respect to x (Example 5; the matrix-kernel benchmarks of Section 7):
 *   J(j, k) = beta sum_i A(i, j) A(i, k)
 * taken the way the differentiated, normalised program of Example 5 runs:
 * for every stored row r of A, the outer product r x r is inserted into the
 * result with the semi-ring += (Section 5.4, destination-passing code of
 * Section 5.5).  A key of J exists for every pair of stored keys of A that
 * share a row, also when the product is 0 (stored zeros keep their keys).
 * Emitted as an n x n CSR (n = columns of A) in (row, col) order, with mag =
 * the sum of |terms| of every value.  cap must hold the number of keys
 * (sum over rows of length^2 suffices).  Returns the number of keys.
 */
int64_t orc_batax_jacobian(const orc_dok *A, double beta, int64_t cap, int32_t *rowptr,
                           int32_t *colind, double *val, double *mag)
{
    int64_t m = A->dims[0], n = A->dims[1], nnz = A->n;
    int32_t *arp = (int32_t *)malloc(sizeof(int32_t) * (m + 1));
    int32_t *aci = (int32_t *)malloc(sizeof(int32_t) * (nnz ? nnz : 1));
    double *av = (double *)malloc(sizeof(double) * (nnz ? nnz : 1));
    int64_t *afirst = (int64_t *)malloc(sizeof(int64_t) * (nnz ? nnz : 1));
    orc_coo_to_csr(A, arp, aci, av, afirst);
    int64_t pairs = 0;
    for (int64_t i = 0; i < m; ++i) {
        int64_t len = arp[i + 1] - arp[i];
        pairs += len * len;
    }
    int64_t dims[3] = {n, n, 1};
    orc_dok *J = dok_new(2, dims, pairs);
    orc_dok *Jm = dok_new(2, dims, pairs);
    int64_t tag = 0;
    for (int64_t i = 0; i < m; ++i)               /* every stored row r ...     */
        for (int32_t p = arp[i]; p < arp[i + 1]; ++p)      /* ... r x r into J */
            for (int32_t q = arp[i]; q < arp[i + 1]; ++q) {
                int64_t key = (int64_t)aci[p] * n + aci[q];
                double t = beta * av[p] * av[q];
                dok_add(J, key, t, tag);
                dok_add(Jm, key, fabs(t), tag);
                ++tag;
            }
    int64_t nk = J->n;
    if (nk <= cap) {
        int64_t *first = (int64_t *)malloc(sizeof(int64_t) * (nk ? nk : 1));
        orc_coo_to_csr(J, rowptr, colind, val, first);
        for (int64_t r = 0; r < n; ++r)
            for (int32_t p = rowptr[r]; p < rowptr[r + 1]; ++p)
                mag[p] = dok_get(Jm, r * n + colind[p], NULL);
        free(first);
    }
    orc_dok_free(J);
    orc_dok_free(Jm);
    free(arp); free(aci); free(av); free(afirst);
    return nk;
}

/* ------------------------------------------------- forward-mode tangent */

/*
 * Forward-mode tangent of the matrix product C = A B (the forward-mode rules
 * of Section 4.1 applied to the product's sum over A's stored keys, Section
 * 3), for a tangent dA that lives on A's keys and a dense tangent dB:
 *   C(i,:)  = sum over stored (i,j) of A(i,j) B(j,:)
 *   dC(i,:) = sum over stored (i,j) of dA(i,j) B(j,:) + A(i,j) dB(j,:)
 * dA is read from its own dictionary by key (an absent key is 0).  B, dB are
 * row-major [ncols x k]; C, dC and their mags [nrows x k].
 */
void orc_spmm_jvp(const orc_dok *A, const orc_dok *dA, const double *B, const double *dB,
                  int64_t k, double *C, double *Cmag, double *dC, double *dCmag)
{
    int64_t nr = A->dims[0];
    memset(C, 0, sizeof(double) * nr * k);
    memset(Cmag, 0, sizeof(double) * nr * k);
    memset(dC, 0, sizeof(double) * nr * k);
    memset(dCmag, 0, sizeof(double) * nr * k);
    for (int64_t s = 0; s < A->cap; ++s) {
        if (A->key[s] == -1) continue;
        int64_t i, j;
        unpack2(A, A->key[s], &i, &j);
        double a = A->val[s];
        double da = dok_get(dA, A->key[s], NULL);
        for (int64_t c = 0; c < k; ++c) {
            double b = B[j * k + c], db = dB[j * k + c];
            C[i * k + c] += a * b;
            Cmag[i * k + c] += fabs(a * b);
            dC[i * k + c] += da * b + a * db;
            dCmag[i * k + c] += fabs(da * b) + fabs(a * db);
        }
    }
}


/* ------------------------------------------------ order-N CP gradient */

/* coordinates of a packed key of an order-N DOK (mixed radix, mode 0 most
 * significant) */
static void unpackn(const orc_dok *d, int64_t k, int64_t *c)
{
    for (int n = d->order - 1; n >= 0; --n) {
        c[n] = k % d->dims[n];
        k /= d->dims[n];
    }
}

orc_dok *orc_dok_buildn(int32_t order, const int64_t *dims, int64_t nnz,
                        const int32_t *const *coords, const float *val)
{
    orc_dok *d = dok_new(order, dims, nnz);
    for (int64_t p = 0; p < nnz; ++p) {
        int64_t key = 0;
        for (int n = 0; n < order; ++n) key = key * dims[n] + coords[n][p];
        dok_add(d, key, val ? (double)val[p] : 1.0, p);
    }
    return d;
}

/* m = sum_r prod_n F_n(c_n, r) at one key, R = x - m; *rmag = |x| + sum |terms| */
static double cpn_resid(const orc_dok *X, const double *const *F, int64_t R, const int64_t *c,
                        double x, double *rmag)
{
    double m = 0.0, mm = 0.0;
    for (int64_t r = 0; r < R; ++r) {
        double t = 1.0;
        for (int n = 0; n < X->order; ++n) t *= F[n][c[n] * R + r];
        m += t;
        mm += fabs(t);
    }
    *rmag = fabs(x) + mm;
    return x - m;
}

/*
 * Rank-R CP model of an order-N sparse tensor X (the order-3 case of
 * Section 3's nested dictionaries, with N nested levels):
 *   L = 1/2 sum over stored keys of (x - m)^2,  m = sum_r prod_n F_n(c_n, r)
 */
void orc_cpn_loss(const orc_dok *X, const double *const *F, int64_t R, double *loss,
                  double *mag)
{
    double L = 0.0, M = 0.0;
    int64_t c[ORC_MAX_ORDER];
    for (int64_t s = 0; s < X->cap; ++s) {
        if (X->key[s] == -1) continue;
        unpackn(X, X->key[s], c);
        double rm, r = cpn_resid(X, F, R, c, X->val[s], &rm);
        L += r * r;
        M += rm * rm;
    }
    *loss = 0.5 * L;
    *mag = 0.5 * M;
}

/* residual (the gradient w.r.t. the stored values, keyed by X's keys,
 * Section 4.3) at queried keys;
 * q[n][p] is coordinate n of query p */
void orc_cpn_resid(const orc_dok *X, const double *const *F, int64_t R, int64_t nq,
                   const int32_t *const *q, double *res, double *resmag)
{
    int64_t c[ORC_MAX_ORDER];
    for (int64_t p = 0; p < nq; ++p) {
        int64_t key = 0;
        for (int n = 0; n < X->order; ++n) {
            c[n] = q[n][p];
            key = key * X->dims[n] + c[n];
        }
        int pr;
        double x = dok_get(X, key, &pr);
        if (!pr) { res[p] = 0.0; resmag[p] = 0.0; continue; }
        res[p] = cpn_resid(X, F, R, c, x, &resmag[p]);
    }
}

/*
 * Factor gradient of mode n, the negated mode-n MTTKRP of the residual
 * (reverse gradient of the CP loss, Sections 4.2-4.3):
 *   dF_n(c_n, :) = -sum over stored keys of R * (o_{m != n} F_m(c_m, :))
 */
void orc_cpn_grad(const orc_dok *X, const double *const *F, int64_t R, int mode, int64_t nsel,
                  const int32_t *sel, double *out, double *outmag)
{
    int64_t rows_all = X->dims[mode];
    int64_t *map = select_map(rows_all, nsel, sel);
    int64_t rows = sel ? nsel : rows_all;
    memset(out, 0, sizeof(double) * rows * R);
    memset(outmag, 0, sizeof(double) * rows * R);
#pragma omp parallel
    {
    const int nt = orc_nthr(), me = orc_tid();
    int64_t c[ORC_MAX_ORDER];
    for (int64_t s = 0; s < X->cap; ++s) {
        if (X->key[s] == -1) continue;
        unpackn(X, X->key[s], c);
        int64_t o = map[c[mode]];
        if (o < 0 || o % nt != me) continue;
        double rm, r = cpn_resid(X, F, R, c, X->val[s], &rm);
        for (int64_t t = 0; t < R; ++t) {
            double h = 1.0;
            for (int n = 0; n < X->order; ++n)
                if (n != mode) h *= F[n][c[n] * R + t];
            out[o * R + t] += -r * h;
            outmag[o * R + t] += rm * fabs(h);
        }
    }
    }
    free(map);
}
