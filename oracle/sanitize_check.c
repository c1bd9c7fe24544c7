/*
 * sanitize_check.c -- drives every exported routine of the fp64 oracle once
 * on small random inputs (duplicates, empty rows and columns, stored zeros,
 * a selection, every mode of an order-4 tensor), for a build of the oracle
 * with the address and undefined-behaviour sanitizers.  TEST INFRASTRUCTURE
 * ONLY: built and run by the oracle's CPU tests; it checks memory safety of
 * the oracle, not its values (those are pinned elsewhere).  Exits 0 when
 * every call returned; a sanitizer report aborts with a non-zero status.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

typedef struct orc_dok orc_dok;

void orc_set_threads(int n);
orc_dok *orc_dok_build2(int64_t nr, int64_t nc, int64_t nnz, const int32_t *row,
                        const int32_t *col, const float *val);
orc_dok *orc_dok_build3(int64_t d0, int64_t d1, int64_t d2, int64_t nnz, const int32_t *i,
                        const int32_t *j, const int32_t *l, const float *val);
orc_dok *orc_dok_buildn(int32_t order, const int64_t *dims, int64_t nnz,
                        const int32_t *const *coords, const float *val);
void orc_dok_free(orc_dok *d);
int64_t orc_dok_nkeys(const orc_dok *d);
void orc_dok_lookup2(const orc_dok *d, int64_t nq, const int32_t *qi, const int32_t *qj,
                     double *out, int8_t *present);
int64_t orc_coo_to_csr(const orc_dok *d, int32_t *rowptr, int32_t *colind, double *val,
                       int64_t *first);
void orc_stable_sort_by_key(int64_t n, const int32_t *key, int64_t nkeys, int32_t *segptr,
                            int32_t *skey, int32_t *perm);
void orc_spmm(const orc_dok *A, const double *B, const double *Bmag, int64_t k, int64_t nsel,
              const int32_t *sel, double *out, double *outmag);
void orc_spmm_t(const orc_dok *A, const double *G, const double *Gmag, int64_t k, double alpha,
                int64_t nsel, const int32_t *sel, double *out, double *outmag);
void orc_sddmm(const orc_dok *A, const double *X, const double *Xmag, const double *Y,
               const double *Ymag, int64_t k, double alpha, int64_t nq, const int32_t *qi,
               const int32_t *qj, double *out, double *outmag);
void orc_loss_sum_spmv(const orc_dok *A, const double *x, double *loss, double *mag);
void orc_loss_half_sq(int64_t n, const double *C, const double *Cmag, double *loss, double *mag);
void orc_loss_bilinear(const orc_dok *A, const double *G, const double *H, int64_t k,
                       double *loss, double *mag);
void orc_mf_loss(const orc_dok *A, const double *U, const double *V, int64_t k, double *loss,
                 double *mag);
void orc_mf_resid(const orc_dok *A, const double *U, const double *V, int64_t k, int64_t nq,
                  const int32_t *qi, const int32_t *qj, double *r, double *rmag);
void orc_mf_grad(const orc_dok *A, const double *U, const double *V, int64_t k, int mode,
                 int64_t nsel, const int32_t *sel, double *out, double *outmag);
void orc_cp_loss(const orc_dok *X, const double *F1, const double *F2, const double *F3,
                 int64_t R, double *loss, double *mag);
void orc_cp_resid(const orc_dok *X, const double *F1, const double *F2, const double *F3,
                  int64_t R, int64_t nq, const int32_t *qi, const int32_t *qj,
                  const int32_t *ql, double *res, double *resmag);
void orc_cp_grad(const orc_dok *X, const double *F1, const double *F2, const double *F3,
                 int64_t R, int mode, int64_t nsel, const int32_t *sel, double *out,
                 double *outmag);
int64_t orc_ttv(const orc_dok *X, const double *v, int32_t *yi, int32_t *yj, double *y,
                double *ymag);
void orc_ttv_vjp(const orc_dok *X, const double *v, const orc_dok *gY, int64_t nq,
                 const int32_t *qi, const int32_t *qj, const int32_t *ql, double *dX,
                 double *dXmag, double *dv, double *dvmag);
int64_t orc_ttm(const orc_dok *X, const double *U, int32_t R, int32_t *yi, int32_t *yj,
                double *y, double *ymag);
void orc_ttm_vjp(const orc_dok *X, const double *U, int32_t R, const double *gY, int64_t nq,
                 const int32_t *qi, const int32_t *qj, const int32_t *ql, double *dX,
                 double *dXmag, double *dU, double *dUmag);
int64_t orc_ttmn(const orc_dok *X, int32_t mode, const double *U, int32_t R,
                 int32_t *const *ykey, double *y, double *ymag);
void orc_ttmn_vjp(const orc_dok *X, int32_t mode, const double *U, int32_t R, const double *gY,
                  int64_t nq, const int32_t *const *q, double *dX, double *dXmag, double *dU,
                  double *dUmag);
int64_t orc_batax_jacobian(const orc_dok *A, double beta, int64_t cap, int32_t *rowptr,
                           int32_t *colind, double *val, double *mag);
void orc_spmm_jvp(const orc_dok *A, const orc_dok *dA, const double *B, const double *dB,
                  int64_t k, double *C, double *Cmag, double *dC, double *dCmag);
void orc_cpn_loss(const orc_dok *X, const double *const *F, int64_t R, double *loss,
                  double *mag);
void orc_cpn_resid(const orc_dok *X, const double *const *F, int64_t R, int64_t nq,
                   const int32_t *const *q, double *res, double *resmag);
void orc_cpn_grad(const orc_dok *X, const double *const *F, int64_t R, int mode, int64_t nsel,
                  const int32_t *sel, double *out, double *outmag);

static uint64_t rng_state = 0x2303070300000001ULL;

static uint32_t next_u32(void)
{   /* xorshift64*, enough for test inputs */
    rng_state ^= rng_state >> 12;
    rng_state ^= rng_state << 25;
    rng_state ^= rng_state >> 27;
    return (uint32_t)((rng_state * 0x2545F4914F6CDD1DULL) >> 32);
}

static double next_val(void) { return (double)next_u32() / 4294967296.0 * 2.0 - 1.0; }

static void *xmalloc(size_t n) { void *p = malloc(n ? n : 1); if (!p) exit(3); return p; }
static double *dvec(int64_t n)
{
    double *p = (double *)xmalloc(sizeof(double) * (size_t)n);
    for (int64_t i = 0; i < n; ++i) p[i] = next_val();
    return p;
}
static double *dzero(int64_t n) { return (double *)calloc(n ? (size_t)n : 1, sizeof(double)); }
static int32_t *ivec(int64_t n, int32_t mod)
{
    int32_t *p = (int32_t *)xmalloc(sizeof(int32_t) * (size_t)n);
    for (int64_t i = 0; i < n; ++i) p[i] = (int32_t)(next_u32() % (uint32_t)mod);
    return p;
}

static void matrices(void)
{
    const int64_t nr = 37, nc = 29, nnz = 300, k = 5;
    int32_t *row = ivec(nnz, nr - 3), *col = ivec(nnz, nc - 2);  /* empty tail rows/cols */
    float *val = (float *)xmalloc(sizeof(float) * nnz);
    for (int64_t p = 0; p < nnz; ++p) val[p] = p % 17 == 0 ? 0.0f : (float)next_val();
    orc_dok *A = orc_dok_build2(nr, nc, nnz, row, col, val);  /* duplicates summed */
    int64_t n = orc_dok_nkeys(A);
    int32_t *rowptr = (int32_t *)xmalloc(sizeof(int32_t) * (nr + 1));
    int32_t *colind = (int32_t *)xmalloc(sizeof(int32_t) * n);
    double *v = dzero(n);
    int64_t *first = (int64_t *)xmalloc(sizeof(int64_t) * n);
    orc_coo_to_csr(A, rowptr, colind, v, first);
    int32_t *segptr = (int32_t *)xmalloc(sizeof(int32_t) * (nc + 1));
    int32_t *skey = (int32_t *)xmalloc(sizeof(int32_t) * n), *perm = (int32_t *)xmalloc(sizeof(int32_t) * n);
    orc_stable_sort_by_key(n, colind, nc, segptr, skey, perm);
    int32_t *rows = (int32_t *)xmalloc(sizeof(int32_t) * n);
    for (int64_t r = 0; r < nr; ++r)
        for (int32_t p = rowptr[r]; p < rowptr[r + 1]; ++p) rows[p] = (int32_t)r;
    double *out = dzero(n), *outm = dzero(n);
    int8_t *pres = (int8_t *)xmalloc(n);
    orc_dok_lookup2(A, n, rows, colind, out, pres);
    double *B = dvec(nc * k), *G = dvec(nr * k), *C = dzero(nr * k), *Cm = dzero(nr * k);
    double *T = dzero(nc * k), *Tm = dzero(nc * k);
    int32_t sel[3] = {0, 5, (int32_t)nr - 1};
    orc_spmm(A, B, NULL, k, 0, NULL, C, Cm);
    orc_spmm(A, NULL, NULL, k, 3, sel, C, Cm);
    orc_spmm_t(A, G, NULL, k, -0.5, 0, NULL, T, Tm);
    orc_spmm_t(A, NULL, NULL, 1, 1.0, 2, sel, T, Tm);
    orc_sddmm(A, G, NULL, B, NULL, k, 2.0, n, rows, colind, out, outm);
    orc_sddmm(A, NULL, NULL, B, NULL, k, 1.0, 3, sel, sel, out, outm);
    double L, M;
    orc_loss_sum_spmv(A, B, &L, &M);
    orc_loss_half_sq(nr * k, C, Cm, &L, &M);
    double *H = dvec(nc * k);
    orc_loss_bilinear(A, G, H, k, &L, &M);
    orc_mf_loss(A, G, H, k, &L, &M);
    orc_mf_resid(A, G, H, k, n, rows, colind, out, outm);
    orc_mf_grad(A, G, H, k, 0, 0, NULL, C, Cm);
    orc_mf_grad(A, G, H, k, 1, 2, sel, T, Tm);
    int64_t cap = 0;
    for (int64_t r = 0; r < nr; ++r) cap += (int64_t)(rowptr[r + 1] - rowptr[r]) * (rowptr[r + 1] - rowptr[r]);
    int32_t *jrp = (int32_t *)xmalloc(sizeof(int32_t) * (nc + 1));
    int32_t *jci = (int32_t *)xmalloc(sizeof(int32_t) * cap);
    double *jv = dzero(cap), *jm = dzero(cap);
    orc_batax_jacobian(A, 1.5, cap, jrp, jci, jv, jm);
    orc_dok *dA = orc_dok_build2(nr, nc, nnz, row, col, val);
    double *dB = dvec(nc * k), *dC = dzero(nr * k), *dCm = dzero(nr * k);
    orc_spmm_jvp(A, dA, B, dB, k, C, Cm, dC, dCm);
    orc_dok_free(dA);
    orc_dok_free(A);
    free(row); free(col); free(val); free(rowptr); free(colind); free(v); free(first);
    free(segptr); free(skey); free(perm); free(rows); free(out); free(outm); free(pres);
    free(B); free(G); free(C); free(Cm); free(T); free(Tm); free(H); free(jrp); free(jci);
    free(jv); free(jm); free(dB); free(dC); free(dCm);
}

static void tensors(void)
{
    const int64_t d0 = 9, d1 = 7, d2 = 8, nnz = 200, R = 4;
    int32_t *i = ivec(nnz, d0), *j = ivec(nnz, d1), *l = ivec(nnz, d2 - 1);
    float *x = (float *)xmalloc(sizeof(float) * nnz);
    for (int64_t p = 0; p < nnz; ++p) x[p] = (float)next_val();
    orc_dok *X = orc_dok_build3(d0, d1, d2, nnz, i, j, l, x);
    double *F1 = dvec(d0 * R), *F2 = dvec(d1 * R), *F3 = dvec(d2 * R);
    double L, M, *r = dzero(nnz), *rm = dzero(nnz);
    orc_cp_loss(X, F1, F2, F3, R, &L, &M);
    orc_cp_resid(X, F1, F2, F3, R, nnz, i, j, l, r, rm);
    double *g = dzero(d0 * R), *gm = dzero(d0 * R);
    int32_t sel[2] = {1, 3};
    for (int m = 0; m < 3; ++m) orc_cp_grad(X, F1, F2, F3, R, m, 2, sel, g, gm);
    int64_t cap = orc_dok_nkeys(X);
    int32_t *yi = (int32_t *)xmalloc(sizeof(int32_t) * cap), *yj = (int32_t *)xmalloc(sizeof(int32_t) * cap);
    double *y = dzero(cap * R), *ym = dzero(cap * R);
    int64_t ny = orc_ttv(X, F3, yi, yj, y, ym);
    orc_dok *gY = orc_dok_build2(d0, d1, ny, yi, yj, NULL);
    double *dv = dzero(d2), *dvm = dzero(d2), *dU = dzero(d2 * R), *dUm = dzero(d2 * R);
    orc_ttv_vjp(X, F3, gY, nnz, i, j, l, r, rm, dv, dvm);
    ny = orc_ttm(X, F3, (int32_t)R, yi, yj, y, ym);
    double *gYm = dvec(ny * R);
    orc_ttm_vjp(X, F3, (int32_t)R, gYm, nnz, i, j, l, r, rm, dU, dUm);
    orc_dok_free(gY);
    orc_dok_free(X);
    free(F1); free(F2); free(F3); free(r); free(rm); free(g); free(gm); free(yi); free(yj);
    free(y); free(ym); free(dv); free(dvm); free(dU); free(dUm); free(gYm);

    /* order 4: CP and the mode products in every mode */
    const int64_t dims[4] = {5, 4, 6, 3}, n4 = 150;
    int32_t *c[4];
    for (int m = 0; m < 4; ++m) c[m] = ivec(n4, (int32_t)dims[m]);
    float *x4 = (float *)xmalloc(sizeof(float) * n4);
    for (int64_t p = 0; p < n4; ++p) x4[p] = (float)next_val();
    orc_dok *X4 = orc_dok_buildn(4, dims, n4, (const int32_t *const *)c, x4);
    double *F[4];
    for (int m = 0; m < 4; ++m) F[m] = dvec(dims[m] * R);
    double *r4 = dzero(n4), *rm4 = dzero(n4), *g4 = dzero(6 * R), *gm4 = dzero(6 * R);
    orc_cpn_loss(X4, (const double *const *)F, R, &L, &M);
    orc_cpn_resid(X4, (const double *const *)F, R, n4, (const int32_t *const *)c, r4, rm4);
    for (int m = 0; m < 4; ++m)
        orc_cpn_grad(X4, (const double *const *)F, R, m, 0, NULL, g4, gm4);
    int64_t cap4 = orc_dok_nkeys(X4);
    int32_t *keys[3];
    for (int o = 0; o < 3; ++o) keys[o] = (int32_t *)xmalloc(sizeof(int32_t) * cap4);
    double *y4 = dzero(cap4 * R), *ym4 = dzero(cap4 * R);
    for (int m = 0; m < 4; ++m) {
        int64_t ny4 = orc_ttmn(X4, m, F[m], (int32_t)R, keys, y4, ym4);
        double *gy4 = dvec(ny4 * R), *du = dzero(dims[m] * R), *dum = dzero(dims[m] * R);
        orc_ttmn_vjp(X4, m, F[m], (int32_t)R, gy4, n4, (const int32_t *const *)c, r4, rm4, du,
                     dum);
        free(gy4); free(du); free(dum);
    }
    orc_dok_free(X4);
    for (int m = 0; m < 4; ++m) { free(c[m]); free(F[m]); }
    for (int o = 0; o < 3; ++o) free(keys[o]);
    free(x4); free(r4); free(rm4); free(g4); free(gm4); free(y4); free(ym4);
    free(i); free(j); free(l); free(x);
}

int main(void)
{
    for (int threads = 1; threads <= 3; threads += 2) {
        orc_set_threads(threads);
        matrices();
        tensors();
    }
    puts("oracle sanitize check: every routine ran");
    return 0;
}
