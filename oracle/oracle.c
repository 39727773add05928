/*
 * ORACLE -- test infrastructure only.  Plain, serial, obviously-correct CPU
 * code that the GPU library is checked against.  It shares no code with the
 * GPU path; only tests, the smoke check and the benchmark's CPU-baseline leg
 * may load it.
 *
 * What it computes
 * ----------------
 * 1. oracle_spgemm: the sparse product C = A * B of two CSR matrices, the
 *    GCN aggregation X = A_norm H of Sec. II-A (Eq. 1) with both operands
 *    held in compressed form.  Gustavson's row-wise formulation with a
 *    sparse accumulator (SPA):
 *      for each row i:   for each stored (k, a_ik) of A_i, k ascending:
 *                          for each stored (j, b_kj) of B_k:
 *                            if j not yet seen in row i: acc[j] = +0.0f
 *                            acc[j] = fl32(acc[j] + fl32(a_ik * b_kj))
 *                        emit the seen j in ascending order.
 *    The structure is structural, not numeric: an entry whose sum is 0.0
 *    is kept.  Build with -ffp-contract=off (no FMA) and without
 *    -ffast-math so every product and sum rounds to binary32.
 *    Optionally an fp64 shadow accumulates the same terms in double, plus
 *    the sum of |a_ik b_kj|, for the standard summation error bound.
 * 2. oracle_products: P_i = sum over stored k of A_i of nnz(B_k), the
 *    number of intermediate products of row i (2 P_i flops).
 * 3. oracle_robw: the row-block-wise (RoBW) partition of Algorithm 1
 *    (Sec. III-A): starting at the first unassigned row, keep adding whole
 *    rows while calcMem(k, q) <= M_A, where k is the number of rows in the
 *    block and q their stored entries; never split a row.  calcMem is not
 *    given in the paper; it is read here as the bytes of the block's own
 *    CSR arrays: (k + 1) row-pointer words plus q (column, value) pairs of
 *    4 + 4 bytes.  A first row that alone exceeds M_A is an error (the
 *    paper's loop would not advance).
 * 4. oracle_validate: canonical CSR check (row_ptr starts at 0, is
 *    non-decreasing, ends at nnz; columns strictly increasing in range).
 * 5. oracle_spmm: Y = act(A * W) for a CSR A and a dense row-major W, the
 *    combination step of a GCN layer (Sec. II-A, Eq. 3: aggregated features
 *    times the weights, then the activation sigma, ReLU here), written out
 *    from its definition: y_ij = act(sum over stored k of A_i of
 *    a_ik * w_kj), accumulated in double in ascending k, together with the
 *    sum of |a_ik * w_kj| for the standard summation error bound.
 * 6. oracle_sym_norm: the values of the normalised adjacency of Sec. II-A
 *    (Eq. 2) from a square pattern alone, D^-1/2 (A + I) D^-1/2 with the
 *    self-loops already in the pattern: a_ij = 1 / sqrt(r_i r_j), r_i the
 *    stored entries of row i, evaluated in double and rounded once to
 *    binary32.
 *
 * Row pointers are passed as int64 (the Python side widens int32 arrays).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
    int64_t r0, r1;     /* rows [r0, r1) of C */
    int64_t nnz;
    int64_t products;   /* sum of P_i over the rows */
    int64_t *rp;        /* r1 - r0 + 1, starting at 0 */
    int32_t *col;
    float *val;
    double *val64;      /* fp64 shadow sums (optional) */
    double *abs64;      /* sum of |a_ik b_kj| per entry (optional) */
    int64_t cap;
} oracle_result;

static int cmp_i32(const void *a, const void *b)
{
    int32_t x = *(const int32_t *)a, y = *(const int32_t *)b;
    return (x > y) - (x < y);
}

static int grow(oracle_result *r, int64_t need, int f64)
{
    if (need <= r->cap) return 0;
    int64_t cap = r->cap ? r->cap : 1024;
    while (cap < need) cap *= 2;
    int32_t *c = (int32_t *)realloc(r->col, sizeof(int32_t) * (size_t)cap);
    if (!c) return -1;
    r->col = c;
    float *v = (float *)realloc(r->val, sizeof(float) * (size_t)cap);
    if (!v) return -1;
    r->val = v;
    if (f64) {
        double *d = (double *)realloc(r->val64, sizeof(double) * (size_t)cap);
        if (!d) return -1;
        r->val64 = d;
        d = (double *)realloc(r->abs64, sizeof(double) * (size_t)cap);
        if (!d) return -1;
        r->abs64 = d;
    }
    r->cap = cap;
    return 0;
}

void oracle_result_free(oracle_result *r)
{
    if (!r) return;
    free(r->rp); free(r->col); free(r->val); free(r->val64); free(r->abs64); free(r);
}

/* Rows [r0, r1) of C = A * B.  Returns NULL on allocation failure. */
oracle_result *oracle_spgemm(int64_t N,
                             const int64_t *arp, const int32_t *acol, const float *aval,
                             const int64_t *brp, const int32_t *bcol, const float *bval,
                             int64_t r0, int64_t r1, int want_f64)
{
    oracle_result *r = (oracle_result *)calloc(1, sizeof(oracle_result));
    if (!r) return NULL;
    r->r0 = r0;
    r->r1 = r1;
    r->rp = (int64_t *)malloc(sizeof(int64_t) * (size_t)(r1 - r0 + 1));
    int64_t *mark = (int64_t *)malloc(sizeof(int64_t) * (size_t)(N > 0 ? N : 1));
    float *acc = (float *)malloc(sizeof(float) * (size_t)(N > 0 ? N : 1));
    double *acc64 = want_f64 ? (double *)malloc(sizeof(double) * (size_t)(N > 0 ? N : 1)) : NULL;
    double *abs64 = want_f64 ? (double *)malloc(sizeof(double) * (size_t)(N > 0 ? N : 1)) : NULL;
    int32_t *touched = (int32_t *)malloc(sizeof(int32_t) * (size_t)(N > 0 ? N : 1));
    if (!r->rp || !mark || !acc || !touched || (want_f64 && (!acc64 || !abs64))) goto fail;
    for (int64_t j = 0; j < N; ++j) mark[j] = -1;

    r->rp[0] = 0;
    int64_t nnz = 0, products = 0;
    for (int64_t i = r0; i < r1; ++i) {
        int64_t nt = 0;
        for (int64_t p = arp[i]; p < arp[i + 1]; ++p) {
            int64_t k = acol[p];
            float a = aval[p];
            for (int64_t q = brp[k]; q < brp[k + 1]; ++q) {
                int32_t j = bcol[q];
                float prod = a * bval[q];
                if (mark[j] != i) {
                    mark[j] = i;
                    acc[j] = 0.0f;
                    if (want_f64) { acc64[j] = 0.0; abs64[j] = 0.0; }
                    touched[nt++] = j;
                }
                acc[j] = acc[j] + prod;
                if (want_f64) {
                    double t = (double)a * (double)bval[q];
                    acc64[j] += t;
                    abs64[j] += t < 0 ? -t : t;
                }
                ++products;
            }
        }
        qsort(touched, (size_t)nt, sizeof(int32_t), cmp_i32);
        if (grow(r, nnz + nt, want_f64)) goto fail;
        for (int64_t t = 0; t < nt; ++t) {
            int32_t j = touched[t];
            r->col[nnz + t] = j;
            r->val[nnz + t] = acc[j];
            if (want_f64) { r->val64[nnz + t] = acc64[j]; r->abs64[nnz + t] = abs64[j]; }
        }
        nnz += nt;
        r->rp[i - r0 + 1] = nnz;
    }
    r->nnz = nnz;
    r->products = products;
    free(mark); free(acc); free(acc64); free(abs64); free(touched);
    return r;

fail:
    free(mark); free(acc); free(acc64); free(abs64); free(touched);
    oracle_result_free(r);
    return NULL;
}

int64_t oracle_result_nnz(const oracle_result *r) { return r->nnz; }
int64_t oracle_result_products(const oracle_result *r) { return r->products; }

void oracle_result_export(const oracle_result *r, int64_t *rp, int32_t *col, float *val,
                          double *val64, double *abs64)
{
    memcpy(rp, r->rp, sizeof(int64_t) * (size_t)(r->r1 - r->r0 + 1));
    if (r->nnz) {
        memcpy(col, r->col, sizeof(int32_t) * (size_t)r->nnz);
        memcpy(val, r->val, sizeof(float) * (size_t)r->nnz);
        if (val64 && r->val64) memcpy(val64, r->val64, sizeof(double) * (size_t)r->nnz);
        if (abs64 && r->abs64) memcpy(abs64, r->abs64, sizeof(double) * (size_t)r->nnz);
    }
}

/* Intermediate products per row: P_i = sum_{k in A_i} nnz(B_k). Returns the total. */
int64_t oracle_products(const int64_t *arp, const int32_t *acol, const int64_t *brp,
                        int64_t r0, int64_t r1, int64_t *P)
{
    int64_t total = 0;
    for (int64_t i = r0; i < r1; ++i) {
        int64_t s = 0;
        for (int64_t p = arp[i]; p < arp[i + 1]; ++p) s += brp[acol[p] + 1] - brp[acol[p]];
        if (P) P[i - r0] = s;
        total += s;
    }
    return total;
}

/*
 * Algorithm 1 (RoBW partitioning), boundaries as read above.  Writes the
 * first row of each block to starts[] (at most max_tiles entries) and
 * returns the number of blocks, -1 if a single row exceeds M_A, -2 if
 * max_tiles is too small.
 */
int64_t oracle_robw(int64_t m, const int64_t *rp, int64_t rp_bytes, int64_t M_A,
                    int64_t *starts, int64_t max_tiles)
{
    int64_t start = 0, n = 0;
    while (start < m) {
        int64_t end = start;
        for (;;) {
            if (end >= m) break;
            int64_t k = end + 1 - start;              /* rows if row `end` joins */
            int64_t q = rp[end + 1] - rp[start];      /* their stored entries */
            int64_t mem = (k + 1) * rp_bytes + q * 8; /* calcMem(k, q) */
            if (mem > M_A) break;
            ++end;
        }
        if (end == start) return -1;
        if (n >= max_tiles) return -2;
        starts[n++] = start;
        start = end;
    }
    return n;
}

/*
 * Canonical CSR check.  Returns 0 if valid, otherwise a positive code:
 * 1 row_ptr[0] != 0, 2 row_ptr decreasing, 3 row_ptr[m] != nnz,
 * 4 column out of range, 5 columns not strictly increasing in a row.
 */
int oracle_validate(int64_t m, int64_t ncols, int64_t nnz, const int64_t *rp, const int32_t *col)
{
    if (rp[0] != 0) return 1;
    for (int64_t i = 0; i < m; ++i)
        if (rp[i + 1] < rp[i]) return 2;
    if (rp[m] != nnz) return 3;
    for (int64_t i = 0; i < m; ++i)
        for (int64_t p = rp[i]; p < rp[i + 1]; ++p) {
            if (col[p] < 0 || col[p] >= ncols) return 4;
            if (p > rp[i] && col[p] <= col[p - 1]) return 5;
        }
    return 0;
}

/* Y (m x F, double, row-major) = act(A * W) with act = ReLU when relu;
   Yabs = sum over k of |a_ik * w_kj| (before the activation). */
void oracle_spmm(int64_t m, const int64_t *arp, const int32_t *acol, const float *aval, const float *W,
                 int64_t ldw, int64_t F, int relu, double *Y, double *Yabs)
{
    for (int64_t i = 0; i < m; ++i) {
        double *y = Y + i * F, *ya = Yabs + i * F;
        for (int64_t j = 0; j < F; ++j) { y[j] = 0.0; ya[j] = 0.0; }
        for (int64_t p = arp[i]; p < arp[i + 1]; ++p) {
            const double a = (double)aval[p];
            const float *w = W + (int64_t)acol[p] * ldw;
            for (int64_t j = 0; j < F; ++j) {
                const double t = a * (double)w[j];
                y[j] += t;
                ya[j] += t < 0 ? -t : t;
            }
        }
        if (relu)
            for (int64_t j = 0; j < F; ++j) if (y[j] < 0.0) y[j] = 0.0;
    }
}

/* out[p] = 1 / sqrt(r_i r_j) for the stored entry p = (i, j) of the pattern */
void oracle_sym_norm(int64_t m, const int64_t *rp, const int32_t *col, float *out)
{
    for (int64_t i = 0; i < m; ++i) {
        const double ri = (double)(rp[i + 1] - rp[i]);
        for (int64_t p = rp[i]; p < rp[i + 1]; ++p) {
            const int64_t j = col[p];
            const double rj = (double)(rp[j + 1] - rp[j]);
            out[p] = (float)(1.0 / sqrt(ri * rj));
        }
    }
}
