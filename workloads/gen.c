/*
 * Seeded synthetic inputs for the GCN aggregation product C = A_norm * X.
 *
 * This file builds INPUTS only.  It holds none of the sparse-product
 * arithmetic: both the oracle and the GPU library consume what it writes.
 *
 *  - rmat_*  : a symmetric R-MAT graph with self-loops, normalised as in
 *              the GCN aggregation operator (Sec. II-A, Eq. 2): the
 *              augmented adjacency A + I scaled on both sides by
 *              D^{-1/2}, so the stored value of (i, j) is 1/sqrt(d_i d_j)
 *              with d the row length of A + I.
 *  - feat_*  : a sparse feature matrix whose entries are present
 *              independently with probability rho ("uniform random
 *              positions") and valued U[-1, 1).
 *
 * Randomness: every draw is a pure function of (seed, stream, counter)
 * through the SplitMix64 output function (Steele, Lea, Flood, OOPSLA
 * 2014), so results do not depend on the number of threads.
 *
 * R-MAT sampling (Chakrabarti, Zhan, Faloutsos, SDM 2004): each sample
 * picks one of four quadrants per bit level, MSB first, with
 * probabilities (a, b, c, d).  A sample with an endpoint >= n is redrawn
 * (attempt counter), so exactly n*D/2 samples are accepted; samples with
 * u == v are then dropped.  A seeded Fisher-Yates permutation relabels
 * vertices so hubs do not cluster in low row ids.  The graph is then
 * symmetrised, sorted and de-duplicated, and (i, i) is added to every row.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <omp.h>
#include <stdio.h>

static inline uint64_t sm64_mix(uint64_t z)
{
    z += 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

/* Counter-based draw: stream and counter folded through two mixes. */
static inline uint64_t draw(uint64_t seed, uint64_t stream, uint64_t ctr)
{
    return sm64_mix(sm64_mix(seed * 0xD1342543DE82EF95ull + stream) ^ ctr);
}

/* Uniform double in [0, 1) from the top 53 bits. */
static inline double u01(uint64_t h) { return (double)(h >> 11) * (1.0 / 9007199254740992.0); }

enum { STREAM_EDGE = 1, STREAM_PERM = 2, STREAM_FEAT_POS = 3, STREAM_FEAT_VAL = 4 };

typedef struct {
    int64_t n;
    int64_t nnz;
    int64_t *rp;    /* n + 1 */
    int32_t *col;   /* nnz, sorted within each row, unique */
    float *val;     /* nnz */
    int64_t samples;        /* accepted R-MAT samples (n*D/2) */
    int64_t self_samples;   /* accepted samples with u == v (dropped) */
} rmat_graph;

static int cmp_i32(const void *a, const void *b)
{
    int32_t x = *(const int32_t *)a, y = *(const int32_t *)b;
    return (x > y) - (x < y);
}

/* One accepted R-MAT sample for index e: redraw until both ends < n. */
static void rmat_sample(uint64_t seed, int64_t e, int levels, int64_t n,
                        uint32_t ta, uint32_t tab, uint32_t tabc,
                        int64_t *pu, int64_t *pv)
{
    for (uint64_t attempt = 0;; ++attempt) {
        int64_t u = 0, v = 0;
        /* counter = sample index | attempt | 2-level block (levels <= 62) */
        uint64_t base = ((uint64_t)e << 20) | ((attempt & 0x7fffu) << 5);
        int lvl = 0;
        uint64_t blk = 0;
        while (lvl < levels) {
            uint64_t h = draw(seed, STREAM_EDGE, base | blk++);
            for (int half = 0; half < 2 && lvl < levels; ++half, ++lvl) {
                uint32_t r = (uint32_t)(half ? (h >> 32) : h);
                int bu, bv;
                if (r < ta)        { bu = 0; bv = 0; }
                else if (r < tab)  { bu = 0; bv = 1; }
                else if (r < tabc) { bu = 1; bv = 0; }
                else               { bu = 1; bv = 1; }
                u = (u << 1) | bu;
                v = (v << 1) | bv;
            }
        }
        if (u < n && v < n) { *pu = u; *pv = v; return; }
    }
}

/*
 * Build the normalised symmetric R-MAT graph.  Returns NULL on allocation
 * failure.  deg_target is D (accepted samples = n*D/2).
 */
rmat_graph *rmat_build(int64_t n, double deg_target, double a, double b, double c,
                       uint64_t seed, int verbose)
{
    const double t0 = omp_get_wtime();
#define GEN_STAGE(name) \
    do { if (verbose) { fprintf(stderr, "[gen] n=%lld %s %.1fs\n", (long long)n, name, omp_get_wtime() - t0); fflush(stderr); } } while (0)
    if (n <= 0) return NULL;
    int levels = 0;
    while (((int64_t)1 << levels) < n) ++levels;
    const int64_t E = (int64_t)((double)n * deg_target / 2.0);
    const double scale = 4294967296.0;
    uint32_t ta = (uint32_t)fmin(a * scale, 4294967295.0);
    uint32_t tab = (uint32_t)fmin((a + b) * scale, 4294967295.0);
    uint32_t tabc = (uint32_t)fmin((a + b + c) * scale, 4294967295.0);

    rmat_graph *g = (rmat_graph *)calloc(1, sizeof(rmat_graph));
    if (!g) return NULL;
    g->n = n;
    g->samples = E;

    /* Vertex permutation: Fisher-Yates with counter-based draws. */
    int32_t *perm = (int32_t *)malloc(sizeof(int32_t) * (size_t)n);
    int64_t *cnt = (int64_t *)calloc((size_t)n + 1, sizeof(int64_t));
    uint64_t *pairs = (uint64_t *)malloc(sizeof(uint64_t) * (size_t)(E > 0 ? E : 1));
    if (!perm || !cnt || !pairs) goto fail;
    for (int64_t i = 0; i < n; ++i) perm[i] = (int32_t)i;
    for (int64_t i = n - 1; i > 0; --i) {
        uint64_t h = draw(seed, STREAM_PERM, (uint64_t)i);
        int64_t j = (int64_t)(((unsigned __int128)h * (uint64_t)(i + 1)) >> 64);
        int32_t t = perm[i]; perm[i] = perm[j]; perm[j] = t;
    }
    GEN_STAGE("permutation");

    /* Samples, relabelled; self samples marked with all-ones. */
    int64_t selfs = 0;
#pragma omp parallel for schedule(static) reduction(+ : selfs)
    for (int64_t e = 0; e < E; ++e) {
        int64_t u, v;
        rmat_sample(seed, e, levels, n, ta, tab, tabc, &u, &v);
        if (u == v) { pairs[e] = ~0ull; ++selfs; continue; }
        uint64_t pu = (uint64_t)(uint32_t)perm[u], pv = (uint64_t)(uint32_t)perm[v];
        pairs[e] = (pu << 32) | pv;
#pragma omp atomic
        cnt[pu]++;
#pragma omp atomic
        cnt[pv]++;
    }
    g->self_samples = selfs;
    GEN_STAGE("samples");

    /* Bucket both directions by row (+1 slot per row for the self-loop). */
    int64_t *off = (int64_t *)malloc(sizeof(int64_t) * ((size_t)n + 1));
    if (!off) goto fail;
    off[0] = 0;
    for (int64_t i = 0; i < n; ++i) off[i + 1] = off[i] + cnt[i] + 1;
    int32_t *tmp = (int32_t *)malloc(sizeof(int32_t) * (size_t)off[n]);
    int64_t *cur = cnt; /* reuse as cursors */
    if (!tmp) { free(off); goto fail; }
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) { tmp[off[i]] = (int32_t)i; cur[i] = off[i] + 1; }
#pragma omp parallel for schedule(static)
    for (int64_t e = 0; e < E; ++e) {
        uint64_t p = pairs[e];
        if (p == ~0ull) continue;
        int64_t u = (int64_t)(p >> 32), v = (int64_t)(p & 0xffffffffu);
        int64_t pu, pv;
#pragma omp atomic capture
        pu = cur[u]++;
#pragma omp atomic capture
        pv = cur[v]++;
        tmp[pu] = (int32_t)v;
        tmp[pv] = (int32_t)u;
    }
    free(pairs); pairs = NULL;
    GEN_STAGE("bucketed");

    /* Sort + dedupe each row in place; record the unique length. */
    int64_t *len = cur;
#pragma omp parallel for schedule(dynamic, 1024)
    for (int64_t i = 0; i < n; ++i) {
        int32_t *r = tmp + off[i];
        int64_t L = off[i + 1] - off[i];
        qsort(r, (size_t)L, sizeof(int32_t), cmp_i32);
        int64_t w = 0;
        for (int64_t t = 0; t < L; ++t)
            if (w == 0 || r[t] != r[w - 1]) r[w++] = r[t];
        len[i] = w;
    }
    g->rp = (int64_t *)malloc(sizeof(int64_t) * ((size_t)n + 1));
    if (!g->rp) { free(off); free(tmp); goto fail; }
    g->rp[0] = 0;
    for (int64_t i = 0; i < n; ++i) g->rp[i + 1] = g->rp[i] + len[i];
    g->nnz = g->rp[n];
    GEN_STAGE("sorted and deduplicated");
    g->col = (int32_t *)malloc(sizeof(int32_t) * (size_t)(g->nnz > 0 ? g->nnz : 1));
    g->val = (float *)malloc(sizeof(float) * (size_t)(g->nnz > 0 ? g->nnz : 1));
    if (!g->col || !g->val) { free(off); free(tmp); goto fail; }
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i)
        memcpy(g->col + g->rp[i], tmp + off[i], sizeof(int32_t) * (size_t)len[i]);
    free(tmp);
    free(off);

    /* Symmetric normalisation: 1/sqrt(d_i d_j), d = row length incl. self-loop. */
#pragma omp parallel for schedule(dynamic, 4096)
    for (int64_t i = 0; i < n; ++i) {
        double di = (double)(g->rp[i + 1] - g->rp[i]);
        for (int64_t t = g->rp[i]; t < g->rp[i + 1]; ++t) {
            int64_t j = g->col[t];
            double dj = (double)(g->rp[j + 1] - g->rp[j]);
            g->val[t] = (float)(1.0 / sqrt(di * dj));
        }
    }
    free(perm);
    free(cnt);
    GEN_STAGE("normalised");
#undef GEN_STAGE
    return g;

fail:
    free(perm);
    free(cnt);
    free(pairs);
    if (g) { free(g->rp); free(g->col); free(g->val); free(g); }
    return NULL;
}

int64_t rmat_nnz(const rmat_graph *g) { return g->nnz; }
int64_t rmat_samples(const rmat_graph *g) { return g->samples; }
int64_t rmat_self_samples(const rmat_graph *g) { return g->self_samples; }

/* Copy the graph into caller buffers; rp is written as int32 when rp_is64 == 0. */
void rmat_export(const rmat_graph *g, void *rp, int rp_is64, int32_t *col, float *val)
{
    int64_t n = g->n;
    if (rp_is64) {
        memcpy(rp, g->rp, sizeof(int64_t) * ((size_t)n + 1));
    } else {
        int32_t *r = (int32_t *)rp;
#pragma omp parallel for schedule(static)
        for (int64_t i = 0; i <= n; ++i) r[i] = (int32_t)g->rp[i];
    }
    int64_t nnz = g->nnz;
    int nt = omp_get_max_threads();
#pragma omp parallel for schedule(static)
    for (int t = 0; t < nt; ++t) {
        int64_t lo = nnz * t / nt, hi = nnz * (t + 1) / nt;
        memcpy(col + lo, g->col + lo, sizeof(int32_t) * (size_t)(hi - lo));
        memcpy(val + lo, g->val + lo, sizeof(float) * (size_t)(hi - lo));
    }
}

void rmat_free(rmat_graph *g)
{
    if (!g) return;
    free(g->rp); free(g->col); free(g->val); free(g);
}

/* ---- sparse features ---------------------------------------------------- */

static inline int feat_present(uint64_t seed, int64_t i, int64_t j, int64_t F, double rho)
{
    return u01(draw(seed, STREAM_FEAT_POS, (uint64_t)(i * F + j))) < rho;
}

/* Row lengths of the feature matrix (n rows); returns nnz. */
int64_t feat_count(int64_t n, int64_t F, double rho, uint64_t seed, int64_t *rowlen)
{
    int64_t total = 0;
#pragma omp parallel for schedule(static) reduction(+ : total)
    for (int64_t i = 0; i < n; ++i) {
        int64_t c = 0;
        for (int64_t j = 0; j < F; ++j) c += feat_present(seed, i, j, F, rho);
        rowlen[i] = c;
        total += c;
    }
    return total;
}

/* Fill the feature matrix given row_ptr (int64, from feat_count's lengths). */
void feat_fill(int64_t n, int64_t F, double rho, uint64_t seed, const int64_t *rp,
               int32_t *col, float *val)
{
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        int64_t w = rp[i];
        for (int64_t j = 0; j < F; ++j) {
            if (!feat_present(seed, i, j, F, rho)) continue;
            double u = u01(draw(seed, STREAM_FEAT_VAL, (uint64_t)(i * F + j)));
            col[w] = (int32_t)j;
            val[w] = (float)(-1.0 + 2.0 * u);
            ++w;
        }
    }
}
