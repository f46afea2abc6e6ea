/*
 * Seeded synthetic inputs for the GCN aggregation workloads.
 *
 * Holds the input recipe only: graph structure (Erdos-Renyi or Chung-Lu),
 * the symmetric GCN normalisation that turns a structure into the operand
 * A_hat = D^-1/2 (A+I) D^-1/2 (paper section 2.1), and dense N(0,1) matrices.
 * Nothing here computes any step of the aggregation, the scores, the
 * selection or the slicing.
 *
 * Every random draw is a pure function of (seed, stream, counter), so the
 * result does not depend on the number of threads.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <omp.h>

/* splitmix64 finaliser (Steele, Lea & Flood, OOPSLA 2014) used as a hash. */
static inline uint64_t mix64(uint64_t x) {
    x += 0x9E3779B97F4A7C15ull;
    x = (x ^ (x >> 30)) * 0xBF58476D1CE4E5B9ull;
    x = (x ^ (x >> 27)) * 0x94D049BB133111EBull;
    return x ^ (x >> 31);
}

static inline uint64_t draw(uint64_t seed, uint64_t stream, uint64_t i) {
    return mix64(mix64(seed * 0xD1342543DE82EF95ull + stream) ^ (i * 0x9E3779B97F4A7C15ull + 0x632BE59BD9B4E019ull));
}

/* uniform double in [0, 1) with 53 random bits */
static inline double unif(uint64_t r) { return (double)(r >> 11) * 0x1.0p-53; }

enum { ST_PERM = 1, ST_WEIGHT = 2, ST_EDGE_U = 3, ST_EDGE_V = 4, ST_EDGE_P = 5, ST_ER = 6, ST_DENSE = 7,
       ST_BUCKET_C = 8, ST_BUCKET_V = 9 };

/* ---- dense N(0,1) fp32 matrix, Box-Muller on counter pairs ---------------- */
void syn_dense_normal(uint64_t seed, int64_t rows, int64_t cols, int64_t ld, float *out) {
    int64_t total = rows * cols;
    int64_t pairs = (total + 1) / 2;
#pragma omp parallel for schedule(static)
    for (int64_t p = 0; p < pairs; ++p) {
        double u1 = ((double)(draw(seed, ST_DENSE, 2 * p) >> 11) + 1.0) * 0x1.0p-53; /* (0,1] */
        double u2 = unif(draw(seed, ST_DENSE, 2 * p + 1));
        double r = sqrt(-2.0 * log(u1));
        double th = 6.283185307179586476925 * u2;
        int64_t e0 = 2 * p, e1 = 2 * p + 1;
        out[(e0 / cols) * ld + (e0 % cols)] = (float)(r * cos(th));
        if (e1 < total) out[(e1 / cols) * ld + (e1 % cols)] = (float)(r * sin(th));
    }
}

/* ---- helpers -------------------------------------------------------------- */
static int cmp_i32(const void *a, const void *b) {
    int32_t x = *(const int32_t *)a, y = *(const int32_t *)b;
    return (x > y) - (x < y);
}

/* Fisher-Yates permutation of [0, n) from the seeded stream. */
static void make_perm(uint64_t seed, int32_t n, int32_t *perm) {
    for (int32_t i = 0; i < n; ++i) perm[i] = i;
    for (int32_t i = n - 1; i > 0; --i) {
        uint64_t r = draw(seed, ST_PERM, (uint64_t)i);
        int32_t j = (int32_t)(((unsigned __int128)r * (uint64_t)(i + 1)) >> 64);
        int32_t t = perm[i]; perm[i] = perm[j]; perm[j] = t;
    }
}

/*
 * Build a symmetric CSR with self-loops from an undirected edge list
 * (u[e], v[e]), e < m, with u != v (self pairs are dropped here anyway).
 * Duplicates are removed, columns sorted within each row, the diagonal added.
 * Returns nnz; rowptr has n+1 entries; col is allocated here (caller frees
 * with syn_free).
 */
static int64_t build_sym_csr(int32_t n, int64_t m, const int32_t *u, const int32_t *v,
                             int32_t *rowptr, int32_t **col_out) {
    int64_t *cnt = (int64_t *)calloc((size_t)n + 1, sizeof(int64_t));
#pragma omp parallel for schedule(static)
    for (int64_t e = 0; e < m; ++e) {
        if (u[e] == v[e]) continue;
#pragma omp atomic
        cnt[u[e] + 1]++;
#pragma omp atomic
        cnt[v[e] + 1]++;
    }
    for (int32_t i = 0; i < n; ++i) cnt[i + 1] += cnt[i];
    int64_t tot = cnt[n];
    int32_t *buf = (int32_t *)malloc((size_t)(tot > 0 ? tot : 1) * sizeof(int32_t));
    int64_t *pos = (int64_t *)malloc((size_t)n * sizeof(int64_t));
    memcpy(pos, cnt, (size_t)n * sizeof(int64_t));
#pragma omp parallel for schedule(static)
    for (int64_t e = 0; e < m; ++e) {
        if (u[e] == v[e]) continue;
        int64_t p, q;
#pragma omp atomic capture
        p = pos[u[e]]++;
#pragma omp atomic capture
        q = pos[v[e]]++;
        buf[p] = v[e];
        buf[q] = u[e];
    }
    free(pos);
    /* sort + unique each row, count distinct + self-loop */
    int32_t *len = (int32_t *)malloc((size_t)n * sizeof(int32_t));
#pragma omp parallel for schedule(dynamic, 1024)
    for (int32_t i = 0; i < n; ++i) {
        int32_t *r = buf + cnt[i];
        int64_t L = cnt[i + 1] - cnt[i];
        qsort(r, (size_t)L, sizeof(int32_t), cmp_i32);
        int64_t w = 0;
        for (int64_t t = 0; t < L; ++t)
            if (w == 0 || r[t] != r[w - 1]) r[w++] = r[t];
        len[i] = (int32_t)w + 1;
    }
    rowptr[0] = 0;
    int64_t acc = 0;
    for (int32_t i = 0; i < n; ++i) { acc += len[i]; rowptr[i + 1] = (int32_t)acc; }
    int32_t *col = (int32_t *)malloc((size_t)acc * sizeof(int32_t));
#pragma omp parallel for schedule(dynamic, 1024)
    for (int32_t i = 0; i < n; ++i) {
        const int32_t *r = buf + cnt[i];
        int32_t L = len[i] - 1, o = rowptr[i], t = 0;
        while (t < L && r[t] < i) col[o++] = r[t++];
        col[o++] = i;
        while (t < L) col[o++] = r[t++];
    }
    free(len); free(buf); free(cnt);
    *col_out = col;
    return acc;
}

/* Symmetric GCN normalisation of a 0/1 structure that already holds the
 * diagonal: val_ij = fl32(1 / sqrt(deg_i * deg_j)), deg = row length of A+I
 * (paper section 2.1, the normalised adjacency). */
void syn_gcn_values(int32_t n, const int32_t *rowptr, const int32_t *col, float *val) {
#pragma omp parallel for schedule(dynamic, 1024)
    for (int32_t i = 0; i < n; ++i) {
        double di = (double)(rowptr[i + 1] - rowptr[i]);
        for (int32_t t = rowptr[i]; t < rowptr[i + 1]; ++t) {
            double dj = (double)(rowptr[col[t] + 1] - rowptr[col[t]]);
            val[t] = (float)(1.0 / sqrt(di * dj));
        }
    }
}

/* ---- Erdos-Renyi G(n, p), symmetric, self-loops added ---------------------- */
int64_t syn_er(uint64_t seed, int32_t n, double p, int32_t *rowptr, int32_t **col_out) {
    /* one Bernoulli(p) draw per unordered pair (i < j), pair index i*n + j */
    int64_t m = 0, cap = (int64_t)((double)n * (n - 1) / 2 * p * 1.5) + 1024;
    int32_t *u = (int32_t *)malloc((size_t)cap * sizeof(int32_t));
    int32_t *v = (int32_t *)malloc((size_t)cap * sizeof(int32_t));
    for (int32_t i = 0; i < n; ++i)
        for (int32_t j = i + 1; j < n; ++j)
            if (unif(draw(seed, ST_ER, (uint64_t)i * (uint64_t)n + (uint64_t)j)) < p) {
                if (m == cap) {
                    cap *= 2;
                    u = (int32_t *)realloc(u, (size_t)cap * sizeof(int32_t));
                    v = (int32_t *)realloc(v, (size_t)cap * sizeof(int32_t));
                }
                u[m] = i; v[m] = j; ++m;
            }
    int64_t nnz = build_sym_csr(n, m, u, v, rowptr, col_out);
    free(u); free(v);
    return nnz;
}

/* ---- Chung-Lu with given expected weights ---------------------------------
 * Each of m draws picks two endpoints independently with probability
 * proportional to w (Walker/Vose alias table), endpoints are mapped through a
 * seeded random permutation (no artificial locality), then the multigraph is
 * reduced to a simple symmetric graph with self-loops. */
static int64_t chung_lu(uint64_t seed, int32_t n, const double *w, int64_t m,
                        int32_t *rowptr, int32_t **col_out) {
    double *prob = (double *)malloc((size_t)n * sizeof(double));
    int32_t *alias = (int32_t *)malloc((size_t)n * sizeof(int32_t));
    int32_t *small = (int32_t *)malloc((size_t)n * sizeof(int32_t));
    int32_t *large = (int32_t *)malloc((size_t)n * sizeof(int32_t));
    double W = 0.0;
    for (int32_t i = 0; i < n; ++i) W += w[i];
    int32_t ns = 0, nl = 0;
    for (int32_t i = 0; i < n; ++i) {
        prob[i] = w[i] * (double)n / W;
        alias[i] = i;
        if (prob[i] < 1.0) small[ns++] = i; else large[nl++] = i;
    }
    while (ns > 0 && nl > 0) {
        int32_t s = small[--ns], l = large[nl - 1];
        alias[s] = l;
        prob[l] = (prob[l] + prob[s]) - 1.0;
        if (prob[l] < 1.0) { --nl; small[ns++] = l; }
    }
    while (nl > 0) prob[large[--nl]] = 1.0;
    while (ns > 0) prob[small[--ns]] = 1.0;
    free(small); free(large);

    int32_t *perm = (int32_t *)malloc((size_t)n * sizeof(int32_t));
    make_perm(seed, n, perm);
    int32_t *u = (int32_t *)malloc((size_t)m * sizeof(int32_t));
    int32_t *v = (int32_t *)malloc((size_t)m * sizeof(int32_t));
#pragma omp parallel for schedule(static)
    for (int64_t e = 0; e < m; ++e) {
        uint64_t ru = draw(seed, ST_EDGE_U, (uint64_t)e), rv = draw(seed, ST_EDGE_V, (uint64_t)e);
        int32_t iu = (int32_t)(((unsigned __int128)ru * (uint64_t)n) >> 64);
        int32_t iv = (int32_t)(((unsigned __int128)rv * (uint64_t)n) >> 64);
        double fu = unif(draw(seed, ST_EDGE_P, 2 * (uint64_t)e));
        double fv = unif(draw(seed, ST_EDGE_P, 2 * (uint64_t)e + 1));
        if (fu >= prob[iu]) iu = alias[iu];
        if (fv >= prob[iv]) iv = alias[iv];
        u[e] = perm[iu];
        v[e] = perm[iv];
    }
    free(prob); free(alias); free(perm);
    int64_t nnz = build_sym_csr(n, m, u, v, rowptr, col_out);
    free(u); free(v);
    return nnz;
}

/* Truncated Pareto weights: quantile i of w = wmin * U^(-1/(gamma-1)), clipped
 * at wmax, with wmin solved (bisection on the closed-form clipped mean) so the
 * mean weight equals `mean`. */
int64_t syn_chung_lu_powerlaw(uint64_t seed, int32_t n, double mean, double gamma, double wmax,
                              int64_t m, int32_t *rowptr, int32_t **col_out) {
    double a = gamma - 1.0, e = 1.0 - 1.0 / a;
    double lo = 1e-6, hi = mean;
    for (int it = 0; it < 200; ++it) {
        double wmin = 0.5 * (lo + hi);
        double us = pow(wmin / wmax, a);
        double mu = wmin * (1.0 - pow(us, e)) / e + us * wmax;
        if (mu < mean) lo = wmin; else hi = wmin;
    }
    double wmin = 0.5 * (lo + hi);
    double *w = (double *)malloc((size_t)n * sizeof(double));
    for (int32_t i = 0; i < n; ++i) {
        double U = ((double)i + 0.5) / (double)n;
        double x = wmin * pow(U, -1.0 / a);
        w[i] = x < wmax ? x : wmax;
    }
    int64_t nnz = chung_lu(seed, n, w, m, rowptr, col_out);
    free(w);
    return nnz;
}

/* Near-uniform weights w_i ~ U[wlo, whi]. */
int64_t syn_chung_lu_uniform(uint64_t seed, int32_t n, double wlo, double whi, int64_t m,
                             int32_t *rowptr, int32_t **col_out) {
    double *w = (double *)malloc((size_t)n * sizeof(double));
    for (int32_t i = 0; i < n; ++i) w[i] = wlo + (whi - wlo) * unif(draw(seed, ST_WEIGHT, (uint64_t)i));
    int64_t nnz = chung_lu(seed, n, w, m, rowptr, col_out);
    free(w);
    return nnz;
}

void syn_copy_free(int32_t *src, int64_t count, int32_t *dst) {
    memcpy(dst, src, (size_t)count * sizeof(int32_t));
    free(src);
}

/* ---- bucketed CSR of given row lengths (large-size edge cases) ------------
 * Row r with L_r <= n_cols entries splits [0, n_cols) into L_r buckets of
 * near-equal width and takes one uniformly random column from each, so the
 * columns of a row are strictly increasing without sorting; values are
 * uniform in [-1, 1). O(1) work per entry and parallel over rows. */
void syn_bucket_csr(uint64_t seed, int32_t n_rows, int32_t n_cols, const int64_t *rowptr, int32_t *col,
                    float *val) {
#pragma omp parallel for schedule(dynamic, 1024)
    for (int32_t r = 0; r < n_rows; ++r) {
        const int64_t s = rowptr[r], len = rowptr[r + 1] - s;
        for (int64_t j = 0; j < len; ++j) {
            const int64_t lo = j * (int64_t)n_cols / len, hi = (j + 1) * (int64_t)n_cols / len;
            const uint64_t t = (uint64_t)(s + j);
            col[s + j] = (int32_t)(lo + (int64_t)(draw(seed, ST_BUCKET_C, t) % (uint64_t)(hi - lo)));
            val[s + j] = (float)(2.0 * unif(draw(seed, ST_BUCKET_V, t)) - 1.0);
        }
    }
}
