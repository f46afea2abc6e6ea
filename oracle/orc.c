/*
 * CPU oracle for the RSC aggregation hot path.
 *
 * TEST INFRASTRUCTURE ONLY. This file is the plain, slow, obviously correct
 * reference that the GPU library is checked against. Only the test suite,
 * the smoke check and the benchmark's CPU-baseline leg may load it; the
 * product path never calls it. It shares no code, header or table with the
 * GPU library.
 *
 * Paper: Liu et al., "RSC: Accelerate Graph Neural Networks Training via
 * Randomized Sparse Computations", ICML 2023 (arXiv 2210.10737).
 *
 * Arithmetic conventions (the paper does not state precision; these are the
 * readings this oracle fixes):
 *   - every floating-point reduction runs in fp64, in plain sequential index
 *     order; products of two fp32 values are exact in fp64;
 *   - the pair key is q = cn2 * rn2 (squared norms, no square root), encoded
 *     as the unsigned integer u = isnan(q) ? 0 : bits(q) + 1, whose unsigned
 *     order equals the order of q for q >= 0 and puts NaN last;
 *   - top-k ties go to the lower index.
 *
 * Rows are independent, so the row loops run one row per OpenMP thread
 * iteration; no reduction crosses threads.
 *
 * Pins (tests/test_oracle_pins.py): dense brute force, B = I, permutation
 * matrices, closed forms on regular graphs, Cauchy-Schwarz on the score mass,
 * an independent selection method, slice identities, a hand-worked greedy
 * example with its derivation, and the greedy's invariants; for SpMM_MEAN the
 * dense definition and the appendix example; for the randomized sampler the
 * generator's published outputs, weights re-derived independently, draw
 * frequencies, infinite scores, unbiasedness and a draw constructed to fall
 * exactly on a CDF boundary (the W_i > u rule: column i owns [W_{i-1}, W_i));
 * for the scaled slice the dense definition.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------------ */
/* O0. CSR well-formedness (section 3.3.1: row i occupies Rowptr[i] ..
 * Rowptr[i+1]-1 of Col and Val). Columns must be strictly increasing within a
 * row (sorted and unique: a duplicate (i, j) entry would make the column norm
 * differ from the norm of the merged column).
 * Returns 0 if valid, else a positive code naming the first violation. */
int orc_check_csr(int32_t n_rows, int32_t n_cols, const int32_t *rowptr, const int32_t *col) {
    if (n_rows < 0 || n_cols < 0) return 1;
    if (rowptr[0] != 0) return 2;
    for (int32_t i = 0; i < n_rows; ++i) {
        if (rowptr[i + 1] < rowptr[i]) return 3;
        for (int32_t t = rowptr[i]; t < rowptr[i + 1]; ++t) {
            if (col[t] < 0 || col[t] >= n_cols) return 4;
            if (t > rowptr[i] && col[t] <= col[t - 1]) return 5;
        }
    }
    return 0;
}

/* O1. The normalised adjacency (section 2.1): A_hat = D^-1/2 (A + I) D^-1/2,
 * D the degree matrix of A + I. For a 0/1 symmetric structure that already
 * holds the diagonal, deg_i is the length of row i and
 * val_ij = fl32(1 / sqrt(deg_i * deg_j)) (fp64 arithmetic, one rounding to
 * fp32). Returns how many stored values differ bitwise from that. */
int64_t orc_check_gcn_values(int32_t n, const int32_t *rowptr, const int32_t *col, const float *val) {
    int64_t bad = 0;
    for (int32_t i = 0; i < n; ++i) {
        int has_diag = 0;
        for (int32_t t = rowptr[i]; t < rowptr[i + 1]; ++t) {
            int32_t j = col[t];
            if (j == i) has_diag = 1;
            double di = (double)(rowptr[i + 1] - rowptr[i]);
            double dj = (double)(rowptr[j + 1] - rowptr[j]);
            float want = (float)(1.0 / sqrt(di * dj));
            if (memcmp(&want, &val[t], sizeof(float)) != 0) ++bad;
        }
        if (!has_diag) ++bad;
    }
    return bad;
}

/* ------------------------------------------------------------------------ */
/* O2 / O7. Sparse-dense product Y = A B (the SpMM of Eq. 1's implementation
 * form, section 2.1; the same routine applied to a sliced matrix is the
 * top-k approximation of section 2.2.1, whose kept pairs are summed with
 * scale 1). For each row i and feature j, accumulate val[t] * B[col[t], j]
 * over t = Rowptr[i] .. Rowptr[i+1]-1 in order, in fp64, then round once to
 * fp32. If S is given, also store S[i, j] = sum |val[t]| * |B[col[t], j]|
 * (fp64), the magnitude the relative-error metric divides by.
 * If `rows` is given, only rows[0..n_sel) are computed, and output row r of
 * Y / S corresponds to rows[r]; otherwise all n_rows rows are computed. */
void orc_spmm(int32_t n_rows, const int32_t *rowptr, const int32_t *col, const float *val,
              const float *B, int32_t d, int64_t ldb, float *Y, int64_t ldy,
              double *S, int64_t lds, const int32_t *rows, int32_t n_sel) {
    int32_t count = rows ? n_sel : n_rows;
#pragma omp parallel for schedule(dynamic, 64)
    for (int32_t r = 0; r < count; ++r) {
        int32_t i = rows ? rows[r] : r;
        for (int32_t j = 0; j < d; ++j) {
            double acc = 0.0, mag = 0.0;
            for (int32_t t = rowptr[i]; t < rowptr[i + 1]; ++t) {
                double a = (double)val[t];
                double b = (double)B[(int64_t)col[t] * ldb + j];
                acc += a * b;
                mag += fabs(a) * fabs(b);
            }
            Y[(int64_t)r * ldy + j] = (float)acc;
            if (S) S[(int64_t)r * lds + j] = mag;
        }
    }
    (void)n_rows;
}

/* ------------------------------------------------------------------------ */
/* O3. Column square-norms of the sparse operand X (Eq. 3's ||X[:, i]||, and
 * the ||A_hat^T[:, i]|| of Eq. 4a). Column i of X is row i of X^T, so given
 * the CSR of X^T: cn2[i] = sum over row i of X^T of val^2, fp64, in order.
 * colnnz[i] = number of stored entries in column i of X (Eq. 4b's #nnz_i). */
void orc_col_sqnorms(int32_t n, const int32_t *rowptr_t, const float *val_t, double *cn2,
                     int32_t *colnnz) {
#pragma omp parallel for schedule(dynamic, 256)
    for (int32_t i = 0; i < n; ++i) {
        double acc = 0.0;
        for (int32_t t = rowptr_t[i]; t < rowptr_t[i + 1]; ++t) {
            double v = (double)val_t[t];
            acc += v * v;
        }
        cn2[i] = acc;
        if (colnnz) colnnz[i] = rowptr_t[i + 1] - rowptr_t[i];
    }
}

/* O4. Pair scores (Eq. 3 and the top-k rule of section 2.2.1). The pair i
 * score is ||X[:, i]|| * ||Y[i, :]|| divided by a positive constant common
 * to all pairs; ranking by it equals ranking by q_i = cn2_i * rn2_i, since
 * squaring is monotone on non-negative values.
 *   rn2[i] = sum_{j < d} B[i, j]^2 (fp64, ascending j)
 *   q[i]   = cn2[i] * rn2[i] (fp64)
 *   key[i] = isnan(q) ? 0 : bits(q) + 1
 *   score[i] = fl32(sqrt(q[i])), the unnormalised pair score.
 * Any of rn2 / q / score may be NULL. */
void orc_pair_keys(int32_t n, const double *cn2, const float *B, int32_t d, int64_t ldb,
                   double *rn2, double *q, uint64_t *key, float *score) {
#pragma omp parallel for schedule(static)
    for (int32_t i = 0; i < n; ++i) {
        double acc = 0.0;
        for (int32_t j = 0; j < d; ++j) {
            double b = (double)B[(int64_t)i * ldb + j];
            acc += b * b;
        }
        double qq = cn2[i] * acc;
        uint64_t bits;
        memcpy(&bits, &qq, sizeof bits);
        if (rn2) rn2[i] = acc;
        if (q) q[i] = qq;
        key[i] = isnan(qq) ? 0u : bits + 1u;
        if (score) score[i] = (float)sqrt(qq);
    }
}

/* ------------------------------------------------------------------------ */
/* O5. Top-k selection (section 2.2.1): the k pairs with the largest score,
 * kept deterministically. Ties are broken by the lower index. Sort all
 * indices by (key descending, index ascending), keep the first k, and return
 * them in ascending index order plus an n-bit mask (bit i of word i/32). */
static const uint64_t *g_sort_keys;
static int cmp_key_desc_idx_asc(const void *pa, const void *pb) {
    int32_t a = *(const int32_t *)pa, b = *(const int32_t *)pb;
    uint64_t ka = g_sort_keys[a], kb = g_sort_keys[b];
    if (ka != kb) return ka > kb ? -1 : 1;
    return (a > b) - (a < b);
}
static int cmp_i32(const void *pa, const void *pb) {
    int32_t a = *(const int32_t *)pa, b = *(const int32_t *)pb;
    return (a > b) - (a < b);
}

/* Fills order[0..n) with the indices sorted by (key desc, index asc).
 * Not reentrant (qsort has no context argument in C99). */
void orc_rank_order(int32_t n, const uint64_t *key, int32_t *order) {
    for (int32_t i = 0; i < n; ++i) order[i] = i;
    g_sort_keys = key;
    qsort(order, (size_t)n, sizeof(int32_t), cmp_key_desc_idx_asc);
    g_sort_keys = NULL;
}

void orc_topk(int32_t n, const uint64_t *key, int32_t k, int32_t *idx, uint32_t *mask) {
    int32_t *order = (int32_t *)malloc((size_t)(n > 0 ? n : 1) * sizeof(int32_t));
    orc_rank_order(n, key, order);
    memcpy(idx, order, (size_t)k * sizeof(int32_t));
    qsort(idx, (size_t)k, sizeof(int32_t), cmp_i32);
    memset(mask, 0, (size_t)((n + 31) / 32) * sizeof(uint32_t));
    for (int32_t t = 0; t < k; ++t) mask[idx[t] >> 5] |= 1u << (idx[t] & 31);
    free(order);
}

/* ------------------------------------------------------------------------ */
/* O6. Column slice of a CSR matrix (section 3.3.1 and Fig. 5's rebuild of
 * Rowptr and Col; appendix C: whole columns are dropped and every row is
 * kept). For each row in order, copy (col[t], val[t]) when bit col[t] of
 * the mask is set; Rowptr'[i+1] = Rowptr'[i] + kept count of row i.
 * Column ids stay global. Returns nnz'. */
int64_t orc_slice(int32_t n_rows, const int32_t *rowptr, const int32_t *col, const float *val,
                  const uint32_t *mask, int32_t *rowptr_out, int32_t *col_out, float *val_out) {
    int64_t w = 0;
    rowptr_out[0] = 0;
    for (int32_t i = 0; i < n_rows; ++i) {
        for (int32_t t = rowptr[i]; t < rowptr[i + 1]; ++t) {
            int32_t c = col[t];
            if ((mask[c >> 5] >> (c & 31)) & 1u) {
                col_out[w] = c;
                val_out[w] = val[t];
                ++w;
            }
        }
        rowptr_out[i + 1] = (int32_t)w;
    }
    return w;
}

/* ------------------------------------------------------------------------ */
/* O8 (i). Uniform column budget (section 5.2.2, k_l = C |V|), with C given
 * as the rational num/den: k = floor(n * num / den) in integer arithmetic. */
int32_t orc_k_from_fraction(int32_t n, int32_t num, int32_t den) {
    return (int32_t)(((int64_t)n * (int64_t)num) / (int64_t)den);
}

/* O8 (ii). Layer-wise budget allocation, the greedy solution of Eq. 4a/4b
 * (section 3.2.1 and Algorithm 1 of appendix B).
 *
 * Inputs per layer l < L: pair keys key[l][0..n) (O4 encoding), hidden width
 * d[l], and ||grad H^(l+1)||_F^2 as fro_b2[l]; shared: colnnz[0..n), |E| =
 * nnz, ||A||_F^2 = fro_a2, budget C = C_num/C_den, step alpha|V| with
 * alpha = a_num/a_den.
 *
 * Readings fixed here:
 *   - per layer, pairs are ranked by (key desc, index asc), so Top_k is the
 *     first k of that order;
 *   - pair i contributes sqrt(q_i) / (||A||_F ||grad H||_F) to the objective,
 *     with ||.||_F = sqrt of the given squared norm; a NaN key (u = 0)
 *     contributes 0;
 *   - the step is max(1, floor(n * a_num / a_den));
 *   - the error increment of shrinking layer l from k to k' = max(0, k-step)
 *     is the fp64 sum, in rank order, of the contributions at ranks
 *     k' .. k-1, divided by the layer's normaliser;
 *   - the loop runs while Bud * C_den > C_num * sum_l |E| d_l (the budget of
 *     Eq. 4b is met with equality), picks the eligible layer (k_l > 0) with
 *     the smallest increment, the lowest layer index on ties, and stops when
 *     no layer is eligible;
 *   - Bud starts at sum_l |E| d_l and drops by d_m times the colnnz sum of
 *     the removed ranks.
 * Writes k_out[0..L) and returns the final Bud. */
int64_t orc_greedy(int32_t L, int32_t n, int64_t nnz, const uint64_t *const *key,
                   const int32_t *colnnz, const int32_t *d, double fro_a2, const double *fro_b2,
                   int32_t C_num, int32_t C_den, int32_t a_num, int32_t a_den, int32_t *k_out) {
    int32_t **order = (int32_t **)malloc((size_t)L * sizeof(int32_t *));
    int64_t total = 0;
    for (int32_t l = 0; l < L; ++l) {
        order[l] = (int32_t *)malloc((size_t)(n > 0 ? n : 1) * sizeof(int32_t));
        orc_rank_order(n, key[l], order[l]);
        k_out[l] = n;
        total += nnz * (int64_t)d[l];
    }
    int32_t step = (int32_t)(((int64_t)n * a_num) / a_den);
    if (step < 1) step = 1;
    int64_t bud = total;
    while ((__int128)bud * C_den > (__int128)C_num * total) {  /* exact: both sides may pass 2^63 */
        int32_t best = -1;
        double best_inc = 0.0;
        for (int32_t l = 0; l < L; ++l) {
            if (k_out[l] <= 0) continue;
            int32_t k2 = k_out[l] - step > 0 ? k_out[l] - step : 0;
            double s = 0.0;
            for (int32_t p = k2; p < k_out[l]; ++p) {
                uint64_t u = key[l][order[l][p]];
                if (u == 0) continue;
                uint64_t bits = u - 1;
                double qq;
                memcpy(&qq, &bits, sizeof qq);
                s += sqrt(qq);
            }
            double inc = s / (sqrt(fro_a2) * sqrt(fro_b2[l]));
            if (best < 0 || inc < best_inc) { best = l; best_inc = inc; }
        }
        if (best < 0) break;
        int32_t k2 = k_out[best] - step > 0 ? k_out[best] - step : 0;
        int64_t drop = 0;
        for (int32_t p = k2; p < k_out[best]; ++p) drop += colnnz[order[best][p]];
        bud -= (int64_t)d[best] * drop;
        k_out[best] = k2;
    }
    for (int32_t l = 0; l < L; ++l) free(order[l]);
    free(order);
    return bud;
}

/* Threads the oracle's row loops use (OpenMP's current maximum). */
#include <omp.h>
int32_t orc_num_threads(void) { return (int32_t)omp_get_max_threads(); }

/* Sets the thread count of the following row loops (the CPU baseline times
 * the oracle on all host cores and on one); returns the count now in force. */
int32_t orc_set_num_threads(int32_t t) {
    if (t >= 1) omp_set_num_threads(t);
    return (int32_t)omp_get_max_threads();
}

/* ------------------------------------------------------------------------ */
/* SpMM_MEAN (appendix A.3): the MEAN aggregator D^-1 A H, D the degree
 * matrix of A, read as D_ii = number of stored entries of row i (the paper's
 * worked example divides every row by 2, the column count, which disagrees
 * with D^-1 A for its rows 0 and 1; the definition D^-1 A is followed here).
 * Y[i, j] = fl32( (sum_t val[t] * B[col[t], j]) / len_i ), the sum in fp64
 * in stored order; empty rows give 0. */
void orc_spmm_mean(int32_t n_rows, const int32_t *rowptr, const int32_t *col, const float *val,
                   const float *B, int32_t d, int64_t ldb, float *Y, int64_t ldy) {
#pragma omp parallel for schedule(dynamic, 64)
    for (int32_t i = 0; i < n_rows; ++i) {
        int32_t len = rowptr[i + 1] - rowptr[i];
        for (int32_t j = 0; j < d; ++j) {
            double acc = 0.0;
            for (int32_t t = rowptr[i]; t < rowptr[i + 1]; ++t)
                acc += (double)val[t] * (double)B[(int64_t)col[t] * ldb + j];
            Y[(int64_t)i * ldy + j] = len ? (float)(acc / (double)len) : 0.0f;
        }
    }
}

/* ------------------------------------------------------------------------ */
/* Randomized column-row sampling (section 2.2, Eq. 2 with the probabilities
 * of Eq. 3): k i.i.d. draws i_t ~ p, p_i = ||X[:, i]|| ||Y[i, :]|| / sum_j
 * (the same product), and the t-th sampled pair scaled by 1/(k p_{i_t}), the
 * unbiased estimator the section builds on. Readings fixed here:
 *   - p is held as integer weights w_i = floor(sqrt(q_i) * (2^S / m)),
 *     m = max_j sqrt(q_j), q decoded from the key (NaN -> 0), so the CDF is an
 *     exact int64 prefix sum W_i = w_0 + ... + w_i, total = W_{n-1}; S = 38
 *     for n <= 2^24, else 62 - ceil(log2 n), so that total <= 2^62;
 *   - draw t uses the t-th output (t = 0, 1, ...) of the SplitMix64
 *     generator seeded with `seed` (Steele, Lea & Flood 2014),
 *     u_t = floor(z_t * total / 2^64), and i_t = the smallest i with W_i > u_t;
 *   - the pairs drawn c_i times enter once, scaled by
 *     colw_i = c_i * total / (k * w_i) (fp64), i.e. c_i / (k p_i);
 *   - if some score is +Inf, the infinite ones share the mass uniformly
 *     (weight 2^S each, every other weight 0).
 * Outputs count[i] = c_i, colw[i] (0 where c_i = 0) and the mask of columns
 * with c_i > 0. If every weight is 0 nothing is drawn. */
uint64_t orc_splitmix64(uint64_t seed, uint64_t t) {
    uint64_t z = seed + (t + 1) * 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

static double key_sqrt(uint64_t u) {
    if (u == 0) return 0.0;
    uint64_t bits = u - 1;
    double q;
    memcpy(&q, &bits, sizeof q);
    return sqrt(q);
}

void orc_sample_columns(int32_t n, const uint64_t *key, int32_t k, uint64_t seed, int32_t *count,
                        double *colw, uint32_t *mask, int64_t *w_out) {
    int64_t *W = (int64_t *)malloc((size_t)(n > 0 ? n : 1) * sizeof(int64_t));
    int64_t *w = (int64_t *)malloc((size_t)(n > 0 ? n : 1) * sizeof(int64_t));
    double m = 0.0;
    for (int32_t i = 0; i < n; ++i) {
        double r = key_sqrt(key[i]);
        if (r > m) m = r;
    }
    int bits = 38; /* weight resolution S */
    if (n > (1 << 24)) {
        int lg = 0;
        while (((int64_t)1 << lg) < (int64_t)n) ++lg;
        bits = 62 - lg;
    }
    double scale = m > 0.0 ? ldexp(1.0, bits) / m : 0.0;
    int64_t acc = 0;
    for (int32_t i = 0; i < n; ++i) {
        double r = key_sqrt(key[i]);
        /* infinite scores share the mass uniformly */
        w[i] = isinf(m) ? (isinf(r) ? ((int64_t)1 << bits) : 0) : (int64_t)(r * scale);
        acc += w[i];
        W[i] = acc;
        count[i] = 0;
        if (w_out) w_out[i] = w[i];
    }
    int64_t total = acc;
    for (int32_t t = 0; total > 0 && t < k; ++t) {
        uint64_t z = orc_splitmix64(seed, (uint64_t)t);
        uint64_t u = (uint64_t)(((unsigned __int128)z * (uint64_t)total) >> 64);
        int32_t lo = 0, hi = n - 1; /* smallest i with W[i] > u */
        while (lo < hi) {
            int32_t mid = lo + (hi - lo) / 2;
            if ((uint64_t)W[mid] > u) hi = mid; else lo = mid + 1;
        }
        count[lo] += 1;
    }
    memset(mask, 0, (size_t)((n + 31) / 32) * sizeof(uint32_t));
    for (int32_t i = 0; i < n; ++i) {
        colw[i] = count[i] ? (double)count[i] * (double)total / ((double)k * (double)w[i]) : 0.0;
        if (count[i]) mask[i >> 5] |= 1u << (i & 31);
    }
    free(W);
    free(w);
}

/* Slice with per-column scale: as orc_slice, each kept value becomes
 * fl32(val * colw[col]) (fp64 product, one rounding). */
int64_t orc_slice_scaled(int32_t n_rows, const int32_t *rowptr, const int32_t *col, const float *val,
                         const uint32_t *mask, const double *colw, int32_t *rowptr_out,
                         int32_t *col_out, float *val_out) {
    int64_t w = 0;
    rowptr_out[0] = 0;
    for (int32_t i = 0; i < n_rows; ++i) {
        for (int32_t t = rowptr[i]; t < rowptr[i + 1]; ++t) {
            int32_t c = col[t];
            if ((mask[c >> 5] >> (c & 31)) & 1u) {
                col_out[w] = c;
                val_out[w] = (float)((double)val[t] * colw[c]);
                ++w;
            }
        }
        rowptr_out[i + 1] = (int32_t)w;
    }
    return w;
}

/* ------------------------------------------------------------------------ */
/* Eq. 4a's normalisers: ||A||_F^2 is the sum of the column square-norms cn2
 * and ||grad H||_F^2 the sum of the row square-norms rn2. The plain
 * sequential fp64 sum of x[0..n). */
double orc_sum_sequential(int64_t n, const double *x) {
    double s = 0.0;
    for (int64_t i = 0; i < n; ++i) s += x[i];
    return s;
}

/* Staleness of a cached selection (section 3.3.1, Fig. 4: how well the top-k
 * pairs chosen at one refresh still match the ranking at the next). With S
 * the previous selection (prev_mask bit i set iff i in S, |S| = k) and
 * `order` the new ranking of the n pairs, best first, the matching score is
 * the AUC of S under that ranking: among all pairs (i in S, j not in S), the
 * fraction in which i is ranked before j. Counted directly: walking the
 * ranking from the best pair, each pair outside S is preceded by every pair
 * of S seen so far. Returns NaN when S is empty or holds every pair.
 * *overlap_count (nullable) receives |S cap S_new| with S_new given by
 * new_mask (nullable: then 0). */
double orc_selection_auc(int32_t n, const int32_t *order, const uint32_t *prev_mask, const uint32_t *new_mask,
                         int64_t *overlap_count) {
    int64_t k = 0, seen = 0, pairs_above = 0, both = 0;
    for (int32_t i = 0; i < n; ++i) {
        int in_prev = (prev_mask[i >> 5] >> (i & 31)) & 1u;
        k += in_prev;
        if (new_mask && in_prev && ((new_mask[i >> 5] >> (i & 31)) & 1u)) ++both;
    }
    if (overlap_count) *overlap_count = both;
    if (k == 0 || k == n) return NAN;
    for (int32_t p = 0; p < n; ++p) {
        int32_t i = order[p];
        if ((prev_mask[i >> 5] >> (i & 31)) & 1u)
            ++seen;
        else
            pairs_above += seen;
    }
    return (double)pairs_above / ((double)k * (double)(n - k));
}
