/*
 * XAttention CPU oracle -- TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT PATH.
 *
 * Only the tests, the smoke check and the benchmark's CPU-baseline leg may
 * load this library. It shares no code, header, table or helper with the GPU
 * library: it is a plain, slow, fp64 restatement of the paper's definitions
 * (XAttention, arXiv 2503.16428), written to be checked by eye against:
 *   - Sec. 3.2 "Threshold Block Selection": antidiagonal summation inside each
 *     S x S sub-block, softmax normalisation, and the find_blocks equation
 *     (minimal block set whose cumulative mass reaches tau);
 *   - Algorithm 1 "Block Selection": the strided reshape of the query block
 *     (sub-rows S-1 .. 0) and of the keys (sub-rows 0 .. S-1), scaled by
 *     1 / (sqrt(d_h) * S), softmax, find_blocks per query block;
 *   - Fig. 1 (right): attention computed only on the selected blocks.
 *
 * Readings where the paper is silent (listed with reasons in the design notes):
 *   - the append in Algorithm 1 concatenates along the feature axis, so
 *     reduced row R / column c have inner product
 *       sum_{t<S} q[R*S + S-1-t] . k[c*S + t];
 *   - causal masking is applied at reduced granularity (c <= R); blocks right
 *     of the diagonal block are never candidates;
 *   - a block's score is the mean over its B/S reduced rows of the reduced
 *     softmax mass in its B/S reduced columns (each query-block row sums to 1);
 *   - find_blocks: masses are taken as integers u_j = floor(score_j * 2^32)
 *     (score clamped to [0, 1]),
 *     the row total T = sum u_j, the target ceil(tau * T) (one IEEE fp64
 *     product), candidates ordered by (u desc, j asc), the shortest prefix of
 *     length >= 1 whose integer cumulative sum reaches the target; tau >= 1
 *     selects every candidate;
 *   - attention scale 1/sqrt(d); the softmax runs over the selected keys only
 *     (and keys <= query when causal).
 *
 * Inputs are bfloat16 bit patterns (uint16), widened exactly; every product
 * and sum is in fp64. Work is split over rows (head, query block) with OpenMP.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

typedef struct {
    int32_t batch, hq, hkv, seq, head_dim, causal;
} oracle_dims;

/* Exact widening of a bfloat16 bit pattern. */
static double bf(uint16_t h)
{
    union { uint32_t u; float f; } x;
    x.u = ((uint32_t)h) << 16;
    return (double)x.f;
}

/* Query head index (over batch*hq) -> its key/value head index (over batch*hkv):
 * contiguous grouping, g(h) = h // (hq / hkv) inside one batch element. */
static int kv_head(const oracle_dims *d, int h)
{
    int n = h / d->hq, hh = h % d->hq;
    return n * d->hkv + hh / (d->hq / d->hkv);
}

int oracle_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/*
 * Block scores of the query-block rows (row_h[i], row_b[i]).
 * out: nrows x NB doubles, NB = seq / B. Entries of non-candidate blocks are 0.
 */
void oracle_score_rows(const uint16_t *q, const uint16_t *k, const oracle_dims *d,
                       int B, int S, int nrows, const int32_t *row_h,
                       const int32_t *row_b, double *out)
{
    const int L = d->seq, D = d->head_dim, NB = L / B, NR = L / S, nr = B / S;
    const double scale = 1.0 / (sqrt((double)D) * (double)S);
#pragma omp parallel for schedule(dynamic, 1)
    for (int i = 0; i < nrows; ++i) {
        const int h = row_h[i], b = row_b[i];
        const uint16_t *Q = q + (size_t)h * L * D;
        const uint16_t *K = k + (size_t)kv_head(d, h) * L * D;
        double *row = out + (size_t)i * NB;
        double *x = (double *)malloc(sizeof(double) * NR);
        for (int j = 0; j < NB; ++j) row[j] = 0.0;
        for (int r = 0; r < nr; ++r) {
            const int R = b * nr + r;                 /* global reduced row */
            const int ncol = d->causal ? R + 1 : NR;   /* valid reduced columns */
            /* antidiagonal logits: sub-row S-1-t of the query group meets
             * sub-row t of the key group (Algorithm 1, reshape + product) */
            for (int c = 0; c < ncol; ++c) {
                double acc = 0.0;
                for (int t = 0; t < S; ++t) {
                    const uint16_t *qr = Q + (size_t)(R * S + S - 1 - t) * D;
                    const uint16_t *kr = K + (size_t)(c * S + t) * D;
                    for (int e = 0; e < D; ++e) acc += bf(qr[e]) * bf(kr[e]);
                }
                x[c] = acc * scale;
            }
            /* softmax over the reduced row */
            double m = -INFINITY;
            for (int c = 0; c < ncol; ++c) if (x[c] > m) m = x[c];
            double l = 0.0;
            for (int c = 0; c < ncol; ++c) l += exp(x[c] - m);
            /* mass per key block (B/S reduced columns per block) */
            for (int c = 0; c < ncol; ++c) row[c / nr] += exp(x[c] - m) / l;
        }
        for (int j = 0; j < NB; ++j) row[j] /= (double)nr;
        free(x);
    }
}

/*
 * Scoring-pattern variants of the pattern ablation (Sec. 4.5, Table 4): the
 * S positions summed inside each S x S sub-block are (qsub[t], t), t < S, for
 * a permutation qsub of 0 .. S-1 (one position per sub-block row and column).
 * qsub[t] = S-1-t is the antidiagonal of Algorithm 1, qsub[t] = t the main
 * diagonal, a random permutation the random pattern. Otherwise as
 * oracle_score_rows: scale 1/(sqrt(d) S), softmax per reduced row over
 * c <= R (causal), block mass averaged over the block's reduced rows.
 */
void oracle_score_pattern_rows(const uint16_t *q, const uint16_t *k, const oracle_dims *d,
                               int B, int S, const int32_t *qsub, int nrows,
                               const int32_t *row_h, const int32_t *row_b, double *out)
{
    const int L = d->seq, D = d->head_dim, NB = L / B, NR = L / S, nr = B / S;
    const double scale = 1.0 / (sqrt((double)D) * (double)S);
#pragma omp parallel for schedule(dynamic, 1)
    for (int i = 0; i < nrows; ++i) {
        const int h = row_h[i], b = row_b[i];
        const uint16_t *Q = q + (size_t)h * L * D;
        const uint16_t *K = k + (size_t)kv_head(d, h) * L * D;
        double *row = out + (size_t)i * NB;
        double *x = (double *)malloc(sizeof(double) * NR);
        for (int j = 0; j < NB; ++j) row[j] = 0.0;
        for (int r = 0; r < nr; ++r) {
            const int R = b * nr + r;
            const int ncol = d->causal ? R + 1 : NR;
            for (int c = 0; c < ncol; ++c) {
                double acc = 0.0;
                for (int t = 0; t < S; ++t) {
                    const uint16_t *qr = Q + (size_t)(R * S + qsub[t]) * D;
                    const uint16_t *kr = K + (size_t)(c * S + t) * D;
                    for (int e = 0; e < D; ++e) acc += bf(qr[e]) * bf(kr[e]);
                }
                x[c] = acc * scale;
            }
            double m = -INFINITY;
            for (int c = 0; c < ncol; ++c) if (x[c] > m) m = x[c];
            double l = 0.0;
            for (int c = 0; c < ncol; ++c) l += exp(x[c] - m);
            for (int c = 0; c < ncol; ++c) row[c / nr] += exp(x[c] - m) / l;
        }
        for (int j = 0; j < NB; ++j) row[j] /= (double)nr;
        free(x);
    }
}

typedef struct { uint64_t u; int32_t j; } cand;

static int cand_cmp(const void *a, const void *b)
{
    const cand *x = (const cand *)a, *y = (const cand *)b;
    if (x->u != y->u) return x->u > y->u ? -1 : 1;   /* mass descending */
    return x->j < y->j ? -1 : (x->j > y->j);          /* then index ascending */
}

static int int_cmp(const void *a, const void *b)
{
    int32_t x = *(const int32_t *)a, y = *(const int32_t *)b;
    return (x > y) - (x < y);
}

/*
 * find_blocks per row. scores: nrows x NB (any non-negative values; rows need
 * not be normalised). row_b gives the query block of each row (candidates are
 * j <= row_b when causal, all j otherwise).
 * idx: nrows x NB int32, first cnt[i] entries valid, ascending.
 */
void oracle_select_rows(const double *scores, int NB, int causal, int nrows,
                        const int32_t *row_b, float tau, int32_t *idx, int32_t *cnt)
{
#pragma omp parallel for schedule(dynamic, 16)
    for (int i = 0; i < nrows; ++i) {
        const int m = causal ? row_b[i] + 1 : NB;
        const double *s = scores + (size_t)i * NB;
        int32_t *out = idx + (size_t)i * NB;
        for (int j = 0; j < NB; ++j) out[j] = -1;
        if (tau >= 1.0f) {
            for (int j = 0; j < m; ++j) out[j] = j;
            cnt[i] = m;
            continue;
        }
        cand *c = (cand *)malloc(sizeof(cand) * m);
        uint64_t total = 0;
        for (int j = 0; j < m; ++j) {
            /* a block mass lies in [0, 1]; NaN counts as 0 */
            double v = s[j] > 0.0 ? (s[j] < 1.0 ? s[j] : 1.0) : 0.0;
            c[j].u = (uint64_t)floor(v * 4294967296.0);
            c[j].j = j;
            total += c[j].u;
        }
        const double prod = (double)tau * (double)total;
        const uint64_t target = (uint64_t)ceil(prod);
        qsort(c, (size_t)m, sizeof(cand), cand_cmp);
        uint64_t cum = 0;
        int n = 0;
        while (n < m) {
            cum += c[n].u;
            ++n;
            if (cum >= target) break;
        }
        for (int t = 0; t < n; ++t) out[t] = c[t].j;
        qsort(out, (size_t)n, sizeof(int32_t), int_cmp);
        cnt[i] = n;
        free(c);
    }
}

/*
 * Fixed-size selection (Sec. 4.5, Top-K vs. Top-Ratio ablation, Table 6): per
 * row keep the k_row[i] candidates that come first in the same (u desc,
 * j asc) order as find_blocks, u = floor(clamp(score, 0, 1) * 2^32); k is
 * clamped to [1, m] (m candidates), the output sorted ascending.
 */
void oracle_select_topk_rows(const double *scores, int NB, int causal, int nrows,
                             const int32_t *row_b, const int32_t *k_row, int32_t *idx,
                             int32_t *cnt)
{
#pragma omp parallel for schedule(dynamic, 16)
    for (int i = 0; i < nrows; ++i) {
        const int m = causal ? row_b[i] + 1 : NB;
        const double *s = scores + (size_t)i * NB;
        int32_t *out = idx + (size_t)i * NB;
        for (int j = 0; j < NB; ++j) out[j] = -1;
        int k = k_row[i] < 1 ? 1 : (k_row[i] > m ? m : k_row[i]);
        cand *c = (cand *)malloc(sizeof(cand) * m);
        for (int j = 0; j < m; ++j) {
            double v = s[j] > 0.0 ? (s[j] < 1.0 ? s[j] : 1.0) : 0.0;
            c[j].u = (uint64_t)floor(v * 4294967296.0);
            c[j].j = j;
        }
        qsort(c, (size_t)m, sizeof(cand), cand_cmp);
        for (int t = 0; t < k; ++t) out[t] = c[t].j;
        qsort(out, (size_t)k, sizeof(int32_t), int_cmp);
        cnt[i] = k;
        free(c);
    }
}

/*
 * Top-Ratio: the block count of a row is the fraction ratio of its m
 * candidates, rounded to the nearest whole block (halves up) and clamped to
 * [1, m]; ratio is the caller's fp32 value, the product taken in fp64. Then
 * as Top-K.
 */
void oracle_select_ratio_rows(const double *scores, int NB, int causal, int nrows,
                              const int32_t *row_b, const float *ratio_row, int32_t *idx,
                              int32_t *cnt)
{
    int32_t *k = (int32_t *)malloc(sizeof(int32_t) * (nrows > 0 ? nrows : 1));
    for (int i = 0; i < nrows; ++i) {
        const int m = causal ? row_b[i] + 1 : NB;
        const double want = floor((double)ratio_row[i] * (double)m + 0.5);
        k[i] = want < 1.0 ? 1 : (want > (double)m ? m : (int32_t)want);
    }
    oracle_select_topk_rows(scores, NB, causal, nrows, row_b, k, idx, cnt);
    free(k);
}

/* softmax(q.k/sqrt(d)) v over an explicit key list, one query. */
static void attend_one(const uint16_t *qi, const uint16_t *K, const uint16_t *V, int D,
                       const int32_t *keys, int nk, double *sbuf, double *o, double *lse)
{
    const double scale = 1.0 / sqrt((double)D);
    double m = -INFINITY;
    for (int t = 0; t < nk; ++t) {
        const uint16_t *kr = K + (size_t)keys[t] * D;
        double acc = 0.0;
        for (int e = 0; e < D; ++e) acc += bf(qi[e]) * bf(kr[e]);
        sbuf[t] = acc * scale;
        if (sbuf[t] > m) m = sbuf[t];
    }
    for (int e = 0; e < D; ++e) o[e] = 0.0;
    if (nk == 0) { *lse = -INFINITY; return; }
    double l = 0.0;
    for (int t = 0; t < nk; ++t) {
        const double p = exp(sbuf[t] - m);
        const uint16_t *vr = V + (size_t)keys[t] * D;
        l += p;
        for (int e = 0; e < D; ++e) o[e] += p * bf(vr[e]);
    }
    for (int e = 0; e < D; ++e) o[e] /= l;
    *lse = m + log(l);
}

/*
 * Block-sparse attention for query blocks (row_h[i], row_b[i]) restricted to
 * the key blocks idx[i][0 .. cnt[i]). o: nrows x B x D, lse: nrows x B.
 */
void oracle_sparse_attn_rows(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                             const oracle_dims *d, int B, int nrows, const int32_t *row_h,
                             const int32_t *row_b, const int32_t *idx, int NBidx,
                             const int32_t *cnt, double *o, double *lse)
{
    const int L = d->seq, D = d->head_dim;
#pragma omp parallel for schedule(dynamic, 1)
    for (int i = 0; i < nrows; ++i) {
        const int h = row_h[i], b = row_b[i], g = kv_head(d, h);
        const uint16_t *Q = q + (size_t)h * L * D;
        const uint16_t *K = k + (size_t)g * L * D;
        const uint16_t *V = v + (size_t)g * L * D;
        const int32_t *sel = idx + (size_t)i * NBidx;
        int32_t *keys = (int32_t *)malloc(sizeof(int32_t) * ((size_t)cnt[i] * B + 1));
        double *sbuf = (double *)malloc(sizeof(double) * ((size_t)cnt[i] * B + 1));
        for (int r = 0; r < B; ++r) {
            const int qi = b * B + r;
            int nk = 0;
            for (int t = 0; t < cnt[i]; ++t)
                for (int kk = sel[t] * B; kk < (sel[t] + 1) * B; ++kk)
                    if (!d->causal || kk <= qi) keys[nk++] = kk;
            attend_one(Q + (size_t)qi * D, K, V, D, keys, nk, sbuf,
                       o + ((size_t)i * B + r) * D, lse + (size_t)i * B + r);
        }
        free(keys);
        free(sbuf);
    }
}

/* Dense (full causal or full bidirectional) attention for the same rows. */
void oracle_dense_attn_rows(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                            const oracle_dims *d, int B, int nrows, const int32_t *row_h,
                            const int32_t *row_b, double *o, double *lse)
{
    const int L = d->seq, D = d->head_dim;
#pragma omp parallel for schedule(dynamic, 1)
    for (int i = 0; i < nrows; ++i) {
        const int h = row_h[i], b = row_b[i], g = kv_head(d, h);
        const uint16_t *Q = q + (size_t)h * L * D;
        const uint16_t *K = k + (size_t)g * L * D;
        const uint16_t *V = v + (size_t)g * L * D;
        int32_t *keys = (int32_t *)malloc(sizeof(int32_t) * (size_t)L);
        double *sbuf = (double *)malloc(sizeof(double) * (size_t)L);
        for (int r = 0; r < B; ++r) {
            const int qi = b * B + r;
            const int nk = d->causal ? qi + 1 : L;
            for (int kk = 0; kk < nk; ++kk) keys[kk] = kk;
            attend_one(Q + (size_t)qi * D, K, V, D, keys, nk, sbuf,
                       o + ((size_t)i * B + r) * D, lse + (size_t)i * B + r);
        }
        free(keys);
        free(sbuf);
    }
}

/*
 * Diagnostics (not used by selection): per query-block row, the exact softmax
 * mass of every key block ("true mass", rows sum to 1), and the same softmax
 * summed only over the antidiagonal positions (i mod S) + (k mod S) = S-1,
 * renormalised per row ("antidiagonal probability mass").
 */
void oracle_block_mass_rows(const uint16_t *q, const uint16_t *k, const oracle_dims *d,
                            int B, int S, int nrows, const int32_t *row_h,
                            const int32_t *row_b, double *true_mass, double *antidiag_mass)
{
    const int L = d->seq, D = d->head_dim, NB = L / B;
    const double scale = 1.0 / sqrt((double)D);
#pragma omp parallel for schedule(dynamic, 1)
    for (int i = 0; i < nrows; ++i) {
        const int h = row_h[i], b = row_b[i];
        const uint16_t *Q = q + (size_t)h * L * D;
        const uint16_t *K = k + (size_t)kv_head(d, h) * L * D;
        double *tm = true_mass + (size_t)i * NB;
        double *am = antidiag_mass + (size_t)i * NB;
        double *s = (double *)malloc(sizeof(double) * (size_t)L);
        for (int j = 0; j < NB; ++j) { tm[j] = 0.0; am[j] = 0.0; }
        for (int r = 0; r < B; ++r) {
            const int qi = b * B + r;
            const int nk = d->causal ? qi + 1 : L;
            double m = -INFINITY;
            for (int kk = 0; kk < nk; ++kk) {
                double acc = 0.0;
                for (int e = 0; e < D; ++e)
                    acc += bf(Q[(size_t)qi * D + e]) * bf(K[(size_t)kk * D + e]);
                s[kk] = acc * scale;
                if (s[kk] > m) m = s[kk];
            }
            double l = 0.0;
            for (int kk = 0; kk < nk; ++kk) l += exp(s[kk] - m);
            for (int kk = 0; kk < nk; ++kk) {
                const double p = exp(s[kk] - m) / l;
                tm[kk / B] += p;
                if ((qi % S) + (kk % S) == S - 1) am[kk / B] += p;
            }
        }
        double tot = 0.0;
        for (int j = 0; j < NB; ++j) { tm[j] /= (double)B; tot += am[j]; }
        if (tot > 0.0)
            for (int j = 0; j < NB; ++j) am[j] /= tot;
        free(s);
    }
}
