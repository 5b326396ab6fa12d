/*
 * WaveFilter CPU oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, fp64 implementation of the filter+attend path of WaveFilter
 * (arXiv 2606.00724, Section 3 and Algorithm 1), written for reading, not for
 * speed.  Only the test-suite, the package smoke check and the benchmark's CPU
 * baseline load it.  It shares no code, header, table or helper with the GPU
 * library; inputs arrive as float64 arrays that the caller upcast exactly from
 * the rounded bf16/fp32 tensors.
 *
 * Each unit (one batch element, one head) is independent.  Per unit, with
 * L prompt keys of dimension d, B query rows, J levels, S kept segments and a
 * token budget k:
 *
 *   O1  J-level 1-D DWT of every key channel along the sequence (eq. 5 with
 *       its recursion on the approximation, eq. 6).
 *   O2  skim: perception weights softmax(Q A_J^T / sqrt(d)) per query row
 *       (eq. 7) and their column sums W (eq. 8).
 *   O3  top-S coarse regions by W (eq. 9, with S given as a count).
 *   O4  regions -> token indices, region j covers tokens 2^J j .. 2^J j+2^J-1
 *       (eq. 10).
 *   O5  scan: the eq. 7-8 scoring repeated at token resolution over the pool
 *       of O4 (Section 3.2, refinement down to single tokens).
 *   O6  top-k tokens by the scan weights -> the index set mu^0.
 *   O7  sparse cache [K[mu^0]; K_g], [V[mu^0]; V_g] (Section 3.2, last
 *       paragraph; Algorithm 1, sparse-cache step).
 *   O8  attention of the query block over the sparse cache, no mask
 *       (the cached-attention form of eq. 3).
 *   R1  the paper's full multi-scale recursion (eqs. 9-11, Algorithm 1):
 *       scales B..1 with selection proportions m_b, each scale a DWT of the
 *       gathered candidate keys, then O7-O8 over the final positions.
 *
 * Readings where the paper is silent (each is also listed in the design
 * notes of the repository):
 *   - orthonormal filters: Haar g = (1, 1)/sqrt2, h = (1, -1)/sqrt2; db2 is
 *     Daubechies' 4-tap filter g = (1+r3, 3+r3, 3-r3, 1-r3)/(4 sqrt2) with
 *     h_m = (-1)^m g_{3-m};
 *   - phase: A[n] = sum_m g_m y[2n+m], so Haar coefficient j at level J
 *     covers exactly the tokens eq. 10 maps region j to;
 *   - past the right end, db2 reads a per-level half-sample symmetric
 *     extension (y[N] = y[N-1], y[N+1] = y[N-2]) or a periodic one;
 *   - eq. 8 sums over the query rows (column-wise sum), giving one weight
 *     per coarse coefficient;
 *   - ties in every top-k are broken by the lower index; index sets are
 *     returned in ascending order;
 *   - the effective token budget is min(k, S 2^J).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

/* Wavelet and boundary codes used by this file's entry points. */
#define REF_HAAR 0
#define REF_DB2 1
#define REF_SYMMETRIC 0
#define REF_PERIODIC 1

/* Analysis filters (low-pass g, high-pass h) and their length M. */
static int ref_filters(int wavelet, double g[4], double h[4]) {
    if (wavelet == REF_HAAR) {
        const double s = 1.0 / sqrt(2.0);
        g[0] = s;  g[1] = s;
        h[0] = s;  h[1] = -s;
        return 2;
    }
    if (wavelet == REF_DB2) {
        const double r3 = sqrt(3.0);
        const double den = 4.0 * sqrt(2.0);
        g[0] = (1.0 + r3) / den;
        g[1] = (3.0 + r3) / den;
        g[2] = (3.0 - r3) / den;
        g[3] = (1.0 - r3) / den;
        for (int m = 0; m < 4; ++m) {
            double sign = (m % 2 == 0) ? 1.0 : -1.0;
            h[m] = sign * g[3 - m];
        }
        return 4;
    }
    return 0;
}

/* y[i] of a length-N sequence, extended past its right end. */
static double ref_ext(const double* y, long N, long i, int boundary) {
    if (i < N) return y[i];
    if (boundary == REF_PERIODIC) return y[i % N];
    return y[2 * N - 1 - i];
}

/*
 * O1: J-level DWT of one unit's keys x [L][d] (row-major).
 * approx  [L>>J][d]                         : A_J
 * details (nullable) [sum_{j=1..J} L>>j][d] : D_1 rows, then D_2, ... D_J
 * Returns 0, or -1 on unsupported arguments.
 */
int wf_ref_dwt(const double* x, int L, int d, int levels, int wavelet,
               int boundary, double* approx, double* details) {
    double g[4], h[4];
    int M = ref_filters(wavelet, g, h);
    if (M == 0 || levels < 1 || L < 2 || (L % (1 << levels)) != 0) return -1;
    double* y = (double*)malloc(sizeof(double) * (size_t)L);
    double* a = (double*)malloc(sizeof(double) * (size_t)L);
    if (!y || !a) { free(y); free(a); return -1; }
    for (int c = 0; c < d; ++c) {
        for (int t = 0; t < L; ++t) y[t] = x[(size_t)t * d + c];
        long N = L;
        long drow = 0; /* first detail row of the current level */
        for (int j = 1; j <= levels; ++j) {
            long half = N / 2;
            for (long n = 0; n < half; ++n) {
                double sa = 0.0, sd = 0.0;
                for (int m = 0; m < M; ++m) {
                    double v = ref_ext(y, N, 2 * n + m, boundary);
                    sa += g[m] * v;
                    sd += h[m] * v;
                }
                a[n] = sa;
                if (details) details[(size_t)(drow + n) * d + c] = sd;
            }
            drow += half;
            memcpy(y, a, sizeof(double) * (size_t)half);
            N = half;
        }
        for (long n = 0; n < N; ++n) approx[(size_t)n * d + c] = y[n];
    }
    free(y);
    free(a);
    return 0;
}

/*
 * Column sums of the row-wise softmax of scale * Q X^T over the n rows of X:
 * the perception weights of eq. 7 summed over query rows as in eq. 8.
 * Q [B][d], X [n][d] -> W [n].  Logits are kept in `logit` [B][n] (scratch).
 */
static void ref_column_softmax_sum(const double* Q, const double* X, int B,
                                   long n, int d, double scale, double* W,
                                   double* logit) {
    for (long j = 0; j < n; ++j) W[j] = 0.0;
    for (int i = 0; i < B; ++i) {
        double* s = logit + (size_t)i * n;
        double mx = -INFINITY;
        for (long j = 0; j < n; ++j) {
            double acc = 0.0;
            for (int c = 0; c < d; ++c)
                acc += Q[(size_t)i * d + c] * X[(size_t)j * d + c];
            s[j] = scale * acc;
            if (s[j] > mx) mx = s[j];
        }
        double z = 0.0;
        for (long j = 0; j < n; ++j) z += exp(s[j] - mx);
        for (long j = 0; j < n; ++j) W[j] += exp(s[j] - mx) / z;
    }
}

/*
 * O2: skim weights W [n] of one unit from its coarse keys A [n][d].
 */
int wf_ref_skim(const double* Q, const double* A, int B, int n, int d,
                double scale, double* W) {
    double* logit = (double*)malloc(sizeof(double) * (size_t)B * n);
    if (!logit) return -1;
    ref_column_softmax_sum(Q, A, B, n, d, scale, W, logit);
    free(logit);
    return 0;
}

typedef struct {
    double score;
    long index;
} ref_item;

/* Higher score first; equal scores: lower index first. */
static int ref_rank_cmp(const void* pa, const void* pb) {
    const ref_item* a = (const ref_item*)pa;
    const ref_item* b = (const ref_item*)pb;
    if (a->score > b->score) return -1;
    if (a->score < b->score) return 1;
    return (a->index < b->index) ? -1 : (a->index > b->index) ? 1 : 0;
}

static int ref_index_cmp(const void* pa, const void* pb) {
    long a = *(const long*)pa, b = *(const long*)pb;
    return (a < b) ? -1 : (a > b) ? 1 : 0;
}

/*
 * O3/O6: the k best positions of score[0..n) (eq. 9), ties to the lower
 * index, written in ascending order to out[0..k).  Requires 1 <= k <= n.
 */
int wf_ref_topk(const double* score, long n, long k, long* out) {
    if (k < 1 || k > n) return -1;
    ref_item* items = (ref_item*)malloc(sizeof(ref_item) * (size_t)n);
    if (!items) return -1;
    for (long i = 0; i < n; ++i) {
        items[i].score = score[i];
        items[i].index = i;
    }
    qsort(items, (size_t)n, sizeof(ref_item), ref_rank_cmp);
    for (long i = 0; i < k; ++i) out[i] = items[i].index;
    qsort(out, (size_t)k, sizeof(long), ref_index_cmp);
    free(items);
    return 0;
}

/*
 * O4 + O5 + O6 for one unit.  seg [S] ascending region ids at level J.
 * Outputs: pool_score [S 2^J] (scan weights W' in pool order, nullable) and
 * tok [k_eff] ascending token ids, k_eff = min(k, S 2^J).
 */
int wf_ref_scan(const double* Q, const double* K, int B, int L, int d,
                int levels, const long* seg, int S, long budget, double scale,
                double* pool_score, long* tok) {
    long run = 1L << levels;
    long P = (long)S * run;
    long keff = budget < P ? budget : P;
    long* pool = (long*)malloc(sizeof(long) * (size_t)P);
    double* X = (double*)malloc(sizeof(double) * (size_t)P * d);
    double* W = (double*)malloc(sizeof(double) * (size_t)P);
    double* logit = (double*)malloc(sizeof(double) * (size_t)B * P);
    long* pick = (long*)malloc(sizeof(long) * (size_t)keff);
    int rc = -1;
    if (!pool || !X || !W || !logit || !pick) goto done;
    /* O4: eq. 10, region j -> tokens run*j + r, r < run. */
    for (int q = 0; q < S; ++q) {
        /* regions must be valid and strictly ascending, so that pool order
           is ascending token order (the tie-break of O6) */
        if (seg[q] < 0 || (seg[q] + 1) * run > L) goto done;
        if (q > 0 && seg[q] <= seg[q - 1]) goto done;
        for (long r = 0; r < run; ++r) pool[q * run + r] = seg[q] * run + r;
    }
    for (long p = 0; p < P; ++p)
        memcpy(X + (size_t)p * d, K + (size_t)pool[p] * d, sizeof(double) * d);
    /* O5: eq. 7-8 over the pool tokens. */
    ref_column_softmax_sum(Q, X, B, P, d, scale, W, logit);
    if (pool_score) memcpy(pool_score, W, sizeof(double) * (size_t)P);
    /* O6: eq. 9 over the pool; pool order is ascending token order. */
    if (wf_ref_topk(W, P, keff, pick) != 0) goto done;
    for (long i = 0; i < keff; ++i) tok[i] = pool[pick[i]];
    rc = 0;
done:
    free(pool); free(X); free(W); free(logit); free(pick);
    return rc;
}

/*
 * O7 + O8 for one unit: attention of Q [B][d] over the rows K[tok[r]]
 * (r < n_tok) followed by the G tail rows Kg [G][d], values likewise.
 * O [B][d].
 */
int wf_ref_attn(const double* Q, const double* K, const double* V,
                const long* tok, long n_tok, const double* Kg,
                const double* Vg, long G, int B, int d, double scale,
                double* O) {
    long n = n_tok + G;
    if (n < 1) return -1;
    double* Ks = (double*)malloc(sizeof(double) * (size_t)n * d);
    double* Vs = (double*)malloc(sizeof(double) * (size_t)n * d);
    double* p = (double*)malloc(sizeof(double) * (size_t)n);
    if (!Ks || !Vs || !p) { free(Ks); free(Vs); free(p); return -1; }
    /* O7: [K[mu0]; Kg], [V[mu0]; Vg]. */
    for (long r = 0; r < n_tok; ++r) {
        memcpy(Ks + (size_t)r * d, K + (size_t)tok[r] * d, sizeof(double) * d);
        memcpy(Vs + (size_t)r * d, V + (size_t)tok[r] * d, sizeof(double) * d);
    }
    for (long r = 0; r < G; ++r) {
        memcpy(Ks + (size_t)(n_tok + r) * d, Kg + (size_t)r * d, sizeof(double) * d);
        memcpy(Vs + (size_t)(n_tok + r) * d, Vg + (size_t)r * d, sizeof(double) * d);
    }
    /* O8: softmax(scale Q Ks^T) Vs, every row sees every key. */
    for (int i = 0; i < B; ++i) {
        double mx = -INFINITY;
        for (long r = 0; r < n; ++r) {
            double acc = 0.0;
            for (int c = 0; c < d; ++c)
                acc += Q[(size_t)i * d + c] * Ks[(size_t)r * d + c];
            p[r] = scale * acc;
            if (p[r] > mx) mx = p[r];
        }
        double z = 0.0;
        for (long r = 0; r < n; ++r) {
            p[r] = exp(p[r] - mx);
            z += p[r];
        }
        for (int c = 0; c < d; ++c) {
            double acc = 0.0;
            for (long r = 0; r < n; ++r) acc += p[r] * Vs[(size_t)r * d + c];
            O[(size_t)i * d + c] = acc / z;
        }
    }
    free(Ks); free(Vs); free(p);
    return 0;
}

/*
 * The whole path O1..O8 for one unit.  Every output pointer but O is
 * nullable: approx [L>>J][d], W [L>>J], seg [S], pool_score [S 2^J],
 * tok [k_eff].  When L is not a multiple of 2^J the first Lf = 2^J floor(L /
 * 2^J) positions are filtered and the last L - Lf are always kept: the
 * attention runs over [K[tok]; K[Lf..L); K_g] (tok itself holds the k_eff
 * selected positions).
 */
int wf_ref_filter_attend_unit(const double* Q, const double* K, const double* V,
                              const double* Kg, const double* Vg, int L, int d,
                              int B, int G, int levels, int wavelet,
                              int boundary, int S, long budget, double scale,
                              double* O, double* approx_out, double* W_out,
                              long* seg_out, double* pool_score_out,
                              long* tok_out) {
    /* a length that is not a multiple of 2^J: the first Lf positions are
       filtered, the last L - Lf are always kept after the selection */
    long run = 1L << levels;
    long Lf = (L / run) * run;
    long R = L - Lf;
    long n = Lf >> levels;
    long P = (long)S * run;
    long keff = budget < P ? budget : P;
    if (n < 1 || S < 1 || S > n || budget < 1) return -1;
    double* A = (double*)malloc(sizeof(double) * (size_t)n * d);
    double* W = (double*)malloc(sizeof(double) * (size_t)n);
    long* seg = (long*)malloc(sizeof(long) * (size_t)S);
    long* tok = (long*)malloc(sizeof(long) * (size_t)(keff + R));
    int rc = -1;
    if (!A || !W || !seg || !tok) goto done;
    if (wf_ref_dwt(K, (int)Lf, d, levels, wavelet, boundary, A, NULL) != 0) goto done;
    if (wf_ref_skim(Q, A, B, (int)n, d, scale, W) != 0) goto done;
    if (wf_ref_topk(W, n, S, seg) != 0) goto done;
    if (wf_ref_scan(Q, K, B, (int)Lf, d, levels, seg, S, budget, scale,
                    pool_score_out, tok) != 0) goto done;
    for (long r = 0; r < R; ++r) tok[keff + r] = Lf + r;
    if (wf_ref_attn(Q, K, V, tok, keff + R, Kg, Vg, G, B, d, scale, O) != 0) goto done;
    if (approx_out) memcpy(approx_out, A, sizeof(double) * (size_t)n * d);
    if (W_out) memcpy(W_out, W, sizeof(double) * (size_t)n);
    if (seg_out) memcpy(seg_out, seg, sizeof(long) * (size_t)S);
    if (tok_out) memcpy(tok_out, tok, sizeof(long) * (size_t)keff);
    rc = 0;
done:
    free(A); free(W); free(seg); free(tok);
    return rc;
}

/*
 * The whole path over `units` independent units, one OpenMP thread per unit
 * at a time.  Arrays are unit-major: Q [units][B][d], K/V [units][L][d],
 * Kg/Vg [units][G][d] (nullable when G == 0), O [units][B][d], tok
 * [units][k_eff] (nullable).  Returns 0 when every unit succeeded.
 */
int wf_ref_filter_attend(const double* Q, const double* K, const double* V,
                         const double* Kg, const double* Vg, int units, int L,
                         int d, int B, int G, int levels, int wavelet,
                         int boundary, int S, long budget, double scale,
                         double* O, long* tok) {
    long P = (long)S * (1L << levels);
    long keff = budget < P ? budget : P;
    int failures = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(+ : failures)
    for (int u = 0; u < units; ++u) {
        const double* kg = G ? Kg + (size_t)u * G * d : NULL;
        const double* vg = G ? Vg + (size_t)u * G * d : NULL;
        int rc = wf_ref_filter_attend_unit(
            Q + (size_t)u * B * d, K + (size_t)u * L * d, V + (size_t)u * L * d,
            kg, vg, L, d, B, G, levels, wavelet, boundary, S, budget, scale,
            O + (size_t)u * B * d, NULL, NULL, NULL, NULL,
            tok ? tok + (size_t)u * keff : NULL);  /* selected positions only */
        failures += (rc != 0);
    }
    return failures == 0 ? 0 : -1;
}

/*
 * Multi-scale recursive filtering of one unit (Section 3.2, eqs. 9-11;
 * Algorithm 1, the loop over scales) with scale B = `levels` and selection
 * proportions m_b = prop[b - 1], b = 1..B:
 *
 *   mu^B = all L prompt positions (ascending)
 *   for b = B, B-1, .., 1:
 *     C_b  = b-level DWT of the gathered keys K[mu^b], taken as one sequence
 *            (eq. 11; at b = B this is eq. 6 on the whole prompt)
 *     W    = column sums of softmax(scale Q C_b^T), softmax over C_b's rows
 *            only (eqs. 7-8 on the current candidates)
 *     J_b  = the c_b best rows of W (eq. 9), ties to the lower index,
 *            c_b = max(1, ceil(m_b n_b)) with n_b = |mu^b| / 2^b, at most n_b
 *     mu^{b-1} = { mu^b[2^b j + r] : j in J_b ascending, r < 2^b }
 *            (eq. 10, composed with mu^b so that indices stay prompt
 *            positions)
 *   tok = mu^0, ascending, 2 c_1 positions, followed by the last L mod 2^B
 *   positions when L is not a multiple of 2^B (always kept).
 *
 * counts [levels] (nullable) receives c_b at index b - 1; tok must hold
 * L entries (the largest possible mu^0); *n_tok receives |mu^0|.
 */
long wf_ref_recursion_count(double m, long n) {
    long c = (long)ceil(m * (double)n);
    if (c < 1) c = 1;
    if (c > n) c = n;
    return c;
}

int wf_ref_recursive_select(const double* Q, const double* K, int B, int L,
                            int d, int levels, int wavelet, int boundary,
                            const double* prop, double scale, long* counts,
                            long* tok, long* n_tok) {
    /* a length that is not a multiple of 2^B: the recursion runs over the
       first Lf positions; the last L - Lf are always kept after mu^0 */
    long Lr = L % (1L << levels);
    L -= (int)Lr;
    if (levels < 1 || L < (1 << levels)) return -1;
    for (int b = 1; b <= levels; ++b)
        if (!(prop[b - 1] > 0.0 && prop[b - 1] <= 1.0)) return -1;
    long* mu = (long*)malloc(sizeof(long) * (size_t)L);
    long* next = (long*)malloc(sizeof(long) * (size_t)L);
    double* X = (double*)malloc(sizeof(double) * (size_t)L * d);
    double* C = (double*)malloc(sizeof(double) * (size_t)L * d);
    double* W = (double*)malloc(sizeof(double) * (size_t)L);
    double* logit = (double*)malloc(sizeof(double) * (size_t)B * L);
    long* pick = (long*)malloc(sizeof(long) * (size_t)L);
    int rc = -1;
    if (!mu || !next || !X || !C || !W || !logit || !pick) goto done;
    long m = L; /* |mu^b| */
    for (long t = 0; t < L; ++t) mu[t] = t;
    for (int b = levels; b >= 1; --b) {
        long run = 1L << b;
        long n = m / run;
        /* eq. 11: gather, then a b-level transform of the gathered sequence */
        for (long t = 0; t < m; ++t)
            memcpy(X + (size_t)t * d, K + (size_t)mu[t] * d, sizeof(double) * d);
        if (wf_ref_dwt(X, (int)m, d, b, wavelet, boundary, C, NULL) != 0) goto done;
        /* eqs. 7-8 over the n coefficients of this scale */
        ref_column_softmax_sum(Q, C, B, n, d, scale, W, logit);
        /* eq. 9 with a proportion */
        long c = wf_ref_recursion_count(prop[b - 1], n);
        if (counts) counts[b - 1] = c;
        if (wf_ref_topk(W, n, c, pick) != 0) goto done;
        /* eq. 10 through mu^b */
        for (long i = 0; i < c; ++i)
            for (long r = 0; r < run; ++r) next[i * run + r] = mu[pick[i] * run + r];
        m = c * run;
        memcpy(mu, next, sizeof(long) * (size_t)m);
    }
    memcpy(tok, mu, sizeof(long) * (size_t)m);
    for (long r = 0; r < Lr; ++r) tok[m + r] = L + r;
    *n_tok = m + Lr;
    rc = 0;
done:
    free(mu); free(next); free(X); free(C); free(W); free(logit); free(pick);
    return rc;
}

/*
 * The recursive path for `units` units: R1 above, then O7-O8 over
 * [K[mu^0]; K_g].  Arrays as in wf_ref_filter_attend; tok [units][L]
 * (nullable) receives mu^0 in its first n_tok entries, n_tok [units]
 * (nullable) its size.
 */
int wf_ref_filter_attend_recursive(const double* Q, const double* K,
                                   const double* V, const double* Kg,
                                   const double* Vg, int units, int L, int d,
                                   int B, int G, int levels, int wavelet,
                                   int boundary, const double* prop,
                                   double scale, double* O, long* tok,
                                   long* n_tok) {
    int failures = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(+ : failures)
    for (int u = 0; u < units; ++u) {
        long* t = (long*)malloc(sizeof(long) * (size_t)L);
        long nt = 0;
        int rc = t ? wf_ref_recursive_select(Q + (size_t)u * B * d,
                                             K + (size_t)u * L * d, B, L, d,
                                             levels, wavelet, boundary, prop,
                                             scale, NULL, t, &nt)
                   : -1;
        if (rc == 0)
            rc = wf_ref_attn(Q + (size_t)u * B * d, K + (size_t)u * L * d,
                             V + (size_t)u * L * d, t, nt,
                             G ? Kg + (size_t)u * G * d : NULL,
                             G ? Vg + (size_t)u * G * d : NULL, G, B, d, scale,
                             O + (size_t)u * B * d);
        if (rc == 0 && tok) memcpy(tok + (size_t)u * L, t, sizeof(long) * (size_t)nt);
        if (rc == 0 && n_tok) n_tok[u] = nt;
        free(t);
        failures += (rc != 0);
    }
    return failures == 0 ? 0 : -1;
}

/* Threads an OpenMP parallel region of this library would use. */
int wf_ref_max_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
