/*
 * Driver for running the CPU oracle (oracle/wf_oracle.c) under AddressSanitizer
 * and UndefinedBehaviorSanitizer.  Test infrastructure: the test that builds
 * it links it with the oracle source, nothing else.
 *
 * It calls every entry point of the oracle on small seeded inputs that reach
 * its boundary paths (db2 symmetric and periodic ends, a length that is not a
 * multiple of 2^J, a generation tail, exact ties, keep-all selections, several
 * units in the OpenMP loop) and checks each result against a fact fixed by
 * the mathematics, computed here independently:
 *   - Haar closed form: A_J[j] = 2^{-J/2} times the sum of block j;
 *   - Parseval for orthonormal filter banks (Haar, db2 periodic);
 *   - top-k against a brute-force rank count with injected ties;
 *   - keep-all selection equals dense softmax attention;
 *   - the recursion with every proportion 1 keeps every position;
 *   - the OpenMP batch equals per-unit calls.
 * Exit status 0 when every check holds; a sanitizer report aborts.
 */
#include <math.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int wf_ref_dwt(const double* x, int L, int d, int levels, int wavelet,
               int boundary, double* approx, double* details);
int wf_ref_skim(const double* Q, const double* A, int B, int n, int d,
                double scale, double* W);
int wf_ref_topk(const double* score, long n, long k, long* out);
int wf_ref_scan(const double* Q, const double* K, int B, int L, int d,
                int levels, const long* seg, int S, long budget, double scale,
                double* pool_score, long* tok);
int wf_ref_attn(const double* Q, const double* K, const double* V,
                const long* tok, long n_tok, const double* Kg,
                const double* Vg, long G, int B, int d, double scale,
                double* O);
int wf_ref_filter_attend_unit(const double* Q, const double* K, const double* V,
                              const double* Kg, const double* Vg, int L, int d,
                              int B, int G, int levels, int wavelet,
                              int boundary, int S, long budget, double scale,
                              double* O, double* approx_out, double* W_out,
                              long* seg_out, double* pool_score_out,
                              long* tok_out);
int wf_ref_filter_attend(const double* Q, const double* K, const double* V,
                         const double* Kg, const double* Vg, int units, int L,
                         int d, int B, int G, int levels, int wavelet,
                         int boundary, int S, long budget, double scale,
                         double* O, long* tok);
long wf_ref_recursion_count(double m, long n);
int wf_ref_recursive_select(const double* Q, const double* K, int B, int L,
                            int d, int levels, int wavelet, int boundary,
                            const double* prop, double scale, long* counts,
                            long* tok, long* n_tok);
int wf_ref_filter_attend_recursive(const double* Q, const double* K,
                                   const double* V, const double* Kg,
                                   const double* Vg, int units, int L, int d,
                                   int B, int G, int levels, int wavelet,
                                   int boundary, const double* prop,
                                   double scale, double* O, long* tok,
                                   long* n_tok);

static int failures = 0;

#define EXPECT(cond, ...)                  \
    do {                                   \
        if (!(cond)) {                     \
            fprintf(stderr, "FAIL: ");     \
            fprintf(stderr, __VA_ARGS__);  \
            fprintf(stderr, "\n");         \
            ++failures;                    \
        }                                  \
    } while (0)

/* xorshift64* uniform in [-1, 1) */
static unsigned long long rng_state = 88172645463325252ULL;
static double urand(void) {
    rng_state ^= rng_state >> 12;
    rng_state ^= rng_state << 25;
    rng_state ^= rng_state >> 27;
    unsigned long long r = rng_state * 2685821657736338717ULL;
    return (double)(r >> 11) / 9007199254740992.0 * 2.0 - 1.0;
}

static double* rnd(size_t n) {
    double* p = (double*)malloc(sizeof(double) * n);
    for (size_t i = 0; i < n; ++i) p[i] = urand();
    return p;
}

static void check_dwt(void) {
    const int L = 96, d = 3, J = 3;
    double* x = rnd((size_t)L * d);
    double A[(96 >> 3) * 3], D[(48 + 24 + 12) * 3];
    /* Haar closed form */
    EXPECT(wf_ref_dwt(x, L, d, J, 0, 0, A, D) == 0, "haar dwt rejected");
    for (int j = 0; j < (L >> J); ++j)
        for (int c = 0; c < d; ++c) {
            double s = 0.0;
            for (int t = 0; t < (1 << J); ++t) s += x[(size_t)(j * 8 + t) * d + c];
            EXPECT(fabs(A[j * d + c] - s / sqrt(8.0)) < 1e-12, "haar closed form");
        }
    /* Parseval: Haar and db2 periodic (orthonormal analysis) */
    for (int wav = 0; wav < 2; ++wav) {
        int bnd = wav == 0 ? 0 : 1;
        EXPECT(wf_ref_dwt(x, L, d, J, wav, bnd, A, D) == 0, "dwt rejected");
        for (int c = 0; c < d; ++c) {
            double ex = 0.0, ec = 0.0;
            for (int t = 0; t < L; ++t) ex += x[(size_t)t * d + c] * x[(size_t)t * d + c];
            for (int j = 0; j < (L >> J); ++j) ec += A[j * d + c] * A[j * d + c];
            for (int r = 0; r < 48 + 24 + 12; ++r) ec += D[r * d + c] * D[r * d + c];
            EXPECT(fabs(ex - ec) < 1e-10 * ex, "parseval wavelet %d", wav);
        }
    }
    /* db2 symmetric: run for memory safety at the right end, details on */
    EXPECT(wf_ref_dwt(x, L, d, J, 1, 0, A, D) == 0, "db2 symmetric rejected");
    EXPECT(wf_ref_dwt(x, L + 1, d, J, 0, 0, A, D) != 0, "odd length accepted");
    free(x);
}

static void check_topk(void) {
    const long n = 40;
    double s[40];
    for (long i = 0; i < n; ++i) s[i] = floor(urand() * 4.0);  /* many exact ties */
    for (long k = 1; k <= n; k += 7) {
        long out[40];
        EXPECT(wf_ref_topk(s, n, k, out) == 0, "topk rejected");
        int picked[40] = {0};
        for (long i = 0; i < k; ++i) picked[out[i]] = 1;
        for (long i = 1; i < k; ++i) EXPECT(out[i] > out[i - 1], "topk order");
        for (long i = 0; i < n; ++i) {
            long rank = 0; /* items strictly before i in (score desc, index asc) */
            for (long j = 0; j < n; ++j)
                if (s[j] > s[i] || (s[j] == s[i] && j < i)) ++rank;
            EXPECT(picked[i] == (rank < k), "topk brute force i=%ld k=%ld", i, k);
        }
    }
    EXPECT(wf_ref_topk(s, n, 0, NULL) != 0, "k = 0 accepted");
}

/* dense softmax attention of Q over the first n rows of K, V plus a tail */
static void dense_attn(const double* Q, const double* K, const double* V, long n,
                       const double* Kg, const double* Vg, long G, int B, int d,
                       double* O) {
    double* p = (double*)malloc(sizeof(double) * (size_t)(n + G));
    for (int i = 0; i < B; ++i) {
        double mx = -INFINITY;
        for (long r = 0; r < n + G; ++r) {
            const double* k = r < n ? K + (size_t)r * d : Kg + (size_t)(r - n) * d;
            double a = 0.0;
            for (int c = 0; c < d; ++c) a += Q[i * d + c] * k[c];
            p[r] = a / sqrt((double)d);
            if (p[r] > mx) mx = p[r];
        }
        double z = 0.0;
        for (long r = 0; r < n + G; ++r) z += (p[r] = exp(p[r] - mx));
        for (int c = 0; c < d; ++c) {
            double a = 0.0;
            for (long r = 0; r < n + G; ++r)
                a += p[r] * (r < n ? V[(size_t)r * d + c] : Vg[(size_t)(r - n) * d + c]);
            O[i * d + c] = a / z;
        }
    }
    free(p);
}

static void check_keep_all(void) {
    const int d = 4, B = 5, G = 3;
    const int lens[2] = {64, 64 + 3}; /* the second is not a multiple of 2^J */
    for (int wav = 0; wav < 2; ++wav)
        for (int li = 0; li < 2; ++li) {
            const int L = lens[li], J = 2, n = 64 >> J;
            double* Q = rnd((size_t)B * d);
            double* K = rnd((size_t)L * d);
            double* V = rnd((size_t)L * d);
            double* Kg = rnd((size_t)G * d);
            double* Vg = rnd((size_t)G * d);
            double O[5 * 4], R[5 * 4], A[16 * 4], W[16], Wp[64];
            long seg[16], tok[64];
            int rc = wf_ref_filter_attend_unit(Q, K, V, Kg, Vg, L, d, B, G, J, wav,
                                               0, n, 1 << 20, 1.0 / sqrt((double)d), O,
                                               A, W, seg, Wp, tok);
            EXPECT(rc == 0, "keep-all rejected");
            dense_attn(Q, K, V, L, Kg, Vg, G, B, d, R);
            for (int i = 0; i < B * d; ++i)
                EXPECT(fabs(O[i] - R[i]) < 1e-12, "keep-all != dense (wavelet %d L %d)", wav, L);
            for (int t = 0; t < 64; ++t) EXPECT(tok[t] == t, "keep-all tokens");
            double sw = 0.0;
            for (int j = 0; j < n; ++j) sw += W[j];
            EXPECT(fabs(sw - B) < 1e-12, "sum of W is B");
            free(Q); free(K); free(V); free(Kg); free(Vg);
        }
}

static void check_batch_and_recursion(void) {
    const int U = 3, L = 128 + 3, d = 4, B = 6, G = 2, J = 3;
    const double sc = 1.0 / sqrt((double)d);
    double* Q = rnd((size_t)U * B * d);
    double* K = rnd((size_t)U * L * d);
    double* V = rnd((size_t)U * L * d);
    double* Kg = rnd((size_t)U * G * d);
    double* Vg = rnd((size_t)U * G * d);
    double O[3 * 6 * 4], O1[6 * 4];
    long tok[3 * 20], tok1[20];
    for (int wav = 0; wav < 2; ++wav) {
        EXPECT(wf_ref_filter_attend(Q, K, V, Kg, Vg, U, L, d, B, G, J, wav, 0, 4, 20,
                                    sc, O, tok) == 0, "batch rejected");
        for (int u = 0; u < U; ++u) {
            wf_ref_filter_attend_unit(Q + (size_t)u * B * d, K + (size_t)u * L * d,
                                      V + (size_t)u * L * d, Kg + (size_t)u * G * d,
                                      Vg + (size_t)u * G * d, L, d, B, G, J, wav, 0, 4,
                                      20, sc, O1, NULL, NULL, NULL, NULL, tok1);
            EXPECT(memcmp(O1, O + (size_t)u * B * d, sizeof(O1)) == 0, "batch O unit %d", u);
            EXPECT(memcmp(tok1, tok + (size_t)u * 20, sizeof(tok1)) == 0, "batch tok unit %d", u);
        }
    }
    /* scan on given regions, then attention on given tokens */
    long seg[2] = {1, 7}, stok[10];
    double Wp[16];
    EXPECT(wf_ref_scan(Q, K, B, 128, d, J, seg, 2, 10, sc, Wp, stok) == 0, "scan rejected");
    for (int i = 0; i < 10; ++i) EXPECT((stok[i] >> J) == 1 || (stok[i] >> J) == 7, "scan pool");
    long bad[2] = {7, 1};
    EXPECT(wf_ref_scan(Q, K, B, 128, d, J, bad, 2, 10, sc, Wp, stok) != 0, "unsorted regions");
    double Oa[6 * 4];
    EXPECT(wf_ref_attn(Q, K, V, stok, 10, Kg, Vg, G, B, d, sc, Oa) == 0, "attn rejected");
    double Ws[16], Aj[16 * 4];
    EXPECT(wf_ref_dwt(K, 128, d, J, 0, 0, Aj, NULL) == 0 &&
           wf_ref_skim(Q, Aj, B, 16, d, sc, Ws) == 0, "skim rejected");
    /* recursion: every proportion 1 keeps every filtered position */
    double ones[3] = {1.0, 1.0, 1.0}, half[3] = {0.5, 0.5, 0.25};
    long counts[3], rt[3 * 131], nt[3];
    for (int wav = 0; wav < 2; ++wav)
        for (int bnd = 0; bnd < 2; ++bnd) {
            long n_tok = 0;
            EXPECT(wf_ref_recursive_select(Q, K, B, L, d, J, wav, bnd, ones, sc, counts, rt,
                                           &n_tok) == 0, "recursion rejected");
            EXPECT(n_tok == L, "keep-all recursion size %ld", n_tok);
            for (long t = 0; t < n_tok; ++t) EXPECT(rt[t] == t, "keep-all recursion order");
            EXPECT(wf_ref_filter_attend_recursive(Q, K, V, Kg, Vg, U, L, d, B, G, J, wav, bnd,
                                                  half, sc, O, rt, nt) == 0,
                   "recursive batch rejected");
            for (int u = 0; u < U; ++u)
                EXPECT(nt[u] == 2 * wf_ref_recursion_count(0.5, 2 * wf_ref_recursion_count(
                                    0.5, 2 * wf_ref_recursion_count(0.25, 128 >> 3))) + 3,
                       "recursion size");
        }
    free(Q); free(K); free(V); free(Kg); free(Vg);
}

int main(void) {
    check_dwt();
    check_topk();
    check_keep_all();
    check_batch_and_recursion();
    if (failures) {
        fprintf(stderr, "%d checks failed\n", failures);
        return 1;
    }
    printf("oracle sanitizer driver: all checks hold\n");
    return 0;
}
