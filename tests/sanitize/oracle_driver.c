/* Drives the CPU oracle (oracle/exemcl_oracle.c) through every entry point
 * on hand-worked ground sets and small random ones; built and run under
 * AddressSanitizer and UndefinedBehaviorSanitizer by
 * tests/test_sanitizers.py.  Exit status 0 = every check held. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

int oracle_eval(const double *V, int64_t n, int64_t d, const int32_t *sets, int64_t l, int64_t k, double *out,
                int nthreads);
int oracle_gain(const double *V, int64_t n, int64_t d, const int32_t *S, int64_t k, const int32_t *cands,
                int64_t l, double *out, int nthreads);
int oracle_sqnorm(const double *V, int64_t n, int64_t d, double *q);
double oracle_loss_e0(const double *V, int64_t n, int64_t d);
int oracle_greedy(const double *V, int64_t n, int64_t d, int64_t K, int32_t *S_out, double *f_out, int nthreads);

static int failures = 0;
static void expect(int ok, const char *what) {
    if (!ok) {
        fprintf(stderr, "FAILED: %s\n", what);
        ++failures;
    }
}
/* x equals num/3 (the worked examples' values are thirds) */
static int thirds(double x, double num) { return fabs(3.0 * x - num) <= 1e-12 * (1.0 + fabs(num)); }

int main(void) {
    /* V = {1, 2, 3}: L({e0}) = 14/3; f({1}) = 3, f({2}) = f({3}) = 4, pairs 13/3, V 14/3. */
    const double A[3] = {1.0, 2.0, 3.0};
    expect(thirds(oracle_loss_e0(A, 3, 1), 14.0), "L({e0}) of {1,2,3}");
    const int32_t sa[8 * 3] = {0, -1, -1, 1, -1, -1, 2, -1, -1, 0, 1, -1, 0, 2, -1, 1, 2, -1, 0, 1, 2, -1, -1, -1};
    const double wa[8] = {9.0, 12.0, 12.0, 13.0, 13.0, 13.0, 14.0, 0.0};
    double out[8];
    expect(oracle_eval(A, 3, 1, sa, 8, 3, out, 1) == 0, "eval status");
    for (int j = 0; j < 8; ++j) expect(thirds(out[j], wa[j]), "worked example {1,2,3}");
    /* V = {-1, 0, 2}: L({e0}) = 5/3; {-1} 1/3, {0} 0, {2} 4/3, {-1,0} 1/3, {-1,2} 5/3, {0,2} 4/3. */
    const double B[3] = {-1.0, 0.0, 2.0};
    const int32_t sb[6 * 2] = {0, 0, 1, 1, 2, 2, 0, 1, 0, 2, 1, 2};
    const double wb[6] = {1.0, 0.0, 4.0, 1.0, 5.0, 4.0};
    expect(oracle_eval(B, 3, 1, sb, 6, 2, out, 4) == 0, "eval status (4 threads)");
    for (int j = 0; j < 6; ++j) expect(thirds(out[j], wb[j]), "worked example {-1,0,2}");
    /* an index outside [0, n) makes its own set NaN, and only it */
    const int32_t bad[2 * 2] = {0, 3, 1, 2};
    expect(oracle_eval(A, 3, 1, bad, 2, 2, out, 1) == 0 && isnan(out[0]) && thirds(out[1], 13.0), "invalid index");
    /* k = 0: f(empty) = 0 */
    expect(oracle_eval(A, 3, 1, NULL, 2, 0, out, 1) == 0 && out[0] == 0.0 && out[1] == 0.0, "empty sets");
    /* greedy step scoring against S = {2}: candidates 1 and 3 tie at 13/3 */
    const int32_t S[1] = {1}, c[2] = {0, 2};
    expect(oracle_gain(A, 3, 1, S, 1, c, 2, out, 2) == 0 && thirds(out[0], 13.0) && thirds(out[1], 13.0), "gain");
    /* Algorithm 1 on {1,2,3}: 2, then 1 (tie with 3, lowest index), then 3 */
    int32_t gS[3];
    double gf[3];
    expect(oracle_greedy(A, 3, 1, 3, gS, gf, 1) == 0, "greedy status");
    expect(gS[0] == 1 && gS[1] == 0 && gS[2] == 2, "greedy picks");
    expect(thirds(gf[0], 12.0) && thirds(gf[1], 13.0) && thirds(gf[2], 14.0), "greedy values");
    double q[3];
    expect(oracle_sqnorm(A, 3, 1, q) == 0 && q[0] == 1.0 && q[1] == 4.0 && q[2] == 9.0, "sqnorm");
    /* argument checks */
    expect(oracle_eval(NULL, 3, 1, sa, 1, 1, out, 1) != 0, "NULL V");
    expect(oracle_eval(A, 0, 1, sa, 1, 1, out, 1) != 0, "n = 0");
    expect(oracle_greedy(A, 3, 1, 4, gS, gf, 1) != 0, "K > n");

    /* random ground set: gain equals eval of S u {c}; 1 and 7 threads agree bit for bit */
    enum { n = 57, d = 7, l = 11, k = 4 };
    double *V = malloc(sizeof(double) * n * d);
    int32_t *sets = malloc(sizeof(int32_t) * l * (k + 1)), *cand = malloc(sizeof(int32_t) * l);
    double *o1 = malloc(sizeof(double) * l), *o7 = malloc(sizeof(double) * l), *og = malloc(sizeof(double) * l);
    if (!V || !sets || !cand || !o1 || !o7 || !og) return 2;
    uint64_t x = 88172645463325252ull;
    for (int i = 0; i < n * d; ++i) {
        x ^= x << 13, x ^= x >> 7, x ^= x << 17;
        V[i] = (double)(x >> 11) * 0x1.0p-53 * 4.0 - 2.0;
    }
    const int32_t base[k] = {3, 17, 40, 56};
    for (int j = 0; j < l; ++j) {
        for (int p = 0; p < k; ++p) sets[j * (k + 1) + p] = base[p];
        cand[j] = (int32_t)((j * 5 + 1) % n);
        sets[j * (k + 1) + k] = cand[j];
    }
    expect(oracle_eval(V, n, d, sets, l, k + 1, o1, 1) == 0 && oracle_eval(V, n, d, sets, l, k + 1, o7, 7) == 0,
           "random eval status");
    expect(oracle_gain(V, n, d, base, k, cand, l, og, 3) == 0, "random gain status");
    for (int j = 0; j < l; ++j) {
        expect(o1[j] == o7[j], "threads agree bitwise");
        expect(og[j] == o1[j], "gain equals eval of S u {c}");
    }
    free(V), free(sets), free(cand), free(o1), free(o7), free(og);
    if (failures) fprintf(stderr, "%d checks failed\n", failures);
    else printf("oracle checks passed\n");
    return failures ? 1 : 0;
}
