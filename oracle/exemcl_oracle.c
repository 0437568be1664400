/*
 * exemcl_oracle.c -- slow, plain CPU evaluator of exemplar-based clustering.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the correctness oracle against which
 * the GPU library is checked.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may build, load or call it; the library's own
 * code path never does, and the two share no source, header or helper.
 *
 * What it computes (Buschjaeger & Morik, "GPU-Accelerated Optimizer-Aware
 * Evaluation of Submodular Exemplar Clustering"):
 *
 *   k-medoids loss, Eq. (3):  L(X) = |V|^-1 * sum_{v in V} min_{x in X} dist(v, x)
 *   exemplar clustering, Eq. (4):  f(S) = L({e0}) - L(S u {e0})
 *
 * with e0 the all-zero auxiliary vector (Eq. (4) and the sentence after it) and
 * dist the squared Euclidean distance used in all of the paper's experiments
 * (Section V).  The evaluation follows the CPU procedure of Algorithm 2: for
 * every ground point take the running minimum of the dissimilarity over the
 * candidate set, starting from the largest representable value, store it, sum
 * the stored minima, divide by |V|, and return the difference of the two
 * losses.  The union with {e0} is formed explicitly: e0 is a real zero vector
 * that is compared like any other member of the set.
 *
 * Precision: every input is an exact double (fp32/fp16/bf16 values upcast by
 * the caller), all arithmetic is IEEE double, sums run in index order.  No
 * norm expansion, no clamp form, no blocking.
 *
 * Readings where the paper is silent (each listed in the design notes):
 *   - sets are given as int32 row indices into V (S is a subset of V);
 *   - sets of different sizes share one k by padding with the index -1, an
 *     empty slot that is not a member (the blank fields of the evaluation-set
 *     matrix, Section IV-B, Memory Layout);
 *   - a set holding any other index outside [0, n) has no defined value: its
 *     result is a quiet NaN and the other sets are unaffected;
 *   - duplicate indices are allowed (the minimum is idempotent);
 *   - n = 0 is rejected (L would be 0/0).
 *
 * ORACLE_MUTANT (compile-time, default 0) plants one deliberate mistake; it
 * exists only so the test suite can show that its pins catch each mistake.
 */
#include <float.h>
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#ifndef ORACLE_MUTANT
#define ORACLE_MUTANT 0
#endif

enum { ORACLE_OK = 0, ORACLE_EINVAL = 1, ORACLE_ENOMEM = 2 };

/* Padding index of a set shorter than the batch's k. */
#define EMPTY_SLOT (-1)

/* Row i of the row-major n x d matrix V. */
static const double *row(const double *V, int64_t d, int64_t i) { return V + i * d; }

/* Squared Euclidean dissimilarity, the one used throughout Section V. */
static double dissim(const double *x, const double *y, int64_t d) {
    double s = 0.0;
    for (int64_t t = 0; t < d; ++t) {
#if ORACLE_MUTANT == 2 /* sign error inside the difference */
        double diff = x[t] + y[t];
#elif ORACLE_MUTANT == 4 /* index mix-up: coordinates paired in reverse */
        double diff = x[t] - y[d - 1 - t];
#else
        double diff = x[t] - y[t];
#endif
        s += diff * diff;
    }
#if ORACLE_MUTANT == 8 /* plain (not squared) Euclidean distance */
    s = sqrt(s);
#endif
    return s;
}

/*
 * L(X) of Eq. (3) for X = {members of `idx`} u {e0}, computed as in
 * Algorithm 2's function L: per point a running minimum started at the
 * largest double, a stored minimum per point, then the sum and the division
 * by |V|.  e0 is compared first, then the indexed members in slot order;
 * empty slots (-1) are skipped.  Returns NaN when another index is out of
 * range.
 */
static double loss(const double *V, int64_t n, int64_t d, const double *e0, const int32_t *idx,
                   int64_t k, double *scratch) {
    for (int64_t p = 0; p < k; ++p)
        if (idx[p] != EMPTY_SLOT && (idx[p] < 0 || (int64_t)idx[p] >= n)) return NAN;

    for (int64_t i = 0; i < n; ++i) {
        const double *v = row(V, d, i);
#if ORACLE_MUTANT == 1 /* e0 left out of the minimum */
        double t = DBL_MAX;
        (void)e0;
#else
        double t = DBL_MAX;
        {
            double de = dissim(v, e0, d); /* the auxiliary member e0 */
#if ORACLE_MUTANT == 7          /* maximum instead of minimum */
            t = de;
#else
            t = fmin(t, de);
#endif
        }
#endif
#if ORACLE_MUTANT == 5 /* last member of the set skipped */
        for (int64_t p = 0; p + 1 < k; ++p) {
#else
        for (int64_t p = 0; p < k; ++p) {
#endif
            if (idx[p] == EMPTY_SLOT) continue; /* a blank field: no member */
            double ds = dissim(v, row(V, d, idx[p]), d);
#if ORACLE_MUTANT == 7
            t = fmax(t, ds);
#else
            t = fmin(t, ds);
#endif
        }
#if ORACLE_MUTANT == 1
        if (k == 0) t = 0.0; /* keeps the mutant finite on the empty set */
#endif
        scratch[i] = t;
    }
    double sigma = 0.0; /* "reduce by sum", in index order */
    for (int64_t i = 0; i < n; ++i) sigma += scratch[i];
#if ORACLE_MUTANT == 3 /* wrong normaliser */
    return sigma / (double)(n > 1 ? n - 1 : 1);
#else
    return sigma / (double)n;
#endif
}

/* L({e0}) of Eq. (4): mean squared distance of the ground set to e0. */
static double loss_e0(const double *V, int64_t n, int64_t d, const double *e0, double *scratch) {
    double sigma = 0.0;
    for (int64_t i = 0; i < n; ++i) scratch[i] = dissim(row(V, d, i), e0, d);
    for (int64_t i = 0; i < n; ++i) sigma += scratch[i];
#if ORACLE_MUTANT == 3
    return sigma / (double)(n > 1 ? n - 1 : 1);
#else
    return sigma / (double)n;
#endif
}

static int check_args(const double *V, int64_t n, int64_t d, const void *sets, int64_t l,
                      int64_t k, const double *out) {
    if (n <= 0 || d <= 0 || k < 0 || l < 0) return ORACLE_EINVAL;
    if (!V) return ORACLE_EINVAL;
    if (l > 0 && !out) return ORACLE_EINVAL;
    if (l > 0 && k > 0 && !sets) return ORACLE_EINVAL;
    return ORACLE_OK;
}

static int set_threads(int nthreads) {
#ifdef _OPENMP
    return nthreads > 0 ? nthreads : omp_get_max_threads();
#else
    (void)nthreads;
    return 1;
#endif
}

/* L({e0}) for V (n x d, row-major, doubles). */
double oracle_loss_e0(const double *V, int64_t n, int64_t d) {
    if (!V || n <= 0 || d <= 0) return NAN;
    double *e0 = (double *)calloc((size_t)d, sizeof(double));
    double *scratch = (double *)malloc((size_t)n * sizeof(double));
    double r = NAN;
    if (e0 && scratch) r = loss_e0(V, n, d, e0, scratch);
    free(e0);
    free(scratch);
    return r;
}

/*
 * f(S_j) of Eq. (4) for l sets of k indices each (row-major l x k int32).
 * out[j] receives f(S_j).  nthreads = 1 is the single-thread evaluator; more
 * threads evaluate different sets in parallel, the paper's multi-thread
 * baseline (Section V).  Each set's arithmetic is the same either way, so the
 * results are bitwise identical for any thread count.
 */
int oracle_eval(const double *V, int64_t n, int64_t d, const int32_t *sets, int64_t l, int64_t k,
                double *out, int nthreads) {
    int rc = check_args(V, n, d, sets, l, k, out);
    if (rc) return rc;
    if (l == 0) return ORACLE_OK;
    double *e0 = (double *)calloc((size_t)d, sizeof(double));
    double *s0 = (double *)malloc((size_t)n * sizeof(double));
    if (!e0 || !s0) {
        free(e0);
        free(s0);
        return ORACLE_ENOMEM;
    }
    const double le0 = loss_e0(V, n, d, e0, s0);
    free(s0);
    int nt = set_threads(nthreads);
    int failed = 0;
#pragma omp parallel num_threads(nt) reduction(| : failed)
    {
        double *scratch = (double *)malloc((size_t)n * sizeof(double));
        if (!scratch) failed = 1;
#pragma omp for schedule(static)
        for (int64_t j = 0; j < l; ++j) {
            if (!scratch) continue;
            double ls = loss(V, n, d, e0, sets + j * k, k, scratch);
#if ORACLE_MUTANT == 6 /* difference taken the wrong way round */
            out[j] = ls - le0;
#else
            out[j] = le0 - ls;
#endif
        }
        free(scratch);
    }
    free(e0);
    return failed ? ORACLE_ENOMEM : ORACLE_OK;
}

/*
 * Greedy-step scoring: out[j] = f(S u {cands[j]}) for a base set S of k
 * indices and l candidate indices.  This is the multiset the Greedy optimizer
 * (Algorithm 1) builds in every round (Section IV-A); each member is evaluated
 * directly by the definition, with no cached state.
 */
int oracle_gain(const double *V, int64_t n, int64_t d, const int32_t *S, int64_t k,
                const int32_t *cands, int64_t l, double *out, int nthreads) {
    if (k < 0 || (k > 0 && !S) || (l > 0 && !cands)) return ORACLE_EINVAL;
    int rc = check_args(V, n, d, cands, l, k, out);
    if (rc) return rc;
    if (l == 0) return ORACLE_OK;
    const int64_t kk = k + 1;
    int32_t *sets = (int32_t *)malloc((size_t)(l * kk) * sizeof(int32_t));
    if (!sets) return ORACLE_ENOMEM;
    for (int64_t j = 0; j < l; ++j) {
        if (k > 0) memcpy(sets + j * kk, S, (size_t)k * sizeof(int32_t));
        sets[j * kk + k] = cands[j];
    }
    rc = oracle_eval(V, n, d, sets, l, kk, out, nthreads);
    free(sets);
    return rc;
}

/* q_i = ||v_i||^2, the squared distance of each ground point to e0. */
int oracle_sqnorm(const double *V, int64_t n, int64_t d, double *q) {
    if (!V || !q || n <= 0 || d <= 0) return ORACLE_EINVAL;
    double *e0 = (double *)calloc((size_t)d, sizeof(double));
    if (!e0) return ORACLE_ENOMEM;
    for (int64_t i = 0; i < n; ++i) q[i] = dissim(row(V, d, i), e0, d);
    free(e0);
    return ORACLE_OK;
}

/* Number of OpenMP threads an nthreads request resolves to. */
int oracle_threads(int nthreads) { return set_threads(nthreads); }

/*
 * The Greedy optimizer of Algorithm 1 on f: K rounds, each adding the point
 * e in V \ S with the largest f(S u {e}) (equivalently the largest discrete
 * derivative of Definition 1), evaluated directly by the definition.  Ties go
 * to the lowest index (the paper leaves the tie-break open).  S_out[i] is the
 * point added in round i, f_out[i] = f(S_i).
 */
int oracle_greedy(const double *V, int64_t n, int64_t d, int64_t K, int32_t *S_out, double *f_out,
                  int nthreads) {
    if (!V || n <= 0 || d <= 0 || K < 0 || K > n) return ORACLE_EINVAL;
    if (K > 0 && (!S_out || !f_out)) return ORACLE_EINVAL;
    int32_t *cands = (int32_t *)malloc((size_t)n * sizeof(int32_t));
    double *score = (double *)malloc((size_t)n * sizeof(double));
    char *taken = (char *)calloc((size_t)n, 1);
    int rc = ORACLE_OK;
    if (!cands || !score || !taken) rc = ORACLE_ENOMEM;
    for (int64_t i = 0; rc == ORACLE_OK && i < K; ++i) {
        int64_t m = 0;
        for (int64_t c = 0; c < n; ++c)
            if (!taken[c]) cands[m++] = (int32_t)c;
        rc = oracle_gain(V, n, d, S_out, i, cands, m, score, nthreads);
        if (rc) break;
        int64_t best = 0;
        for (int64_t q = 1; q < m; ++q)
            if (score[q] > score[best]) best = q; /* strict: the lowest index wins ties */
        S_out[i] = cands[best];
        f_out[i] = score[best];
        taken[cands[best]] = 1;
    }
    free(cands);
    free(score);
    free(taken);
    return rc;
}
