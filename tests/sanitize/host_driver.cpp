// Drives the C ABI's host-side paths that run before any device call --
// argument validation, the plan query, status strings, the profiling hook
// with nothing recorded -- over ordinary and extreme sizes; built with the
// library's host code under AddressSanitizer and UndefinedBehaviorSanitizer
// by tests/test_sanitizers.py (no GPU needed).  Exit status 0 = every
// check held.
#include <stdint.h>
#include <stdio.h>

#include "exemcl.h"

static int failures = 0;
static void expect(bool ok, const char *what) {
    if (!ok) {
        fprintf(stderr, "FAILED: %s\n", what);
        ++failures;
    }
}

int main() {
    void *fake = (void *)0x1000;  // never dereferenced: every call below stops before using it
    const int32_t *fs = (const int32_t *)fake;
    float *fo = (float *)fake;
    // exemplar_eval / _noalloc / _streamed: each bad argument alone
    struct Case { const void *V; int64_t n, d; const int32_t *sets; int64_t l, k; int prec; float *out; };
    const Case bad[] = {
        {nullptr, 100, 8, fs, 4, 3, 0, fo}, {fake, 0, 8, fs, 4, 3, 0, fo}, {fake, -3, 8, fs, 4, 3, 0, fo},
        {fake, INT64_C(1) << 31, 8, fs, 4, 3, 0, fo}, {fake, 100, 0, fs, 4, 3, 0, fo},
        {fake, 100, (INT64_C(1) << 24) + 1, fs, 4, 3, 0, fo}, {fake, 100, INT64_MAX, fs, 4, 3, 0, fo},
        {fake, 100, 8, fs, 4, -1, 0, fo}, {fake, 100, 8, fs, -1, 3, 0, fo}, {fake, 100, 8, fs, 4, 3, 3, fo},
        {fake, 100, 8, fs, 4, 3, -1, fo}, {fake, 100, 8, nullptr, 4, 3, 0, fo}, {fake, 100, 8, fs, 4, 3, 0, nullptr},
    };
    for (const Case &c : bad) {
        expect(exemplar_eval(c.V, c.n, c.d, c.sets, c.l, c.k, c.prec, c.out, nullptr) == EXEMCL_EINVAL, "eval EINVAL");
        expect(exemplar_eval_noalloc(c.V, c.n, c.d, c.sets, c.l, c.k, c.prec, c.out, nullptr) == EXEMCL_EINVAL,
               "noalloc EINVAL");
        expect(exemplar_eval_streamed(c.V, c.n, c.d, c.sets, c.l, c.k, c.prec, 0, c.out, nullptr) == EXEMCL_EINVAL,
               "streamed EINVAL");
    }
    expect(exemplar_eval(fake, 100, 8, nullptr, 0, 3, 0, nullptr, nullptr) == EXEMCL_OK, "l = 0 is a no-op");
    expect(exemplar_eval_streamed(fake, 100, 8, fs, 4, 3, 0, -1, fo, nullptr) == EXEMCL_EINVAL, "rows_per_block < 0");
    const float *fv = (const float *)fake;
    expect(exemplar_gain(nullptr, 100, 8, fs, 3, fs, 4, fo, nullptr) == EXEMCL_EINVAL, "gain NULL V");
    expect(exemplar_gain(fv, 100, 8, nullptr, 3, fs, 4, fo, nullptr) == EXEMCL_EINVAL, "gain NULL S");
    expect(exemplar_gain(fv, 100, 8, fs, 3, nullptr, 4, fo, nullptr) == EXEMCL_EINVAL, "gain NULL cands");
    expect(exemplar_gain(fv, 100, 8, fs, -1, fs, 4, fo, nullptr) == EXEMCL_EINVAL, "gain k < 0");
    int32_t *fi = (int32_t *)fake;
    expect(exemplar_greedy(fv, 100, 8, 101, fi, fo, nullptr) == EXEMCL_EINVAL, "greedy K > n");
    expect(exemplar_greedy(fv, 100, 8, 5, nullptr, fo, nullptr) == EXEMCL_EINVAL, "greedy NULL S_out");
    expect(exemplar_greedy(fv, 100, 8, 0, nullptr, nullptr, nullptr) == EXEMCL_OK, "greedy K = 0");
    expect(exemplar_sqnorm(nullptr, 10, 2, 0, fo, nullptr) == EXEMCL_EINVAL, "sqnorm NULL V");
    expect(exemplar_sqnorm(fake, 10, 2, 7, fo, nullptr) == EXEMCL_EINVAL, "sqnorm precision");
    // the plan query over ordinary and extreme sizes (host only)
    const int64_t ns[] = {1, 999, 1000000, INT32_MAX};
    const int64_t ds[] = {1, 2, 7, 8, 16, 17, 100, 192, 256, 512, 513, 1024, 1025, 4100, INT64_C(1) << 24};
    const int64_t ls[] = {0, 1, 33, 4096, 1000000};
    const int64_t ks[] = {0, 1, 10, 500};
    for (int64_t n : ns)
        for (int64_t d : ds)
            for (int64_t l : ls)
                for (int64_t k : ks)
                    for (int prec = 0; prec < 3; ++prec) {
                        int path = -1;
                        int64_t ws = -1;
                        expect(exemplar_plan(n, d, l, k, prec, &path, &ws) == EXEMCL_OK && ws >= 0 && path >= 0,
                               "plan");
                    }
    expect(exemplar_plan(10, (INT64_C(1) << 24) + 1, 4, 3, 0, nullptr, nullptr) == EXEMCL_EINVAL, "plan d limit");
    expect(exemplar_plan(10, 8, 4, 3, 9, nullptr, nullptr) == EXEMCL_EINVAL, "plan precision");
    for (int st = -1; st < 8; ++st) expect(exemplar_strerror(st) != nullptr, "strerror");
    expect(exemplar_version() >= 100, "version");
    expect(exemplar_prof_enable(-1) == EXEMCL_EINVAL, "prof_enable < 0");
    double ms = -1.0;
    int64_t launches = -1;
    expect(exemplar_prof_read(&ms, &launches) == EXEMCL_OK && ms == 0.0 && launches == 0, "prof_read empty");
    if (failures) fprintf(stderr, "%d checks failed\n", failures);
    else printf("host checks passed\n");
    return failures ? 1 : 0;
}
