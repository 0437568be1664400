/*
 * exemcl.h -- C ABI of the MI355X exemplar-clustering evaluator.
 *
 * The library scores sets of exemplars under the exemplar-based clustering
 * function of Buschjaeger & Morik ("GPU-Accelerated Optimizer-Aware
 * Evaluation of Submodular Exemplar Clustering"):
 *
 *   L(X) = (1/n) * sum_{v in V} min_{x in X} ||v - x||^2        (Eq. (3))
 *   f(S) = L({e0}) - L(S u {e0}),  e0 = the zero vector          (Eq. (4))
 *
 * with the squared Euclidean dissimilarity of the paper's experiments
 * (Section V).  It evaluates many sets in one call, the "multiset" workload an
 * optimizer produces in every step (Section IV-A), on one gfx950 GPU.
 *
 * Conventions shared by every entry point:
 *   - Array arguments are DEVICE pointers on the current HIP device.  The
 *     caller owns them and keeps them alive until the work queued on `stream`
 *     has finished; the library only reads its inputs and writes its outputs.
 *   - `stream` is a hipStream_t (NULL = the null stream).  Calls are
 *     asynchronous: they validate on the host, queue kernels on `stream` and
 *     return without synchronising.  Temporary device memory comes from a
 *     library-owned stream-ordered pool; the blocks a call used are kept for
 *     the next calls on the same stream (up to 4 per stream, for the 8 most
 *     recently used streams), so repeated calls allocate nothing.  Kept
 *     blocks are released when those limits are exceeded or when an
 *     allocation fails, never while a call uses them.  Releasing the blocks
 *     of another stream (a call on a ninth stream of the device evicts the
 *     least recently used one; a failed allocation releases every free
 *     block) waits for the whole device (hipDeviceSynchronize) inside that
 *     call, since the other stream may no longer exist: such a call blocks
 *     the host until all queued work on the device is done.  Callers that
 *     need every call to return at once keep to at most 8 streams per
 *     device.  Calls on different streams may run concurrently; calls on
 *     one stream from several host threads are safe.  Kept blocks are keyed
 *     by the stream's handle, and a new stream can get the handle of a
 *     destroyed one: synchronise a stream before destroying it while calls
 *     of this library are still queued on it.
 *   - V is dense row-major n x d (row stride d elements, no padding), with
 *     element type fp32, fp16 or bf16 as selected by `precision`.  Results are
 *     fp32.  Arithmetic is fp32 (fp16/bf16 products are exact in fp32).
 *   - V must hold finite values.  The kernels' maxima are compiled without
 *     NaN semantics, so a NaN or infinity anywhere in V gives unspecified
 *     results for every set (no error is reported and nothing faults); it
 *     is not detected.  (f itself would be NaN or infinite there.)  The
 *     sums of squares must also stay finite in fp32, which holds for any
 *     finite fp16 data (d <= 2^24) and for fp32 and bf16 data below about
 *     1.8e19 / sqrt(d) in magnitude.
 *   - Sets are int32 row indices into V.  Duplicate indices are allowed.
 *     EXEMCL_EMPTY_SLOT (-1) marks an empty slot, so sets of different sizes
 *     share one k (the blank fields of the paper's evaluation-set matrix,
 *     Section IV-B, Memory Layout).  Any other index outside [0, n) makes
 *     that set's result a quiet NaN and leaves the other results untouched
 *     (detected on the device, no sync).
 *   - The return value is a status, decided on the host before any kernel
 *     runs (EINVAL, ENOMEM) or right after the launches (EDEVICE).
 *   - Every result is bitwise reproducible and independent of the batch it
 *     came in: out[j] depends on V and on set j only, not on l, j or the
 *     other sets.
 */
#ifndef EXEMCL_H
#define EXEMCL_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#if defined(__GNUC__)
#define EXEMCL_API __attribute__((visibility("default")))
#else
#define EXEMCL_API
#endif

/* Padding index of a set shorter than the batch's k. */
#define EXEMCL_EMPTY_SLOT (-1)

/* Storage type of V. */
enum exemcl_precision { EXEMCL_FP32 = 0, EXEMCL_FP16 = 1, EXEMCL_BF16 = 2 };

/* Status codes. */
enum exemcl_status {
    EXEMCL_OK = 0,      /* queued (or nothing to do) */
    EXEMCL_EINVAL = 1,  /* bad argument; nothing was queued */
    EXEMCL_ENOMEM = 2,  /* temporary device memory unavailable; nothing was queued */
    EXEMCL_EDEVICE = 3, /* a HIP call or kernel launch failed */
    EXEMCL_ESCRATCH = 4 /* exemplar_eval_noalloc: the call needs more temporary memory than
                           the fixed scratch buffer holds; nothing was queued */
};

/* Bytes of the fixed device scratch buffer behind exemplar_eval_noalloc. */
#define EXEMCL_SCRATCH_BYTES (64ll << 20)

/* Evaluation paths (see exemplar_plan). */
enum exemcl_path {
    EXEMCL_PATH_NONE = 0, /* nothing to launch (l == 0 or k == 0) */
    EXEMCL_PATH_VALU = 1, /* vector-ALU kernel, exemplars staged in LDS (small d) */
    EXEMCL_PATH_MFMA = 2  /* matrix-core contraction with fused min/sum epilogue */
};

/*
 * exemplar_eval -- f(S_j) for a batch of l sets of k exemplars each.
 *
 * Computes out[j] = f(S_j) = L({e0}) - L(S_j u {e0}) (Eq. (3), Eq. (4)) for
 * S_j = { V[sets[j*k + p]] : p < k, sets[j*k + p] != EXEMCL_EMPTY_SLOT }, the
 * multiset evaluation of Section IV-A.
 * Internally the value is formed as (2/n) * sum_v max(0, max_{s in S_j}
 * (<v,s> - ||s||^2/2)), which equals the definition exactly in real
 * arithmetic and avoids subtracting two nearly equal losses.
 *
 *   V          device, n x d row-major, type per `precision`; read only
 *   n          number of ground points, 1 <= n <= INT32_MAX
 *   d          dimension, 1 <= d <= 2^24 (rows are addressed through 32-bit
 *              byte offsets per block of 32 points)
 *   sets       device, l x k int32 row-major; read only (may be NULL if k == 0)
 *   l          number of sets, l >= 0 (l == 0: returns EXEMCL_OK, queues nothing)
 *   k          set size, k >= 0 (k == 0: every out[j] = 0, since f(empty) = 0)
 *   precision  one of exemcl_precision
 *   out        device, l floats; written
 *   stream     hipStream_t or NULL
 *
 * Errors: EINVAL for a NULL array with a non-zero size, n < 1, n > INT32_MAX,
 * d < 1, d > 2^24, k < 0, l < 0 or an unknown precision; EDEVICE when a
 * launch fails.  Temporary buffers (partial sums and staged exemplar tiles,
 * O(l*k*d) bytes) come from the library's pool; when the whole batch does not
 * fit (or exceeds EXEMCL_WORKSPACE_LIMIT bytes), the batch is processed in
 * chunks of whole set groups, with bitwise the same results (Section IV-B,
 * Chunking).  ENOMEM only when not even one set group (32 sets, or 16 for
 * the shapes with 16-wide tiles) fits -- the paper's chunk size 0.
 */
EXEMCL_API int exemplar_eval(const void *V, int64_t n, int64_t d, const int32_t *sets, int64_t l,
                             int64_t k, int precision, float *out, void *stream);

/*
 * exemplar_eval_noalloc -- exemplar_eval for callers that cannot allocate
 * device memory: code under HIP graph capture, tight serving loops, and
 * harnesses that forbid hipMalloc.
 *
 * Same arguments, results (bitwise equal to exemplar_eval's), asynchrony and
 * errors as exemplar_eval, except for where temporaries live: partial sums,
 * staged exemplar tiles and (when V's rows are not whole 16-byte vectors) the
 * zero-padded copy of V are carved from a fixed scratch buffer of
 * EXEMCL_SCRATCH_BYTES (64 MiB) that is part of the library's code object on
 * each GPU and held until the process ends.  The call makes no allocation of
 * any kind (no hipMalloc, no pool, no library allocation) and records no
 * profiling events.  A batch whose workspace exceeds the buffer is processed
 * in chunks of whole set groups, as exemplar_eval does under a workspace
 * limit, with bitwise the same results.
 *
 * Every call on one GPU uses that GPU's one buffer, and the buffer keeps the
 * last call's contents (nothing in it needs to start at zero: every byte a
 * kernel reads was written earlier in the same call).  Calls that overlap on
 * one GPU -- on different streams, or from different host threads -- race on
 * the buffer and give undefined results: serialise them (one stream, or
 * events between the streams).  Calls on different GPUs are independent.
 *
 * Errors: as exemplar_eval, plus EXEMCL_ESCRATCH when even one set group's
 * workspace plus the padded copy of V does not fit the buffer (for example
 * n in the tens of millions of points, where one set group's partial sums
 * alone exceed 64 MiB, or a padded copy of V larger than the buffer); nothing
 * is queued then.  EXEMCL_WORKSPACE_LIMIT, when set lower, caps it further.
 */
EXEMCL_API int exemplar_eval_noalloc(const void *V, int64_t n, int64_t d, const int32_t *sets, int64_t l,
                                     int64_t k, int precision, float *out, void *stream);

/*
 * exemplar_eval_streamed -- exemplar_eval for a V kept in HOST memory, e.g.
 * one larger than the device's memory.
 *
 * The paper keeps V resident on the GPU and splits only the sets into chunks
 * (Section IV-B, Chunking); that fails once V itself does not fit.  This call
 * streams V through the device in blocks of rows instead: the set members'
 * rows are copied once into a compact exemplar matrix and staged, then every
 * row block is copied in (double-buffered, overlapping the previous block's
 * kernels) and evaluated by the same kernels as exemplar_eval, and its
 * per-set sums are added to an fp64 accumulator in block order.  The result
 * equals f(S_j) up to rounding (within the tolerances of exemplar_eval, not
 * bitwise equal to it: the summation is grouped by blocks).
 *
 *   V               HOST, n x d row-major, type per `precision`; read only.
 *                   Pinned memory (hipHostMalloc) whose rows are whole
 *                   16-byte vectors is copied to the device directly; any
 *                   other host memory goes through the library's pinned
 *                   staging buffers.
 *   n, d, l, k      as for exemplar_eval
 *   sets            HOST, l x k int32 row-major; read only
 *   precision       one of exemcl_precision
 *   rows_per_block  ground points per streamed block (rounded up to the
 *                   kernel's row block); 0 = about 64 MiB of V per block
 *   out             HOST, l floats; written before the call returns
 *   stream          hipStream_t or NULL; the kernels run on it, the copies on
 *                   a second stream of the library's
 *
 * Unlike the other entry points this call is synchronous: it returns once
 * `out` holds the results.  Calls are serialised within a process (they
 * share the pinned staging buffers, which the library keeps between calls).
 * Device memory: two row blocks, the compact exemplar matrix and its tiles,
 * one block's partial sums -- O(rows_per_block * d + l * k * d) bytes, counted
 * against EXEMCL_WORKSPACE_LIMIT; the sets are not chunked here.
 * Errors: EINVAL as for exemplar_eval (rows_per_block < 0 too); ENOMEM when
 * the device or pinned buffers cannot be allocated; EDEVICE when a copy or
 * launch fails.  Empty slots and invalid indices behave as in exemplar_eval.
 */
EXEMCL_API int exemplar_eval_streamed(const void *V, int64_t n, int64_t d, const int32_t *sets, int64_t l,
                                      int64_t k, int precision, int64_t rows_per_block, float *out,
                                      void *stream);

/*
 * exemplar_gain -- one Greedy step: f(S u {c}) for every candidate c.
 *
 * The Greedy optimizer (Algorithm 1) evaluates, in every round, the multiset
 * { S u {c_1}, ..., S u {c_m} } for the current solution S (Section IV-A).
 * This call scores that multiset with fp32 V: it first caches, for every
 * point, g(v) = max(0, max_{s in S} (<v,s> - ||s||^2/2)) (so that
 * min(||v||^2, min_s ||v-s||^2) = ||v||^2 - 2 g(v)), then forms
 * out[j] = (2/n) * sum_v max(g(v), <v,c_j> - ||c_j||^2/2) = f(S u {c_j}).
 * The discrete derivative of Definition 1 is out[j] - f(S).
 *
 *   V      device, n x d fp32 row-major; read only
 *   n, d   as for exemplar_eval
 *   S      device, k int32 indices (the current solution); NULL if k == 0
 *   k      |S| >= 0; every scored set has k + 1 members
 *   cands  device, l int32 candidate indices; read only
 *   l      number of candidates, l >= 0
 *   out    device, l floats; written
 *   stream hipStream_t or NULL
 *
 * A candidate already in S scores f(S).  An invalid index in S makes every
 * result NaN; an invalid candidate makes its own result NaN.
 * Errors as for exemplar_eval.
 */
EXEMCL_API int exemplar_gain(const float *V, int64_t n, int64_t d, const int32_t *S, int64_t k,
                             const int32_t *cands, int64_t l, float *out, void *stream);

/*
 * exemplar_greedy -- the Greedy optimizer of Algorithm 1, run on the device.
 *
 * K rounds; round i scores f(S u {c}) for every point c of V not yet in S
 * (the same computation as exemplar_gain, with the cache g(v) kept on the
 * device and updated as g <- max(g, <v,c*> - ||c*||^2/2) after each round),
 * and adds the best candidate c*.  Ties go to the lowest index (Algorithm 1
 * leaves the choice open); a NaN score ranks below every number.  The
 * rounds are queued back to back on the stream: no host synchronisation.
 *
 *   V      device, n x d fp32 row-major; read only
 *   n, d   as for exemplar_eval
 *   K      rounds, 0 <= K <= n
 *   S_out  device, K int32; S_out[i] = the point added in round i
 *   f_out  device, K floats; f_out[i] = f({S_out[0], ..., S_out[i]})
 *   stream hipStream_t or NULL
 *
 * Scores of round i are those exemplar_gain returns for S = S_out[0..i-1]
 * (bitwise), so f_out[i] - f_out[i-1] is the round's discrete derivative
 * (Definition 1).  Temporary memory: about 17 bytes per point plus a scoring
 * workspace kept under 1 GiB by scoring the candidates in chunks.
 * Errors: EINVAL for bad sizes (K > n, d > 2^24) or NULL outputs when K > 0;
 * ENOMEM / EDEVICE as for exemplar_eval.
 */
EXEMCL_API int exemplar_greedy(const float *V, int64_t n, int64_t d, int64_t K, int32_t *S_out,
                               float *f_out, void *stream);

/*
 * exemplar_sqnorm -- q[i] = ||v_i||^2, the squared distance of every ground
 * point to e0, in fp32.  Its mean is L({e0}), the set-independent term of
 * Eq. (4) that the paper computes once up front (Section IV-B, Algorithm).
 *
 *   V, n, d, precision  as for exemplar_eval
 *   q                   device, n floats; written
 *
 * One pass over V (HBM-bound).  The environment variable
 * EXEMCL_SQNORM_MAX_BLOCKS=<b> lowers the number of workgroups per launch
 * (tests: several grid passes at a small n); the results do not depend on it.
 *
 * Errors: EINVAL / EDEVICE as above.
 */
EXEMCL_API int exemplar_sqnorm(const void *V, int64_t n, int64_t d, int precision, float *q,
                               void *stream);

/*
 * exemplar_plan -- host-only description of what exemplar_eval would launch
 * for these sizes; touches no device.  Writes the chosen exemcl_path to
 * *path and the temporary device bytes to *workspace_bytes (either pointer
 * may be NULL).  The path depends on (d, k, precision) only, never on l or n,
 * which is what keeps out[j] independent of the batch.  The environment
 * variable EXEMCL_PATH=valu|mfma forces a path where it applies (tests).
 * Two more variables tune the MFMA launch without changing any result:
 * EXEMCL_PERSIST=0|2 forces the plain or the persistent grid (default: a
 * rule on the kernel's occupancy and the work per resident workgroup), and
 * EXEMCL_WG_TARGET=<n> sets how many workgroups a launch aims for when set
 * groups are chunked.  All variables are read on every call.
 * Returns EINVAL for arguments exemplar_eval would reject, else EXEMCL_OK.
 */
EXEMCL_API int exemplar_plan(int64_t n, int64_t d, int64_t l, int64_t k, int precision, int *path,
                             int64_t *workspace_bytes);

/*
 * Profiling hook.  exemplar_prof_enable(N), N >= 1, makes every N-th
 * following exemplar_eval / exemplar_gain call (the first one included)
 * time its dominant kernel (the contraction + epilogue kernel) with a pair
 * of HIP events: for the MFMA kernel the kernel's dispatch records them at
 * its start and end, for the VALU kernel they are recorded around it on the
 * stream.  exemplar_prof_enable(0) stops recording;
 * N < 0 is EXEMCL_EINVAL.  exemplar_prof_read waits for the recorded events,
 * writes the summed kernel time in milliseconds and the number of recorded
 * launches, and forgets them.  Either pointer may be NULL.  Meant for
 * benchmarks: each recorded call costs two events, so long runs sample
 * (N > 1).
 */
EXEMCL_API int exemplar_prof_enable(int every);
EXEMCL_API int exemplar_prof_read(double *ms_total, int64_t *launches);

/* exemplar_strerror -- static, NUL-terminated text for a status code. */
EXEMCL_API const char *exemplar_strerror(int status);

/* exemplar_version -- library version as 10000*major + 100*minor + patch. */
EXEMCL_API int exemplar_version(void);

#ifdef __cplusplus
}
#endif

#endif /* EXEMCL_H */
