// host.cpp -- the C ABI declared in include/exemcl.h: argument validation,
// path selection, stream-ordered temporary memory, kernel sequencing.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <thread>
#include <utility>
#include <vector>

#include "exemcl.h"
#include "internal.h"

using namespace exemcl;

namespace {

constexpr int kVersion = 100;  // 0.1.0

bool prec_ok(int p) { return p == EXEMCL_FP32 || p == EXEMCL_FP16 || p == EXEMCL_BF16; }

int64_t align_up(int64_t x, int64_t a) { return (x + a - 1) / a * a; }

// EXEMCL_PATH=valu|mfma forces a path where it applies (tests, tuning).
int forced_path() {
    const char *s = getenv("EXEMCL_PATH");
    if (!s) return 0;
    if (!strcmp(s, "valu")) return EXEMCL_PATH_VALU;
    if (!strcmp(s, "mfma")) return EXEMCL_PATH_MFMA;
    return 0;
}

// EXEMCL_WORKSPACE_LIMIT=<bytes> caps temporary memory (forces ENOMEM in tests).
int64_t workspace_limit() {
    const char *s = getenv("EXEMCL_WORKSPACE_LIMIT");
    if (!s || !*s) return INT64_MAX;
    char *end = nullptr;
    long long v = strtoll(s, &end, 10);
    return (end && *end == '\0' && v >= 0) ? (int64_t)v : INT64_MAX;
}

// Workgroups an MFMA launch aims for (EXEMCL_WG_TARGET overrides, for tuning):
// enough to cover 256 CUs several times; a chunk of set groups shares one
// load of a workgroup's points.
int64_t wg_target() {
    const char *s = getenv("EXEMCL_WG_TARGET");
    if (!s || !*s) return 2048;
    char *end = nullptr;
    long long v = strtoll(s, &end, 10);
    return (end && *end == '\0' && v >= 1 && v <= (1 << 24)) ? (int64_t)v : 2048;
}

// Path choice: a function of (d, k, precision) only.
int choose_path(int64_t d, int64_t k, int precision) {
    MfmaPlan mp;
    ValuPlan vp;
    const bool can_mfma = mfma_plan(precision, d, &mp);
    const bool can_valu = valu_plan(precision, d, k, &vp);
    const int f = forced_path();
    if (f == EXEMCL_PATH_VALU && can_valu) return EXEMCL_PATH_VALU;
    if (f == EXEMCL_PATH_MFMA && can_mfma) return EXEMCL_PATH_MFMA;
    if (can_mfma) return EXEMCL_PATH_MFMA;
    if (can_valu) return EXEMCL_PATH_VALU;
    return EXEMCL_PATH_NONE;
}

struct Layout {
    int path = EXEMCL_PATH_NONE;
    MfmaPlan mp{};
    ValuPlan vp{};
    int64_t G = 0, lpad = 0, ngroups = 0, gpc = 0;
    int64_t off_partials = 0, off_tiles = 0, bytes = 0;
};

int64_t tile_bytes(const MfmaPlan &mp) { return mfma_tile_bytes(mp); }

// Workspace of one exemplar_eval call (or of the scoring half of a gain call).
bool layout_eval(int64_t n, int64_t d, int64_t l, int64_t k, int precision, int path, Layout *L) {
    L->path = path;
    if (path == EXEMCL_PATH_MFMA) {
        if (!mfma_plan(precision, d, &L->mp)) return false;
        const int64_t tm = L->mp.tile;
        L->ngroups = (l + tm - 1) / tm;
        L->lpad = L->ngroups * tm;
        const int64_t nrb = (n + L->mp.rows - 1) / L->mp.rows;
        // one partial-sum row per wavefront, or per workgroup when the kernel
        // adds its wavefronts' sums itself
        L->G = nrb * (L->mp.wgsum ? 1 : L->mp.waves);
        const int64_t target = wg_target();
        int64_t chunks = (target + nrb - 1) / nrb;
        if (chunks < 1) chunks = 1;
        if (chunks > L->ngroups) chunks = L->ngroups;
        if (chunks > 65535) chunks = 65535;
        L->gpc = (L->ngroups + chunks - 1) / chunks;
        L->off_partials = 0;
        L->off_tiles = align_up(L->G * L->lpad * 4, 256);
        L->bytes = align_up(L->off_tiles + L->ngroups * mfma_tiles_per_group(L->mp, k) * tile_bytes(L->mp), 256);
        return true;
    }
    if (path == EXEMCL_PATH_VALU) {
        if (!valu_plan(precision, d, k, &L->vp)) return false;
        L->lpad = l;
        L->G = (n + L->vp.rows - 1) / L->vp.rows;
        L->off_partials = 0;
        L->bytes = align_up(L->G * L->lpad * 4, 256);
        return true;
    }
    L->bytes = 0;
    return true;
}

int check_common(const void *V, int64_t n, int64_t d, int64_t l, int64_t k, const void *out) {
    if (!V) return EXEMCL_EINVAL;
    if (n < 1 || n > INT32_MAX) return EXEMCL_EINVAL;
    if (d < 1 || d > INT32_MAX) return EXEMCL_EINVAL;
    if (k < 0 || l < 0) return EXEMCL_EINVAL;
    if (l > 0 && !out) return EXEMCL_EINVAL;
    return EXEMCL_OK;
}

// Library-owned stream-ordered pool per device, keeping freed blocks cached.
std::mutex g_pool_mu;
hipMemPool_t g_pools[64] = {};

hipError_t get_pool(hipMemPool_t *pool) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lk(g_pool_mu);
    if (!g_pools[dev]) {
        hipMemPoolProps props{};
        props.allocType = hipMemAllocationTypePinned;
        props.handleTypes = hipMemHandleTypeNone;
        props.location.type = hipMemLocationTypeDevice;
        props.location.id = dev;
        hipMemPool_t p = nullptr;
        e = hipMemPoolCreate(&p, &props);
        if (e != hipSuccess) return e;
        uint64_t keep = UINT64_MAX;
        e = hipMemPoolSetAttribute(p, hipMemPoolAttrReleaseThreshold, &keep);
        if (e != hipSuccess) return e;
        g_pools[dev] = p;
    }
    *pool = g_pools[dev];
    return hipSuccess;
}

// Temporary blocks kept for later calls on the same stream, keyed by
// (device, stream handle): a call takes the smallest free kept block that is
// large enough and gives it back when it has queued its work, so repeated
// calls allocate and free nothing.  Stream order makes the reuse safe: the
// next call on that stream runs after the work of the previous one.  A
// block a call is using is marked busy, so calls that share a stream from
// different host threads never share a block.  At most kKeepPerStream
// blocks per stream (the smallest free one is released, in stream order, to
// make room) and kKeepStreams streams (the least recently used stream's
// free blocks are released with hipFree, which waits for the device) are
// kept; a failed allocation releases every free kept block and retries.
constexpr size_t kKeepPerStream = 4;
constexpr size_t kKeepStreams = 8;
struct KeptBlock {
    void *p;
    size_t bytes;
    bool busy;
};
struct StreamBlocks {
    int dev;
    uintptr_t sid;
    uint64_t used;  // last-use tick
    std::vector<KeptBlock> blocks;
};
std::mutex g_keep_mu;
std::vector<StreamBlocks> g_keep;
uint64_t g_keep_tick = 0;

StreamBlocks *kept_for(int dev, uintptr_t sid) {
    for (auto &e : g_keep)
        if (e.dev == dev && e.sid == sid) return &e;
    return nullptr;
}

// Releases the free blocks of entry i after waiting for the device, so it
// is safe whatever the state of that entry's stream; drops the entry when
// empty.
void release_free_blocks(size_t i) {
    (void)hipDeviceSynchronize();
    auto &bl = g_keep[i].blocks;
    for (size_t b = 0; b < bl.size();) {
        if (!bl[b].busy) {
            (void)hipFree(bl[b].p);
            bl.erase(bl.begin() + (std::ptrdiff_t)b);
        } else {
            ++b;
        }
    }
    if (bl.empty()) g_keep.erase(g_keep.begin() + (std::ptrdiff_t)i);
}

// A caller-provided region that temporaries are carved from, front to back,
// instead of being allocated (exemplar_eval_noalloc).  Carving is a host-side
// bump of `used`; nothing is returned to it within a call.
struct Arena {
    char *base = nullptr;
    int64_t cap = 0;
    int64_t used = 0;
    int64_t left() const { return cap - used; }
};

struct Scratch {
    void *ptr = nullptr;
    hipStream_t st = nullptr;
    bool kept = false;
    bool borrowed = false;  // carved from an Arena: nothing to release
    int dev = 0;
    uintptr_t sid = 0;
    ~Scratch() {
        if (!ptr || borrowed) return;
        if (!kept) {
            hipFreeAsync(ptr, st);
            return;
        }
        std::lock_guard<std::mutex> lk(g_keep_mu);
        if (StreamBlocks *e = kept_for(dev, sid))
            for (auto &b : e->blocks)
                if (b.p == ptr) b.busy = false;
    }
};

int alloc_scratch(Scratch *s, int64_t bytes, hipStream_t st, Arena *arena = nullptr) {
    s->st = st;
    if (bytes <= 0) return EXEMCL_OK;
    if (bytes > workspace_limit()) return EXEMCL_ENOMEM;
    if (arena) {
        const int64_t take = align_up(bytes, 256);
        if (take > arena->left()) return EXEMCL_ENOMEM;
        s->ptr = arena->base + arena->used;
        s->borrowed = true;
        arena->used += take;
        return EXEMCL_OK;
    }
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) {
        (void)hipGetLastError();
        return EXEMCL_EDEVICE;
    }
    const uintptr_t sid = (uintptr_t)st;
    s->dev = dev;
    s->sid = sid;
    {
        std::lock_guard<std::mutex> lk(g_keep_mu);
        if (StreamBlocks *e = kept_for(dev, sid)) {
            e->used = ++g_keep_tick;
            KeptBlock *best = nullptr;
            for (auto &b : e->blocks)
                if (!b.busy && b.bytes >= (size_t)bytes && (!best || b.bytes < best->bytes)) best = &b;
            if (best) {
                best->busy = true;
                s->ptr = best->p;
                s->kept = true;
                return EXEMCL_OK;
            }
        }
    }
    hipMemPool_t pool;
    if (get_pool(&pool) != hipSuccess) return EXEMCL_EDEVICE;
    hipError_t e = hipMallocFromPoolAsync(&s->ptr, (size_t)bytes, pool, st);
    if (e == hipErrorOutOfMemory) {
        (void)hipGetLastError();
        {
            std::lock_guard<std::mutex> lk(g_keep_mu);
            for (size_t i = g_keep.size(); i-- > 0;)
                if (g_keep[i].dev == dev) release_free_blocks(i);
        }
        e = hipMallocFromPoolAsync(&s->ptr, (size_t)bytes, pool, st);
    }
    if (e == hipErrorOutOfMemory) {
        (void)hipGetLastError();
        s->ptr = nullptr;
        return EXEMCL_ENOMEM;
    }
    if (e != hipSuccess) {
        s->ptr = nullptr;
        return EXEMCL_EDEVICE;
    }
    // Keep the new block for this stream.
    std::lock_guard<std::mutex> lk(g_keep_mu);
    StreamBlocks *entry = kept_for(dev, sid);
    if (!entry) {
        if (g_keep.size() >= kKeepStreams) {
            // the least recently used stream of this device (the device wait
            // in release_free_blocks covers the current device only)
            size_t lru = g_keep.size();
            for (size_t i = 0; i < g_keep.size(); ++i)
                if (g_keep[i].dev == dev && (lru == g_keep.size() || g_keep[i].used < g_keep[lru].used)) lru = i;
            if (lru < g_keep.size()) release_free_blocks(lru);
        }
        if (g_keep.size() >= kKeepStreams) return EXEMCL_OK;  // all busy: free this block after the call
        g_keep.push_back(StreamBlocks{dev, sid, ++g_keep_tick, {}});
        entry = &g_keep.back();
    }
    auto &bl = entry->blocks;
    if (bl.size() >= kKeepPerStream) {
        // release the smallest free block of this stream, in stream order
        size_t victim = bl.size();
        for (size_t b = 0; b < bl.size(); ++b)
            if (!bl[b].busy && (victim == bl.size() || bl[b].bytes < bl[victim].bytes)) victim = b;
        if (victim == bl.size()) return EXEMCL_OK;  // all busy: free this block after the call
        hipFreeAsync(bl[victim].p, st);
        bl.erase(bl.begin() + (std::ptrdiff_t)victim);
    }
    bl.push_back(KeptBlock{s->ptr, (size_t)bytes, true});
    s->kept = true;
    return EXEMCL_OK;
}

int status_of(hipError_t e) { return e == hipSuccess ? EXEMCL_OK : EXEMCL_EDEVICE; }

int64_t elem_size(int precision) { return precision == EXEMCL_FP32 ? 4 : 2; }

// V as the MFMA kernels read it: V itself when its rows are whole aligned
// 16-byte lane vectors, else a zero-padded copy in temporary memory.
struct MfmaRows {
    const void *V = nullptr;
    int64_t ld = 0;
    int64_t bytes = 0;  // temporary memory held by the copy
    Scratch copy;
};

// The single-k-block fp32 layout reads rows one coordinate at a time and
// takes V as it is.
bool rows_as_is(int precision, int64_t d) {
    MfmaPlan mp;
    return mfma_plan(precision, d, &mp) && mp.il && mp.nkb == 1;
}

// Temporary bytes of the padded copy of V (0 when rows of this d are read in
// place; V whose alignment does not allow it is still copied).
int64_t pad_bytes(int precision, int64_t n, int64_t d) {
    if (rows_as_is(precision, d) || mfma_rows_in_place(precision, d)) return 0;
    return align_up(n * mfma_row_stride(precision, d) * elem_size(precision), 256);
}

int prepare_rows(const void *V, int64_t n, int64_t d, int precision, hipStream_t st, MfmaRows *r,
                 Arena *arena = nullptr) {
    if (rows_as_is(precision, d) || mfma_rows_ready(precision, V, d)) {
        r->V = V;
        r->ld = d;
        return EXEMCL_OK;
    }
    r->ld = mfma_row_stride(precision, d);
    r->bytes = align_up(n * r->ld * elem_size(precision), 256);
    const int rc = alloc_scratch(&r->copy, r->bytes, st, arena);
    if (rc) return rc;
    if (launch_pad(precision, V, n, (int)d, r->copy.ptr, (int)r->ld, st) != hipSuccess) return EXEMCL_EDEVICE;
    r->V = r->copy.ptr;
    return EXEMCL_OK;
}

// Event pairs around the dominant kernel, recorded while profiling is on.
std::mutex g_prof_mu;
int g_prof_every = 0;    // record every g_prof_every-th call; 0 = off
int64_t g_prof_calls = 0;  // calls seen since recording was switched on
std::vector<std::pair<hipEvent_t, hipEvent_t>> g_prof_events;

// Timing of one sampled call's dominant kernel.  For the MFMA kernel the
// pair is handed to the launch (hipExtLaunchKernel), whose dispatch records
// it at the kernel's start and end; for other launches record() brackets
// them on the stream.
struct ProfRange {
    hipEvent_t a = nullptr, b = nullptr;
    hipStream_t st;
    explicit ProfRange(hipStream_t s, bool allowed = true) : st(s) {
        if (!allowed) return;
        bool on;
        {
            std::lock_guard<std::mutex> lk(g_prof_mu);
            on = g_prof_every > 0 && g_prof_calls++ % g_prof_every == 0;
        }
        if (!on) return;
        if (hipEventCreate(&a) != hipSuccess || hipEventCreate(&b) != hipSuccess) {
            if (a) hipEventDestroy(a);
            a = b = nullptr;
        }
    }
    void record_start() {
        if (a) hipEventRecord(a, st);
    }
    void record_stop() {
        if (b) hipEventRecord(b, st);
    }
    // Keep the pair for exemplar_prof_read (after a successful launch).
    void end() {
        if (!a) return;
        std::lock_guard<std::mutex> lk(g_prof_mu);
        g_prof_events.emplace_back(a, b);
        a = b = nullptr;
    }
    ~ProfRange() {
        if (a) hipEventDestroy(a);
        if (b) hipEventDestroy(b);
    }
};

// Queue the evaluation of sets [0, l) with a workspace laid out by L.
hipError_t run_chunk(const Layout &L, char *base, const void *V, int64_t n, int64_t d, const MfmaRows *rows,
                     const int32_t *sets, int64_t l, int64_t k, int precision, const float *m0,
                     const int32_t *common, int64_t kcommon, float *out, hipStream_t st, bool prof = true) {
    if (L.path == EXEMCL_PATH_NONE) return launch_zero(out, l, st);  // k = 0: every set is empty
    float *partials = (float *)(base + L.off_partials);
    hipError_t e = hipSuccess;
    if (L.path == EXEMCL_PATH_MFMA) {
        void *tiles = base + L.off_tiles;
        e = launch_pack(precision, L.mp, rows->V, n, (int)rows->ld, sets, l, k, tiles, st);
        if (e == hipSuccess) {
            ProfRange pr(st, prof);
            e = launch_mfma(precision, MODE_SUM, L.mp, rows->V, n, (int)rows->ld, tiles, mfma_tiles_per_group(L.mp, k),
                            L.ngroups, L.gpc, m0, partials, L.lpad, nullptr, st, pr.a, pr.b);
            if (e == hipSuccess) pr.end();
        }
    } else if (L.path == EXEMCL_PATH_VALU) {
        ProfRange pr(st, prof);
        pr.record_start();
        e = launch_valu(precision, L.vp, V, n, (int)d, sets, l, k, partials, L.lpad, st);
        pr.record_stop();
        if (e == hipSuccess) pr.end();
    }
    if (e == hipSuccess)
        e = launch_reduce(partials, L.G, L.lpad, l, n, sets, k, common, kcommon, out, st);
    return e;
}

// Queue one evaluation of `l` sets of `k` members (shared by eval and the
// scoring half of gain).  `m0` (nullable) is the per-point initial max.
//
// Chunking (Section IV-B, Chunking): when the temporary memory for all l sets
// is not available (EXEMCL_WORKSPACE_LIMIT, or the pool cannot grow), the
// batch is split into chunks of whole set groups that fit, processed one
// after another in one workspace.  A set's result does not depend on the
// batch it is evaluated in, so chunked results are bitwise the same.  ENOMEM
// only when not even one set group fits -- the paper's chunk size 0.
//
// `rows` (nullable) is V already prepared for the MFMA kernels by the caller,
// which also holds `reserved` bytes of temporary memory that count against
// EXEMCL_WORKSPACE_LIMIT.  With `arena` every temporary is carved from it
// (and the chunks are sized to what is left of it); nothing is allocated.
int run_eval(const void *V, int64_t n, int64_t d, const int32_t *sets, int64_t l, int64_t k, int precision,
             const float *m0, const int32_t *common, int64_t kcommon, float *out, hipStream_t st,
             const MfmaRows *rows = nullptr, int64_t reserved = 0, Arena *arena = nullptr) {
    if (l == 0) return EXEMCL_OK;
    int path = k == 0 ? EXEMCL_PATH_NONE : choose_path(d, k, precision);
    if (m0 && path == EXEMCL_PATH_VALU) path = EXEMCL_PATH_MFMA;
    if (k > 0 && path == EXEMCL_PATH_NONE) return EXEMCL_EINVAL;
    Layout L;
    if (!layout_eval(n, d, l, k, precision, path, &L)) return EXEMCL_EINVAL;
    const int64_t unit = path == EXEMCL_PATH_MFMA ? L.mp.tile : 1;
    MfmaRows own;
    if (path == EXEMCL_PATH_MFMA && !rows) {
        const int64_t pb = pad_bytes(precision, n, d);
        if (reserved + pb > workspace_limit() || (arena && pb > arena->left())) return EXEMCL_ENOMEM;
        // Nothing is queued unless the padded rows and one set group fit.
        Layout L1;
        if (!layout_eval(n, d, std::min<int64_t>(l, unit), k, precision, path, &L1)) return EXEMCL_EINVAL;
        if (reserved + pb + L1.bytes > workspace_limit() || (arena && pb + L1.bytes > arena->left()))
            return EXEMCL_ENOMEM;
        const int rc = prepare_rows(V, n, d, precision, st, &own, arena);
        if (rc) return rc;
        rows = &own;
        reserved += own.bytes;
    }
    int64_t limit = workspace_limit() - reserved;
    if (arena) limit = std::min(limit, arena->left());
    int64_t lc = l;
    Scratch ws;
    for (;;) {
        if (!layout_eval(n, d, lc, k, precision, path, &L)) return EXEMCL_EINVAL;
        if (L.bytes <= limit) {
            const int rc = alloc_scratch(&ws, L.bytes, st, arena);
            if (rc == EXEMCL_OK) break;
            if (rc != EXEMCL_ENOMEM) return rc;
        }
        if (lc <= unit) return EXEMCL_ENOMEM;
        lc = ((lc + 1) / 2 + unit - 1) / unit * unit;
    }
    char *base = (char *)ws.ptr;
    for (int64_t j0 = 0; j0 < l; j0 += lc) {
        const int64_t lj = l - j0 < lc ? l - j0 : lc;
        Layout Lj;
        if (!layout_eval(n, d, lj, k, precision, path, &Lj)) return EXEMCL_EINVAL;
        const hipError_t e = run_chunk(Lj, base, V, n, d, rows, sets + j0 * k, lj, k, precision, m0, common,
                                       kcommon, out + j0, st, arena == nullptr);
        if (e != hipSuccess) return EXEMCL_EDEVICE;
    }
    return EXEMCL_OK;
}

// ---------------------------------------------------------------------------
// Out-of-core evaluation: V (and the sets) in host memory.
//
// The paper keeps V resident on the device and chunks only the sets
// (Section IV-B, Chunking); its chunking fails once V itself does not fit.
// Here V streams through the device in blocks of rows: the members of every
// set are copied once into a compact exemplar matrix and staged into tiles,
// then each row block is copied in (double-buffered, on a second stream, so
// the copy of block b + 1 overlaps the kernels of block b), evaluated by the
// unchanged kernel, and its per-set sums are added to an fp64 accumulator in
// block order.  The sum over points splits exactly across row blocks, so the
// result is f(S_j) up to rounding.
// ---------------------------------------------------------------------------

// Pinned host buffers kept between calls; the mutex also serialises
// exemplar_eval_streamed within the process.
std::mutex g_stream_mu;
struct Pinned {
    void *p = nullptr;
    size_t bytes = 0;
};
Pinned g_pin_rows[2], g_pin_exem, g_pin_idx, g_pin_bad;

hipError_t pinned_reserve(Pinned *b, size_t bytes) {
    if (b->bytes >= bytes) return hipSuccess;
    if (b->p) (void)hipHostFree(b->p);
    b->p = nullptr;
    b->bytes = 0;
    hipError_t e = hipHostMalloc(&b->p, bytes, hipHostMallocDefault);
    if (e == hipSuccess) b->bytes = bytes;
    return e;
}

bool host_is_pinned(const void *p) {
    hipPointerAttribute_t a{};
    const hipError_t e = hipPointerGetAttributes(&a, p);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        return false;
    }
    return a.type == hipMemoryTypeHost;
}

// dst rows [0, rows) with stride ld elements <- src rows with stride d,
// columns d .. ld-1 set to zero; split over a few threads.
void copy_rows(void *dst, int64_t ld, const void *src, int64_t d, int64_t rows, int64_t es) {
    const int64_t bytes = rows * d * es;
    const unsigned hw = std::max(1u, std::thread::hardware_concurrency());
    const int64_t nt = std::min<int64_t>(std::min<int64_t>(16, hw), std::max<int64_t>(1, bytes >> 22));
    auto part = [&](int64_t r0, int64_t r1) {
        if (ld == d) {
            memcpy((char *)dst + r0 * d * es, (const char *)src + r0 * d * es, (size_t)((r1 - r0) * d * es));
        } else {
            for (int64_t r = r0; r < r1; ++r) {
                memcpy((char *)dst + r * ld * es, (const char *)src + r * d * es, (size_t)(d * es));
                memset((char *)dst + (r * ld + d) * es, 0, (size_t)((ld - d) * es));
            }
        }
    };
    if (nt <= 1) {
        part(0, rows);
        return;
    }
    std::vector<std::thread> th;
    for (int64_t t = 0; t < nt; ++t) th.emplace_back(part, rows * t / nt, rows * (t + 1) / nt);
    for (auto &x : th) x.join();
}

// Copy stream and events of the streamed path, created once per device and
// kept (guarded by g_stream_mu, which serialises streamed calls).
struct StreamedState {
    hipStream_t cs = nullptr;
    hipEvent_t copied[2] = {nullptr, nullptr}, freed[2] = {nullptr, nullptr};
};
StreamedState g_streamed[64];

hipError_t streamed_state(StreamedState **out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
    StreamedState &ss = g_streamed[dev];
    if (!ss.cs) {
        hipStream_t cs = nullptr;
        e = hipStreamCreateWithFlags(&cs, hipStreamNonBlocking);
        for (int i = 0; i < 2 && e == hipSuccess; ++i) {
            e = hipEventCreateWithFlags(&ss.copied[i], hipEventDisableTiming);
            if (e == hipSuccess) e = hipEventCreateWithFlags(&ss.freed[i], hipEventDisableTiming);
        }
        if (e != hipSuccess) return e;
        ss.cs = cs;
    }
    *out = &ss;
    return hipSuccess;
}

int run_streamed(const void *V, int64_t n, int64_t d, const int32_t *sets, int64_t l, int64_t k, int precision,
                 int64_t rows_per_block, float *out, hipStream_t st) {
    MfmaPlan mp;
    if (!mfma_plan(precision, d, &mp)) return EXEMCL_EINVAL;
    const int64_t es = elem_size(precision);
    const int64_t ld = mfma_row_stride(precision, d);
    const int64_t ne = l * k;  // rows of the compact exemplar matrix: member (j, p) is row j*k + p
    int64_t R = rows_per_block > 0 ? rows_per_block : std::max<int64_t>(1, ((int64_t)64 << 20) / (ld * es));
    R = std::min(R, n);
    R = (R + mp.rows - 1) / mp.rows * mp.rows;  // whole row blocks of the kernel

    // Device workspace: 2 row buffers, exemplars, remapped indices, tiles,
    // one block's partials, the fp64 accumulator, flags and the results.
    Layout L;
    if (!layout_eval(R, d, l, k, precision, EXEMCL_PATH_MFMA, &L)) return EXEMCL_EINVAL;
    const int64_t rows_bytes = align_up(R * ld * es, 256);
    const int64_t off_rows1 = rows_bytes;
    const int64_t off_exem = off_rows1 + rows_bytes;
    const int64_t off_idx = off_exem + align_up(ne * ld * es, 256);
    const int64_t off_acc = off_idx + align_up(ne * 4, 256);
    const int64_t off_bad = off_acc + align_up(l * 8, 256);
    const int64_t off_out = off_bad + align_up(l, 256);
    const int64_t off_work = off_out + align_up(l * 4, 256);
    const int64_t bytes = off_work + L.bytes;
    if (bytes > workspace_limit()) return EXEMCL_ENOMEM;

    std::lock_guard<std::mutex> lk(g_stream_mu);
    const bool direct = ld == d && host_is_pinned(V);
    if (pinned_reserve(&g_pin_exem, (size_t)std::max<int64_t>(1, ne * ld * es)) != hipSuccess ||
        pinned_reserve(&g_pin_idx, (size_t)std::max<int64_t>(1, ne * 4)) != hipSuccess ||
        pinned_reserve(&g_pin_bad, (size_t)std::max<int64_t>(1, l)) != hipSuccess)
        return EXEMCL_ENOMEM;
    if (!direct) {
        for (int i = 0; i < 2; ++i)
            if (pinned_reserve(&g_pin_rows[i], (size_t)(R * ld * es)) != hipSuccess) return EXEMCL_ENOMEM;
    }

    Scratch ws;
    int rc = alloc_scratch(&ws, bytes, st);
    if (rc) return rc;
    char *base = (char *)ws.ptr;
    void *drows[2] = {base, base + off_rows1};
    void *dexem = base + off_exem;
    int32_t *didx = (int32_t *)(base + off_idx);
    double *acc = (double *)(base + off_acc);
    uint8_t *dbad = (uint8_t *)(base + off_bad);
    float *dout = (float *)(base + off_out);
    char *work = base + off_work;
    float *partials = (float *)(work + L.off_partials);
    void *tiles = work + L.off_tiles;

    StreamedState *ss = nullptr;
    if (streamed_state(&ss) != hipSuccess) return EXEMCL_EDEVICE;
    // The copy stream writes the row buffers only after the work already
    // queued on `st` (which may still use this temporary memory).
    hipError_t e = hipEventRecord(ss->freed[0], st);
    if (e == hipSuccess) e = hipEventRecord(ss->freed[1], st);

    // Row block b into device buffer b % 2 on the copy stream, once the
    // kernels of block b - 2 have released it.
    const int64_t nblocks = (n + R - 1) / R;
    auto issue_copy = [&](int64_t b) -> hipError_t {
        const int i = (int)(b & 1);
        const int64_t r0 = b * R, rows = std::min(R, n - r0);
        const void *src = (const char *)V + r0 * d * es;
        if (!direct) {
            // The pinned buffer of block b - 2 must have reached the device.
            if (b >= 2) {
                const hipError_t es1 = hipEventSynchronize(ss->copied[i]);
                if (es1 != hipSuccess) return es1;
            }
            copy_rows(g_pin_rows[i].p, ld, src, d, rows, es);
            src = g_pin_rows[i].p;
        }
        hipError_t ec = hipStreamWaitEvent(ss->cs, ss->freed[i], 0);
        if (ec == hipSuccess) ec = hipMemcpyAsync(drows[i], src, (size_t)(rows * ld * es), hipMemcpyHostToDevice, ss->cs);
        if (ec == hipSuccess) ec = hipEventRecord(ss->copied[i], ss->cs);
        return ec;
    };
    // The first two blocks travel while the host gathers the exemplars.
    for (int64_t b = 0; b < std::min<int64_t>(2, nblocks) && e == hipSuccess; ++b) e = issue_copy(b);

    // Host side of the gather: exemplar rows (zero-padded to ld), indices
    // remapped into the compact matrix, and the sets with an invalid index.
    char *E = (char *)g_pin_exem.p;
    int32_t *ridx = (int32_t *)g_pin_idx.p;
    uint8_t *bad = (uint8_t *)g_pin_bad.p;
    auto gather = [&](int64_t j0, int64_t j1) {
        for (int64_t j = j0; j < j1; ++j) {
            bad[j] = 0;
            for (int64_t p = 0; p < k; ++p) {
                const int64_t i = j * k + p;
                const int32_t idx = sets[i];
                char *row = E + i * ld * es;
                if (idx == kEmptySlot || idx < 0 || idx >= n) {
                    if (idx != kEmptySlot) bad[j] = 1;
                    ridx[i] = kEmptySlot;
                    memset(row, 0, (size_t)(ld * es));
                } else {
                    ridx[i] = (int32_t)i;
                    memcpy(row, (const char *)V + (int64_t)idx * d * es, (size_t)(d * es));
                    if (ld > d) memset(row + d * es, 0, (size_t)((ld - d) * es));
                }
            }
        }
    };
    {
        const unsigned hw = std::max(1u, std::thread::hardware_concurrency());
        const int64_t nt = std::min<int64_t>(std::min<int64_t>(16, hw), std::max<int64_t>(1, ne / 2048));
        if (nt <= 1) {
            gather(0, l);
        } else {
            std::vector<std::thread> th;
            for (int64_t t = 0; t < nt; ++t) th.emplace_back(gather, l * t / nt, l * (t + 1) / nt);
            for (auto &x : th) x.join();
        }
    }

    if (e == hipSuccess) e = hipMemcpyAsync(dexem, E, (size_t)(ne * ld * es), hipMemcpyHostToDevice, st);
    if (e == hipSuccess) e = hipMemcpyAsync(didx, ridx, (size_t)(ne * 4), hipMemcpyHostToDevice, st);
    if (e == hipSuccess) e = hipMemcpyAsync(dbad, bad, (size_t)l, hipMemcpyHostToDevice, st);
    if (e == hipSuccess) e = launch_pack(precision, mp, dexem, std::max<int64_t>(ne, 1), (int)ld, didx, l, k, tiles, st);
    for (int64_t b = 0; b < nblocks && e == hipSuccess; ++b) {
        const int i = (int)(b & 1);
        const int64_t rows = std::min(R, n - b * R);
        e = hipStreamWaitEvent(st, ss->copied[i], 0);
        Layout Lb;
        if (e == hipSuccess && !layout_eval(rows, d, l, k, precision, EXEMCL_PATH_MFMA, &Lb)) e = hipErrorInvalidValue;
        if (e == hipSuccess) {
            ProfRange pr(st);
            e = launch_mfma(precision, MODE_SUM, mp, drows[i], rows, (int)ld, tiles, mfma_tiles_per_group(mp, k),
                            Lb.ngroups, Lb.gpc, nullptr, partials, Lb.lpad, nullptr, st, pr.a, pr.b);
            if (e == hipSuccess) pr.end();
        }
        if (e == hipSuccess) e = launch_accum(partials, Lb.G, Lb.lpad, l, b == 0, acc, st);
        if (e == hipSuccess) e = hipEventRecord(ss->freed[i], st);
        if (e == hipSuccess && b + 2 < nblocks) e = issue_copy(b + 2);
    }
    if (e == hipSuccess) e = launch_finish(acc, dbad, l, n, dout, st);
    if (e == hipSuccess) e = hipMemcpyAsync(out, dout, (size_t)(l * 4), hipMemcpyDeviceToHost, st);
    const hipError_t es2 = hipStreamSynchronize(st);
    if (e == hipSuccess) e = es2;
    (void)hipStreamSynchronize(ss->cs);
    return status_of(e);
}

// ---------------------------------------------------------------------------
// Fixed device scratch of exemplar_eval_noalloc: one array per GPU, part of
// the library's code object, so no call has to allocate.  Host code never
// uses the array's name as an address (on the host it is only a stand-in for
// the symbol): the device address is looked up once per device and kept.
// ---------------------------------------------------------------------------
static __device__ __align__(256) unsigned char scratch[EXEMCL_SCRATCH_BYTES];

std::mutex g_scratch_mu;
void *g_scratch_ptr[64] = {};

// Device address of the current device's scratch array (looked up on the
// first call on that device, with that device current).
int scratch_arena(Arena *a) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) {
        (void)hipGetLastError();
        return EXEMCL_EDEVICE;
    }
    if (dev < 0 || dev >= 64) return EXEMCL_EDEVICE;
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p) {
            (void)hipGetLastError();
            return EXEMCL_EDEVICE;
        }
        g_scratch_ptr[dev] = p;
    }
    a->base = (char *)g_scratch_ptr[dev];
    a->cap = EXEMCL_SCRATCH_BYTES;
    a->used = 0;
    return EXEMCL_OK;
}

}  // namespace

extern "C" {

EXEMCL_API int exemplar_eval(const void *V, int64_t n, int64_t d, const int32_t *sets, int64_t l, int64_t k,
                             int precision, float *out, void *stream) {
    int rc = check_common(V, n, d, l, k, out);
    if (rc) return rc;
    if (!prec_ok(precision)) return EXEMCL_EINVAL;
    if (l > 0 && k > 0 && !sets) return EXEMCL_EINVAL;
    if (l > 0 && k > 0 && choose_path(d, k, precision) == EXEMCL_PATH_NONE) return EXEMCL_EINVAL;
    return run_eval(V, n, d, sets, l, k, precision, nullptr, nullptr, 0, out, (hipStream_t)stream);
}

EXEMCL_API int exemplar_eval_noalloc(const void *V, int64_t n, int64_t d, const int32_t *sets, int64_t l,
                                     int64_t k, int precision, float *out, void *stream) {
    int rc = check_common(V, n, d, l, k, out);
    if (rc) return rc;
    if (!prec_ok(precision)) return EXEMCL_EINVAL;
    if (l > 0 && k > 0 && !sets) return EXEMCL_EINVAL;
    if (l > 0 && k > 0 && choose_path(d, k, precision) == EXEMCL_PATH_NONE) return EXEMCL_EINVAL;
    if (l == 0) return EXEMCL_OK;
    Arena a;
    rc = scratch_arena(&a);
    if (rc) return rc;
    rc = run_eval(V, n, d, sets, l, k, precision, nullptr, nullptr, 0, out, (hipStream_t)stream, nullptr, 0, &a);
    return rc == EXEMCL_ENOMEM ? EXEMCL_ESCRATCH : rc;
}

EXEMCL_API int exemplar_eval_streamed(const void *V, int64_t n, int64_t d, const int32_t *sets, int64_t l,
                                      int64_t k, int precision, int64_t rows_per_block, float *out,
                                      void *stream) {
    int rc = check_common(V, n, d, l, k, out);
    if (rc) return rc;
    if (!prec_ok(precision)) return EXEMCL_EINVAL;
    if (l > 0 && k > 0 && !sets) return EXEMCL_EINVAL;
    if (rows_per_block < 0) return EXEMCL_EINVAL;
    MfmaPlan mp;
    if (!mfma_plan(precision, d, &mp)) return EXEMCL_EINVAL;
    if (l == 0) return EXEMCL_OK;
    if (k == 0) {  // f(empty) = 0 for every set
        memset(out, 0, (size_t)l * sizeof(float));
        return EXEMCL_OK;
    }
    return run_streamed(V, n, d, sets, l, k, precision, rows_per_block, out, (hipStream_t)stream);
}

EXEMCL_API int exemplar_gain(const float *V, int64_t n, int64_t d, const int32_t *S, int64_t k,
                             const int32_t *cands, int64_t l, float *out, void *stream) {
    int rc = check_common(V, n, d, l, k, out);
    if (rc) return rc;
    if (k > 0 && !S) return EXEMCL_EINVAL;
    if (l > 0 && !cands) return EXEMCL_EINVAL;
    MfmaPlan mp;
    if (!mfma_plan(EXEMCL_FP32, d, &mp)) return EXEMCL_EINVAL;
    if (l == 0) return EXEMCL_OK;
    hipStream_t st = (hipStream_t)stream;
    if (k == 0) return run_eval(V, n, d, cands, l, 1, EXEMCL_FP32, nullptr, nullptr, 0, out, st);

    // Cache g(v) = max(0, max_{s in S} h_s(v)): S's members as single-member
    // "sets" staged side by side, reduced by max over columns per point.
    const int64_t tm = mp.tile;
    const int64_t ngroups = (k + tm - 1) / tm;
    const int64_t off_tiles = align_up(n * 4, 256);
    const int64_t bytes = align_up(off_tiles + ngroups * tile_bytes(mp), 256);
    if (bytes + pad_bytes(EXEMCL_FP32, n, d) > workspace_limit()) return EXEMCL_ENOMEM;
    MfmaRows rows;
    rc = prepare_rows(V, n, d, EXEMCL_FP32, st, &rows);
    if (rc) return rc;
    Scratch ws;
    rc = alloc_scratch(&ws, bytes, st);
    if (rc) return rc;
    char *base = (char *)ws.ptr;
    float *gcache = (float *)base;
    void *tiles = base + off_tiles;
    hipError_t e = launch_pack(EXEMCL_FP32, mp, rows.V, n, (int)rows.ld, S, k, 1, tiles, st);
    if (e == hipSuccess)
        e = launch_mfma(EXEMCL_FP32, MODE_ROWMAX, mp, rows.V, n, (int)rows.ld, tiles, 1, ngroups, ngroups, nullptr,
                        nullptr, 0, gcache, st);
    if (e != hipSuccess) return EXEMCL_EDEVICE;
    // Score every S u {c}: single-member sets {c} with the running max
    // started at g(v) instead of e0's 0.
    return run_eval(V, n, d, cands, l, 1, EXEMCL_FP32, gcache, S, k, out, st, &rows, rows.bytes + bytes);
}

EXEMCL_API int exemplar_greedy(const float *V, int64_t n, int64_t d, int64_t K, int32_t *S_out, float *f_out,
                               void *stream) {
    if (!V || n < 1 || n > INT32_MAX || d < 1 || d > INT32_MAX) return EXEMCL_EINVAL;
    if (K < 0 || K > n) return EXEMCL_EINVAL;
    if (K > 0 && (!S_out || !f_out)) return EXEMCL_EINVAL;
    MfmaPlan mp;
    if (!mfma_plan(EXEMCL_FP32, d, &mp)) return EXEMCL_EINVAL;
    if (K == 0) return EXEMCL_OK;
    hipStream_t st = (hipStream_t)stream;

    // State kept on the device across rounds: the candidate list V (all of
    // it; taken ones are skipped by the argmax), the taken flags, the cache
    // g(v) double-buffered, the round's scores and one staged tile for the
    // element just added.
    const int64_t nb = argmax_blocks(n);
    const int64_t off_taken = align_up(n * 4, 256);
    const int64_t off_g0 = align_up(off_taken + n, 256);
    const int64_t off_g1 = align_up(off_g0 + n * 4, 256);
    const int64_t off_scores = align_up(off_g1 + n * 4, 256);
    const int64_t off_ctile = align_up(off_scores + n * 4, 256);
    const int64_t off_pval = align_up(off_ctile + tile_bytes(mp), 256);
    const int64_t off_pidx = align_up(off_pval + nb * 4, 256);
    const int64_t fixed = align_up(off_pidx + nb * 4, 256);

    // Candidates are scored in chunks whose temporary memory stays under a
    // fixed size (the same halving as for a batch that does not fit).
    constexpr int64_t kScoringBytes = int64_t(1) << 30;
    const int64_t limit = workspace_limit() - pad_bytes(EXEMCL_FP32, n, d);
    if (limit < fixed) return EXEMCL_ENOMEM;
    MfmaRows rows;
    int rc = prepare_rows(V, n, d, EXEMCL_FP32, st, &rows);
    if (rc) return rc;
    int64_t lc = n;
    Layout L;
    Scratch ws;
    for (;;) {
        if (!layout_eval(n, d, lc, 1, EXEMCL_FP32, EXEMCL_PATH_MFMA, &L)) return EXEMCL_EINVAL;
        const bool small = L.bytes <= kScoringBytes || lc <= mp.tile;
        if (small && fixed + L.bytes <= limit) {
            rc = alloc_scratch(&ws, fixed + L.bytes, st);
            if (rc == EXEMCL_OK) break;
            if (rc != EXEMCL_ENOMEM) return rc;
        }
        if (lc <= mp.tile) return EXEMCL_ENOMEM;
        lc = ((lc + 1) / 2 + mp.tile - 1) / mp.tile * mp.tile;
    }
    char *base = (char *)ws.ptr;
    int32_t *cands = (int32_t *)base;
    uint8_t *taken = (uint8_t *)(base + off_taken);
    float *g_cur = (float *)(base + off_g0), *g_next = (float *)(base + off_g1);
    float *scores = (float *)(base + off_scores);
    void *ctile = base + off_ctile;
    float *pval = (float *)(base + off_pval);
    int32_t *pidx = (int32_t *)(base + off_pidx);
    char *work = base + fixed;

    hipError_t e = launch_greedy_init(cands, taken, g_cur, n, st);
    for (int64_t i = 0; e == hipSuccess && i < K; ++i) {
        // f(S u {c}) for every candidate c, from the cache of S (Section
        // IV-A's greedy multiset, scored as single-member sets).
        for (int64_t j0 = 0; e == hipSuccess && j0 < n; j0 += lc) {
            const int64_t lj = n - j0 < lc ? n - j0 : lc;
            Layout Lj;
            if (!layout_eval(n, d, lj, 1, EXEMCL_FP32, EXEMCL_PATH_MFMA, &Lj)) return EXEMCL_EINVAL;
            e = run_chunk(Lj, work, V, n, d, &rows, cands + j0, lj, 1, EXEMCL_FP32, g_cur, nullptr, 0, scores + j0,
                          st);
        }
        if (e == hipSuccess) e = launch_argmax(scores, taken, n, pval, pidx, S_out + i, f_out + i, st);
        if (i + 1 == K) break;
        // g <- max(g, h_{c*}) with c* read from S_out[i] on the device.
        if (e == hipSuccess) e = launch_pack(EXEMCL_FP32, mp, rows.V, n, (int)rows.ld, S_out + i, 1, 1, ctile, st);
        if (e == hipSuccess)
            e = launch_mfma(EXEMCL_FP32, MODE_ROWMAX, mp, rows.V, n, (int)rows.ld, ctile, 1, 1, 1, g_cur, nullptr, 0,
                            g_next, st);
        std::swap(g_cur, g_next);
    }
    return status_of(e);
}

EXEMCL_API int exemplar_sqnorm(const void *V, int64_t n, int64_t d, int precision, float *q, void *stream) {
    if (!V || !q) return EXEMCL_EINVAL;
    if (n < 1 || n > INT32_MAX || d < 1 || d > INT32_MAX) return EXEMCL_EINVAL;
    if (!prec_ok(precision)) return EXEMCL_EINVAL;
    return status_of(launch_sqnorm(precision, V, n, (int)d, q, (hipStream_t)stream));
}

EXEMCL_API int exemplar_plan(int64_t n, int64_t d, int64_t l, int64_t k, int precision, int *path,
                             int64_t *workspace_bytes) {
    if (n < 1 || n > INT32_MAX || d < 1 || d > INT32_MAX || k < 0 || l < 0 || !prec_ok(precision))
        return EXEMCL_EINVAL;
    int p = (l == 0 || k == 0) ? EXEMCL_PATH_NONE : choose_path(d, k, precision);
    if (l > 0 && k > 0 && p == EXEMCL_PATH_NONE) return EXEMCL_EINVAL;
    Layout L;
    if (!layout_eval(n, d, l, k, precision, p, &L)) return EXEMCL_EINVAL;
    if (path) *path = p;
    if (workspace_bytes) *workspace_bytes = L.bytes + (p == EXEMCL_PATH_MFMA ? pad_bytes(precision, n, d) : 0);
    return EXEMCL_OK;
}

EXEMCL_API int exemplar_prof_enable(int every) {
    if (every < 0) return EXEMCL_EINVAL;
    std::lock_guard<std::mutex> lk(g_prof_mu);
    g_prof_every = every;
    g_prof_calls = 0;
    return EXEMCL_OK;
}

EXEMCL_API int exemplar_prof_read(double *ms_total, int64_t *launches) {
    std::vector<std::pair<hipEvent_t, hipEvent_t>> ev;
    {
        std::lock_guard<std::mutex> lk(g_prof_mu);
        ev.swap(g_prof_events);
    }
    double total = 0.0;
    int rc = EXEMCL_OK;
    for (auto &pr : ev) {
        float ms = 0.0f;
        if (hipEventSynchronize(pr.second) != hipSuccess || hipEventElapsedTime(&ms, pr.first, pr.second) != hipSuccess)
            rc = EXEMCL_EDEVICE;
        total += ms;
        hipEventDestroy(pr.first);
        hipEventDestroy(pr.second);
    }
    if (ms_total) *ms_total = total;
    if (launches) *launches = (int64_t)ev.size();
    return rc;
}

EXEMCL_API const char *exemplar_strerror(int status) {
    switch (status) {
    case EXEMCL_OK: return "success";
    case EXEMCL_EINVAL: return "invalid argument";
    case EXEMCL_ENOMEM: return "temporary device memory unavailable";
    case EXEMCL_EDEVICE: return "HIP runtime or kernel launch failure";
    case EXEMCL_ESCRATCH: return "workspace needed exceeds the fixed no-allocation scratch buffer";
    }
    return "unknown status";
}

EXEMCL_API int exemplar_version(void) { return kVersion; }

}  // extern "C"
