// C-ABI of the dd library: handle management, argument checks, and the
// order in which the device passes of each call run.

#include <atomic>
#include <map>
#include <math.h>
#include <mutex>
#include <unordered_map>
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "dd_internal.h"

namespace dd {
// tiled chain ranking (k_graph.hip)
hipError_t launch_rank_tiles(const dd_graph *g, int32_t *dloc, int32_t *ext, int32_t *xlist,
                             int64_t *xidx, uint32_t *err, hipStream_t s);
}  // namespace dd

namespace {

thread_local char g_err[512] = "";
std::atomic<uint64_t> g_next_id{1};

dd_status fail(dd_status s, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof(g_err), fmt, ap);
    va_end(ap);
    return s;
}

dd_status hip_fail(hipError_t e, const char *what) {
    return fail(e == hipErrorOutOfMemory ? DD_ENOMEM : DD_EHIP, "%s: %s", what,
                hipGetErrorString(e));
}

dd_status map_err_bits(uint32_t e) {
    using namespace dd;
    if (e & ERR_THREAD_RANGE) return fail(DD_EINVAL, "thread_id outside [0, n_threads)");
    if (e & ERR_PREV_RANGE) return fail(DD_EINVAL, "thread_prev outside [-1, n) or naming the task itself");
    if (e & ERR_NEG_TIME) return fail(DD_EINVAL, "negative duration or gap");
    if (e & ERR_PTR_ORDER) return fail(DD_EINVAL, "in_ptr is not non-decreasing");
    if (e & ERR_SRC_RANGE) return fail(DD_EINVAL, "in_src outside [0, n)");
    if (e & ERR_EDGE_CLS) return fail(DD_EINVAL, "edge class >= 64");
    if (e & ERR_SCALE) return fail(DD_EINVAL, "scale with p < 0 or q < 1");
    if (e & ERR_BIG_TIME) return fail(DD_ERANGE, "duration or gap >= 2^62 ns");
    if (e & ERR_PREV_THREAD) return fail(DD_ECHAIN, "thread_prev names a task on another thread");
    if (e & ERR_SUCC) return fail(DD_ECHAIN, "two tasks name the same thread_prev");
    if (e & ERR_HEADS) return fail(DD_ECHAIN, "a thread has more than one first task");
    if (e & ERR_CHAIN_CYCLE) return fail(DD_ECHAIN, "thread order loops");
    if (e & ERR_SELF_LOOP) return fail(DD_ECYCLE, "dependency from a task to itself");
    if (e & ERR_BACK_EDGE) return fail(DD_ECYCLE, "dependency goes backwards along one thread");
    if (e & ERR_KAHN_CYCLE) return fail(DD_ECYCLE, "dependencies plus thread order contain a cycle");
    return DD_OK;
}

template <class T>
hipError_t copy_in(T **dst, const T *src, size_t count, hipStream_t s) {
    hipError_t e = dd::dalloc_n(dst, count, s);
    if (e != hipSuccess) return e;
    if (count == 0) return hipSuccess;
    if (src) return hipMemcpyAsync(*dst, src, count * sizeof(T), hipMemcpyDefault, s);
    return hipMemsetAsync(*dst, 0, count * sizeof(T), s);
}

void free_graph_arrays(dd_graph *g) {
    hipStream_t s = g->stream;
    dd::join_uses(g->uses, s);
    dd::dfree(g->thread_prev, s); dd::dfree(g->thread_id, s); dd::dfree(g->dur, s);
    dd::dfree(g->gap, s); dd::dfree(g->cls, s); dd::dfree(g->rank, s);
    dd::dfree(g->thread_base, s); dd::dfree(g->order, s); dd::dfree(g->xin_ptr, s);
    dd::dfree(g->xin_src, s); dd::dfree(g->xin_cls, s);
    dd::free_event_lists(&g->ev, s);
}

void free_sched_arrays(dd_sched *x) {
    hipStream_t s = x->stream;
    dd::join_uses(x->uses, s);
    dd::dfree(x->step_ptr, s); dd::dfree(x->pos_node, s); dd::dfree(x->pos_flags, s);
    dd::dfree(x->pos_dur, s); dd::dfree(x->pos_gap, s); dd::dfree(x->pos_cls, s);
    dd::dfree(x->gat_ptr, s); dd::dfree(x->gat_src, s); dd::dfree(x->gat_pos, s);
    dd::dfree(x->gat_cls, s); dd::dfree(x->gat_gap, s); dd::dfree(x->node_step, s);
    dd::dfree(x->gat_spos, s); dd::dfree(x->rec, s);
}

}  // namespace

namespace dd {

// Device memory cache.  Released blocks wait in a free list keyed by
// (device, stream) and serve later requests on that stream only: work on
// one stream runs in order, so a block released there can be handed out
// again at once.  A cached block serves a request of up to its size and at
// least half of it.  New blocks come from hipMalloc; when that fails, every
// cached block of the device is returned and the allocation retried.
namespace {

struct CacheKey {
    int dev;
    hipStream_t s;
    bool operator<(const CacheKey &o) const { return dev != o.dev ? dev < o.dev : s < o.s; }
};
struct LiveBlock {
    size_t bytes;
    int dev;
};

std::mutex g_mu;
std::map<CacheKey, std::multimap<size_t, void *>> g_free;
std::unordered_map<void *, LiveBlock> g_live;

void release_cached(int dev) {   // caller holds g_mu; dev is the current device
    (void)hipDeviceSynchronize();  // work queued before a release may still read a block
    for (auto it = g_free.begin(); it != g_free.end();) {
        if (it->first.dev == dev) {
            for (auto &b : it->second) (void)hipFree(b.second);
            it = g_free.erase(it);
        } else {
            ++it;
        }
    }
}

}  // namespace

hipError_t dalloc(void **p, size_t bytes, hipStream_t s) {
    *p = nullptr;
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    bytes = (bytes + 511) & ~(size_t)511;
    if (bytes == 0) bytes = 512;
    std::lock_guard<std::mutex> lk(g_mu);
    auto fit = g_free.find(CacheKey{dev, s});
    if (fit != g_free.end()) {
        auto it = fit->second.lower_bound(bytes);
        if (it != fit->second.end() && it->first / 2 <= bytes) {
            *p = it->second;
            g_live[*p] = LiveBlock{it->first, dev};
            fit->second.erase(it);
            return hipSuccess;
        }
    }
    e = hipMalloc(p, bytes);
    if (e == hipErrorOutOfMemory) {
        (void)hipGetLastError();
        release_cached(dev);
        e = hipMalloc(p, bytes);
    }
    if (e != hipSuccess) {
        *p = nullptr;
        return e;
    }
    g_live[*p] = LiveBlock{bytes, dev};
    return hipSuccess;
}

void dfree(void *p, hipStream_t s) {
    if (!p) return;
    std::lock_guard<std::mutex> lk(g_mu);
    auto it = g_live.find(p);
    if (it == g_live.end()) return;
    g_free[CacheKey{it->second.dev, s}].emplace(it->second.bytes, p);
    g_live.erase(it);
}

hipError_t release_cache() {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    std::lock_guard<std::mutex> lk(g_mu);
    release_cached(dev);
    return hipGetLastError();
}

hipError_t note_use(ForeignUses &u, hipStream_t own, hipStream_t s) {
    if (s == own) return hipSuccess;
    std::lock_guard<std::mutex> lk(u.mu);
    hipEvent_t ev = nullptr;
    for (auto &x : u.ev)
        if (x.first == s) ev = x.second;
    if (!ev) {
        hipError_t e = hipEventCreateWithFlags(&ev, hipEventDisableTiming);
        if (e != hipSuccess) return e;
        u.ev.emplace_back(s, ev);
    }
    // re-recording keeps the latest use: earlier work on s precedes it
    return hipEventRecord(ev, s);
}

void join_uses(ForeignUses &u, hipStream_t own) {
    std::lock_guard<std::mutex> lk(u.mu);
    for (auto &x : u.ev) {
        (void)hipStreamWaitEvent(own, x.second, 0);
        (void)hipEventDestroy(x.second);
    }
    u.ev.clear();
}

namespace {
// this host thread's pinned buffer of at least `bytes`; a buffer that is
// outgrown is kept (a copy queued earlier may still target it)
char *stage_buf(size_t bytes, hipError_t *e) {
    thread_local char *buf = nullptr;
    thread_local size_t cap = 0;
    *e = hipSuccess;
    if (bytes > cap) {
        size_t c = cap ? cap : 4096;
        while (c < bytes) c *= 2;
        char *nb = nullptr;
        *e = hipHostMalloc(reinterpret_cast<void **>(&nb), c, hipHostMallocDefault);
        if (*e != hipSuccess) return nullptr;
        buf = nb;
        cap = c;
    }
    return buf;
}
}  // namespace

ReadBack::ReadBack(hipStream_t s, size_t cap) : s_(s) {
    cap_ = cap + 8 * 16;                  // room for aligning up to 16 items
    buf_ = stage_buf(cap_, &err_);
}

hipError_t ReadBack::add(void *dst, const void *src, size_t n) {
    if (err_ != hipSuccess) return err_;
    const size_t off = (used_ + 7) & ~size_t(7);
    if (off + n > cap_) return err_ = hipErrorInvalidValue;
    err_ = hipMemcpyAsync(buf_ + off, src, n, hipMemcpyDefault, s_);
    if (err_ == hipSuccess) {
        items_.push_back(Item{dst, off, n});
        used_ = off + n;
    }
    return err_;
}

hipError_t ReadBack::finish() {
    if (err_ == hipSuccess) err_ = hipStreamSynchronize(s_);
    if (err_ == hipSuccess)
        for (const Item &it : items_) memcpy(it.dst, buf_ + it.off, it.n);
    items_.clear();
    used_ = 0;
    return err_;
}

}  // namespace dd

#define TRY(x, what)                                           \
    do {                                                       \
        hipError_t e_ = (x);                                   \
        if (e_ != hipSuccess) { st = hip_fail(e_, what); goto fail_out; } \
    } while (0)

extern "C" {

const char *dd_status_str(dd_status s) {
    // callers may pass any integer: read it as one, not as the enum
    int code;
    memcpy(&code, &s, sizeof(code));
    switch (code) {
        case DD_OK: return "DD_OK";
        case DD_EINVAL: return "DD_EINVAL";
        case DD_ECYCLE: return "DD_ECYCLE";
        case DD_ECHAIN: return "DD_ECHAIN";
        case DD_ERANGE: return "DD_ERANGE";
        case DD_ENOMEM: return "DD_ENOMEM";
        case DD_EHIP: return "DD_EHIP";
        case DD_EMISMATCH: return "DD_EMISMATCH";
        case DD_ELIMIT: return "DD_ELIMIT";
    }
    return "DD_UNKNOWN";
}

const char *dd_last_error(void) { return g_err; }

dd_status dd_graph_load(int32_t n, int32_t n_threads, const int64_t *in_ptr, const int32_t *in_src,
                        const uint8_t *edge_cls, const int32_t *thread_prev,
                        const int32_t *thread_id, const int64_t *dur_ns, const int64_t *gap_ns,
                        const uint16_t *node_cls, void *stream, dd_graph **out) {
    return dd_graph_load_ex(n, n_threads, in_ptr, in_src, edge_cls, thread_prev, thread_id,
                            dur_ns, gap_ns, node_cls, 0u, stream, out);
}

dd_status dd_graph_load_ex(int32_t n, int32_t n_threads, const int64_t *in_ptr,
                           const int32_t *in_src, const uint8_t *edge_cls,
                           const int32_t *thread_prev, const int32_t *thread_id,
                           const int64_t *dur_ns, const int64_t *gap_ns, const uint16_t *node_cls,
                           uint32_t flags, void *stream, dd_graph **out) {
    g_err[0] = 0;
    if (!out) return fail(DD_EINVAL, "out is NULL");
    *out = nullptr;
    if (flags & ~DD_LOAD_SHARED_THREADS) return fail(DD_EINVAL, "unknown load flags 0x%x", flags);
    if (n < 0) return fail(DD_EINVAL, "n < 0");
    if (n_threads < 1) return fail(DD_EINVAL, "n_threads < 1");
    if (!in_ptr) return fail(DD_EINVAL, "in_ptr is NULL");
    if (n > 0 && (!thread_prev || !thread_id || !dur_ns || !gap_ns))
        return fail(DD_EINVAL, "thread_prev, thread_id, dur_ns and gap_ns are required");
    hipStream_t s = (hipStream_t)stream;
    dd_status st = DD_OK;
    dd_graph *g = new dd_graph();
    g->n = n;
    g->n_threads = n_threads;
    g->shared = (flags & DD_LOAD_SHARED_THREADS) != 0;
    g->stream = s;
    g->id = g_next_id.fetch_add(1);
    (void)hipGetDevice(&g->device);
    int64_t *d_in_ptr = nullptr, *cnt = nullptr, *len = nullptr;
    int32_t *d_in_src = nullptr, *succ = nullptr, *heads = nullptr, *nxt = nullptr,
            *nxt2 = nullptr, *rank2 = nullptr;
    uint8_t *d_ecls = nullptr;
    uint32_t *err = nullptr;
    dd::LoadStats *stats = nullptr;
    int64_t ends[2] = {0, 0};
    uint32_t h_err = 0;
    uint32_t h_err2[2] = {0u, 0u};     // error bits; too many tile exits for the tiled ranking
    dd::LoadStats hs{};
    const size_t N1 = (size_t)n + 1;
    int64_t E = 0;

    TRY(copy_in(&d_in_ptr, in_ptr, N1, s), "copy in_ptr");
    {
        dd::ReadBack rb(s, 2 * sizeof(int64_t));
        TRY(rb.add(&ends[0], d_in_ptr, sizeof(int64_t)), "read in_ptr");
        TRY(rb.add(&ends[1], d_in_ptr + n, sizeof(int64_t)), "read in_ptr");
        TRY(rb.finish(), "sync");
    }
    if (ends[0] != 0) { st = fail(DD_EINVAL, "in_ptr[0] != 0"); goto fail_out; }
    E = ends[1];
    if (E < 0 || E >= (int64_t(1) << 31)) { st = fail(DD_EINVAL, "edge count outside [0, 2^31)"); goto fail_out; }
    if (E > 0 && !in_src) { st = fail(DD_EINVAL, "in_src is NULL"); goto fail_out; }
    g->n_edges = E;
    TRY(copy_in(&d_in_src, in_src, (size_t)E, s), "copy in_src");
    TRY(copy_in(&d_ecls, edge_cls, (size_t)E, s), "copy edge_cls");
    TRY(copy_in(&g->thread_prev, thread_prev, (size_t)n, s), "copy thread_prev");
    TRY(copy_in(&g->thread_id, thread_id, (size_t)n, s), "copy thread_id");
    TRY(copy_in(&g->dur, dur_ns, (size_t)n, s), "copy dur");
    TRY(copy_in(&g->gap, gap_ns, (size_t)n, s), "copy gap");
    TRY(copy_in(&g->cls, node_cls, (size_t)n, s), "copy node_cls");
    TRY(copy_in(&succ, (const int32_t *)nullptr, (size_t)n, s), "alloc");
    TRY(copy_in(&heads, (const int32_t *)nullptr, (size_t)n_threads, s), "alloc");
    TRY(copy_in(&err, (const uint32_t *)nullptr, 2, s), "alloc");
    TRY(copy_in(&stats, (const dd::LoadStats *)nullptr, 1, s), "alloc");
    // the edge pass and the chain ranking clamp every index they follow, so
    // the per-task errors are read together with theirs (invalid-input bits
    // take precedence in map_err_bits)
    if (n > 0) TRY(dd::launch_validate_nodes(g, d_in_ptr, succ, heads, err, stats, s), "validate");
    if (n > 0) TRY(dd::launch_validate_edges(g, d_in_ptr, d_in_src, edge_cls ? d_ecls : nullptr, succ, err, s), "validate edges");
    TRY(dd::dalloc_n(&g->rank, N1, s), "alloc rank");
    TRY(dd::dalloc_n(&nxt, N1, s), "alloc");
    TRY(dd::dalloc_n(&nxt2, N1, s), "alloc");
    TRY(dd::dalloc_n(&rank2, N1, s), "alloc");
    TRY(dd::dalloc_n(&cnt, N1, s), "alloc");
    if (n > 0) TRY(dd::launch_rank_tiles(g, nxt, nxt2, rank2, cnt, err, s), "rank chains");
    {
        dd::ReadBack rb(s, sizeof(h_err2));
        TRY(rb.add(h_err2, err, sizeof(h_err2)), "read err");
        TRY(rb.finish(), "sync");
    }
    if (h_err2[1] && !h_err2[0]) {
        // more tile exits than one workgroup ranks: plain pointer jumping
        TRY(dd::launch_rank_chains(g, succ, nxt, nxt2, rank2, err, s), "rank chains");
        dd::ReadBack rb(s, sizeof(uint32_t));
        TRY(rb.add(h_err2, err, sizeof(uint32_t)), "read err");
        TRY(rb.finish(), "sync");
    }
    h_err = h_err2[0];
    if (h_err) { st = map_err_bits(h_err); goto fail_out; }
    if (g->shared) {
        // several chains per thread: no thread-major order and no dropped
        // edges; every dependency edge stays for the schedule-rule path
        g->xin_ptr = d_in_ptr; d_in_ptr = nullptr;
        g->xin_src = d_in_src; d_in_src = nullptr;
        g->xin_cls = d_ecls; d_ecls = nullptr;
        g->n_cross = E;
        dd::ReadBack rb(s, sizeof(hs));
        TRY(rb.add(&hs, stats, sizeof(hs)), "read stats");
        TRY(rb.finish(), "sync");
    } else {
        TRY(dd::dalloc_n(&g->thread_base, (size_t)n_threads + 1, s), "alloc");
        TRY(dd::dalloc_n(&len, (size_t)n_threads + 1, s), "alloc");
        TRY(dd::dalloc_n(&g->order, N1, s), "alloc");
        TRY(dd::launch_build_order(g, succ, len, s), "order");
        TRY(dd::dalloc_n(&g->xin_ptr, N1, s), "alloc");
        if (n > 0) {
            TRY(dd::launch_cross_edges(g, d_in_ptr, d_in_src, edge_cls ? d_ecls : nullptr, cnt, err, stats, s), "cross edges");
        } else {
            TRY(hipMemsetAsync(g->xin_ptr, 0, sizeof(int64_t), s), "memset");
        }
        // cross-edge lists sized by the edge count (an upper bound), so they are
        // filled before the one read-back of the counts and error bits
        TRY(dd::dalloc_n(&g->xin_src, (size_t)E + 1, s), "alloc");
        TRY(dd::dalloc_n(&g->xin_cls, (size_t)E + 1, s), "alloc");
        if (n > 0) TRY(dd::launch_cross_fill(g, d_in_ptr, d_in_src, edge_cls ? d_ecls : nullptr, s), "cross fill");
        dd::ReadBack rb(s, sizeof(uint32_t) + sizeof(int64_t) + sizeof(hs));
        TRY(rb.add(&h_err, err, sizeof(uint32_t)), "read err");
        TRY(rb.add(&g->n_cross, g->xin_ptr + n, sizeof(int64_t)), "read");
        TRY(rb.add(&hs, stats, sizeof(hs)), "read stats");
        TRY(rb.finish(), "sync");
    }
    if (h_err) { st = map_err_bits(h_err); goto fail_out; }
    g->dsum = ((__int128)hs.dsum_hi << 32) + (__int128)hs.dsum_lo;
    {
        const __int128 gs = ((__int128)hs.gsum_hi << 32) + (__int128)hs.gsum_lo;
        g->gsum = gs >= ((__int128)1 << 62) ? ((int64_t)1 << 62) : (int64_t)gs;
    }
    g->dmax = (int64_t)hs.dmax;
    g->gmax = (int64_t)hs.gmax;
    g->max_cls = (int32_t)hs.cls_max;
    g->cross_mask = hs.cross_mask;
    if (g->dsum + (__int128)g->gsum >= ((__int128)1 << 62)) {
        st = fail(DD_ERANGE, "sum of durations and gaps reaches 2^62 ns");
        goto fail_out;
    }
    TRY(hipStreamSynchronize(s), "sync");
    dd::dfree(d_in_ptr, s); dd::dfree(d_in_src, s); dd::dfree(d_ecls, s); dd::dfree(succ, s);
    dd::dfree(heads, s); dd::dfree(err, s); dd::dfree(stats, s); dd::dfree(nxt, s);
    dd::dfree(nxt2, s); dd::dfree(rank2, s); dd::dfree(cnt, s); dd::dfree(len, s);
    *out = g;
    return DD_OK;
fail_out:
    (void)hipStreamSynchronize(s);
    dd::dfree(d_in_ptr, s); dd::dfree(d_in_src, s); dd::dfree(d_ecls, s); dd::dfree(succ, s);
    dd::dfree(heads, s); dd::dfree(err, s); dd::dfree(stats, s); dd::dfree(nxt, s);
    dd::dfree(nxt2, s); dd::dfree(rank2, s); dd::dfree(cnt, s); dd::dfree(len, s);
    free_graph_arrays(g);
    delete g;
    return st;
}

dd_status dd_levelize(const dd_graph *g, uint64_t active_edge_classes, int32_t mode, void *stream,
                      dd_sched **out, int64_t *n_steps_out) {
    g_err[0] = 0;
    if (!out) return fail(DD_EINVAL, "out is NULL");
    *out = nullptr;
    if (!g) return fail(DD_EINVAL, "graph is NULL");
    if (mode != DD_LEVELS && mode != DD_PHASES) return fail(DD_EINVAL, "mode must be DD_LEVELS or DD_PHASES");
    if (g->shared)
        return fail(DD_EINVAL, "the graph was loaded with shared threads: simulate it with dd_simulate_policy");
    hipStream_t s = (hipStream_t)stream;
    dd_sched *x = new dd_sched();
    x->graph_id = g->id;
    x->stream = s;
    char msg[256] = "";
    dd_status st = dd::levelize_device(g, active_edge_classes, mode, x, s, msg, sizeof(msg));
    if (st != DD_OK) {
        fail(st, "%s", msg);
        (void)hipStreamSynchronize(s);
        free_sched_arrays(x);
        delete x;
        return st;
    }
    if (hipError_t e = dd::note_use(g->uses, g->stream, s)) {
        st = hip_fail(e, "record stream use");
        free_sched_arrays(x);
        delete x;
        return st;
    }
    if (n_steps_out) *n_steps_out = x->n_steps;
    *out = x;
    return DD_OK;
}

dd_status dd_apply_transforms(const dd_graph *g, int32_t n_variants, int32_t n_cls,
                              const dd_ratio *scale, const uint32_t *remove_bits,
                              const uint64_t *edge_on, void *stream, dd_variants **out) {
    g_err[0] = 0;
    if (!out) return fail(DD_EINVAL, "out is NULL");
    *out = nullptr;
    if (!g) return fail(DD_EINVAL, "graph is NULL");
    if (n_variants < 1) return fail(DD_EINVAL, "n_variants < 1");
    if (!scale) n_cls = g->max_cls + 1;
    if (n_cls < 1 || n_cls <= g->max_cls)
        return fail(DD_EINVAL, "n_cls (%d) must exceed the largest task class (%d)", n_cls, g->max_cls);
    if ((int64_t)n_cls * n_variants >= (int64_t(1) << 31))
        return fail(DD_EINVAL, "n_cls * n_variants too large");
    hipStream_t s = (hipStream_t)stream;
    dd_status st = DD_OK;
    dd_variants *x = new dd_variants();
    x->graph_id = g->id;
    x->n = g->n;
    x->V = n_variants;
    x->W = (n_variants + 31) / 32;
    x->n_cls = n_cls;
    x->stream = s;
    dd_ratio *d_scale = nullptr;
    uint32_t *err = nullptr;
    uint32_t h_err[6] = {0, 0, 0, 0, 0, 0};
    uint64_t *h_on = nullptr;
    const size_t cv = (size_t)n_cls * n_variants;
    TRY(dd::dalloc_n(&x->table, cv, s), "alloc table");
    if (scale) TRY(copy_in(&d_scale, scale, cv, s), "copy scale");
    TRY(copy_in(&err, (const uint32_t *)nullptr, 6, s), "alloc");
    TRY(dd::launch_build_scale_table(d_scale, n_cls, n_variants, x->table, err, s), "scale table");
    TRY(copy_in(&x->rm_bits, remove_bits, (size_t)g->n * x->W, s), "copy remove_bits");
    TRY(dd::dalloc_n(&x->edge_on, (size_t)n_variants, s), "alloc edge_on");
    h_on = (uint64_t *)malloc(sizeof(uint64_t) * (size_t)n_variants);
    if (!h_on) { st = fail(DD_ENOMEM, "host allocation"); goto fail_out; }
    {
        dd::ReadBack rb(s, sizeof(uint64_t) * (size_t)n_variants + sizeof(h_err));
        if (edge_on) {
            TRY(rb.add(h_on, edge_on, sizeof(uint64_t) * (size_t)n_variants), "read edge_on");
        } else {
            for (int32_t v = 0; v < n_variants; v++) h_on[v] = ~0ull;
        }
        TRY(rb.add(h_err, err, sizeof(h_err)), "read err");
        TRY(rb.finish(), "sync");
    }
    TRY(hipMemcpyAsync(x->edge_on, h_on, sizeof(uint64_t) * (size_t)n_variants, hipMemcpyHostToDevice, s), "copy edge_on");
    x->used_mask = 0;
    x->all_mask = ~0ull;
    for (int32_t v = 0; v < n_variants; v++) {
        x->used_mask |= h_on[v];
        x->all_mask &= h_on[v];
    }
    x->any_magic = h_err[1] != 0;
    if (h_err[0]) { st = map_err_bits(h_err[0]); goto fail_out; }
    {
        uint64_t pmax, rbits;
        memcpy(&pmax, &h_err[2], 8);
        memcpy(&rbits, &h_err[4], 8);
        double rmax;
        memcpy(&rmax, &rbits, 8);
        // d * p must stay below 2^62, and so must every time in the simulation
        if ((__int128)g->dmax * (__int128)pmax >= ((__int128)1 << 62)) {
            st = fail(DD_ERANGE, "largest duration times largest p reaches 2^62");
            goto fail_out;
        }
        long double bound = (long double)g->dsum * (long double)rmax + (long double)g->gsum;
        if (bound >= 4.0e18L) {   // 2^62 = 4.61e18, kept a margin for rounding
            st = fail(DD_ERANGE, "scaled durations could sum past 2^62 ns");
            goto fail_out;
        }
        // every simulated time is a sum of weights along a path, so below
        // the bound; 2^51 = 2.25e15 (a margin for rounding again)
        x->f64_ok = bound < 2.0e15L &&
                    (__int128)g->dmax * (__int128)pmax < ((__int128)1 << 53);
    }
    TRY(hipStreamSynchronize(s), "sync");
    TRY(dd::note_use(g->uses, g->stream, s), "record stream use");
    free(h_on);
    dd::dfree(d_scale, s);
    dd::dfree(err, s);
    *out = x;
    return DD_OK;
fail_out:
    (void)hipStreamSynchronize(s);
    free(h_on);
    dd::dfree(d_scale, s);
    dd::dfree(err, s);
    dd::dfree(x->table, s); dd::dfree(x->rm_bits, s); dd::dfree(x->edge_on, s);
    delete x;
    return st;
}

}  // extern "C"

namespace {

dd_status simulate_impl(const dd_graph *g, const dd_sched *sched, const dd_variants *var,
                        int64_t *d_finish, int64_t *d_start, int64_t *d_makespan, int vs,
                        void *stream) {
    if (!g || !sched || !var) return fail(DD_EINVAL, "NULL handle");
    if (!d_makespan || (!d_finish && g->n > 0))
        return fail(DD_EINVAL, "d_finish and d_makespan are required");
    if (sched->graph_id != g->id || var->graph_id != g->id)
        return fail(DD_EMISMATCH, "handles come from different graphs");
    const uint64_t missing = var->used_mask & g->cross_mask & ~sched->mask;
    if (missing)
        return fail(DD_EMISMATCH, "variants switch on edge classes 0x%llx that the schedule was not built for",
                    (unsigned long long)missing);
    hipStream_t s = (hipStream_t)stream;
    // few variants over few long steps: each step cut across workgroups
    const int sw = vs < 0 ? -vs : vs == 0 ? dd::split_width(sched, var) : 0;
    if (sw > 0 && (int64_t)sched->h_step_ptr.size() != sched->n_steps + 1)
        return fail(DD_EINVAL, "the split path needs a schedule of at most %lld steps (this one has %lld)",
                    (long long)dd::kSplitMaxSteps, (long long)sched->n_steps);
    hipError_t e = sw > 0 ? dd::launch_split(g, sched, var, d_finish, d_start, d_makespan, sw, s)
                          : dd::launch_simulate(g, sched, var, d_finish, d_start, d_makespan, vs, s);
    if (e != hipSuccess) return hip_fail(e, "simulate launch");
    e = dd::note_use(g->uses, g->stream, s);
    if (e == hipSuccess) e = dd::note_use(sched->uses, sched->stream, s);
    if (e == hipSuccess) e = dd::note_use(var->uses, var->stream, s);
    if (e != hipSuccess) return hip_fail(e, "record stream use");
    return DD_OK;
}

}  // namespace

extern "C" {

dd_status dd_simulate_batch(const dd_graph *g, const dd_sched *sched, const dd_variants *var,
                            int64_t *d_finish, int64_t *d_start, int64_t *d_makespan, void *stream) {
    g_err[0] = 0;
    return simulate_impl(g, sched, var, d_finish, d_start, d_makespan, 0, stream);
}

dd_status dd_simulate_batch_vs(const dd_graph *g, const dd_sched *sched, const dd_variants *var,
                               int64_t *d_finish, int64_t *d_start, int64_t *d_makespan,
                               int32_t variants_per_wg, void *stream) {
    g_err[0] = 0;
    const int w = variants_per_wg < 0 ? -variants_per_wg : variants_per_wg;
    if (!(w == 0 || w == 1 || w == 2 || w == 4 || w == 8 || (w == 16 && variants_per_wg > 0)))
        return fail(DD_EINVAL, "variants_per_wg must be 0, 1, 2, 4, 8, 16, -1, -2, -4 or -8 (got %d)",
                    (int)variants_per_wg);
    return simulate_impl(g, sched, var, d_finish, d_start, d_makespan, variants_per_wg, stream);
}

void dd_set_lookback_polls(int32_t polls) { dd::split_set_polls(polls); }

dd_status dd_runtime_breakdown(const dd_graph *g, const dd_variants *var, const uint8_t *role,
                               const int64_t *d_finish, const int64_t *d_makespan,
                               int64_t *d_out, void *stream) {
    g_err[0] = 0;
    if (!g || !var) return fail(DD_EINVAL, "NULL handle");
    if (!d_makespan || !d_out || (g->n > 0 && (!d_finish || !role)))
        return fail(DD_EINVAL, "role, d_finish, d_makespan and d_out are required");
    if (var->graph_id != g->id) return fail(DD_EMISMATCH, "handles come from different graphs");
    if (g->shared)
        return fail(DD_EINVAL, "the graph was loaded with shared threads: its thread order is "
                               "decided by the schedule rule, not recorded");
    hipStream_t s = (hipStream_t)stream;
    dd_status st = DD_OK;
    uint8_t *d_role = nullptr;
    int64_t *scratch = nullptr;
    int32_t *order = nullptr;
    TRY(copy_in(&d_role, role, (size_t)g->n, s), "copy role");
    TRY(dd::dalloc_n(&scratch, 2 * (size_t)var->V + (size_t)var->n_cls + 2, s), "alloc");
    TRY(dd::dalloc_n(&order, 2 * (size_t)g->n + 1, s), "alloc");
    TRY(dd::launch_breakdown(g, var, d_role, d_finish, d_makespan, scratch, order, d_out, s),
        "breakdown");
    TRY(dd::note_use(g->uses, g->stream, s), "record stream use");
    TRY(dd::note_use(var->uses, var->stream, s), "record stream use");
fail_out:
    dd::dfree(d_role, s);
    dd::dfree(scratch, s);
    dd::dfree(order, s);
    return st;
}

dd_status dd_simulate_policy(const dd_graph *g, const dd_variants *var, int32_t policy,
                             const uint8_t *pp, const int32_t *prio, int64_t *d_finish,
                             int64_t *d_start, int64_t *d_makespan, void *stream) {
    g_err[0] = 0;
    if (!g || !var) return fail(DD_EINVAL, "NULL handle");
    if (policy != DD_POLICY_EARLIEST && policy != DD_POLICY_PRIORITY)
        return fail(DD_EINVAL, "policy must be DD_POLICY_EARLIEST or DD_POLICY_PRIORITY");
    if (policy == DD_POLICY_PRIORITY && g->n > 0 && (!pp || !prio))
        return fail(DD_EINVAL, "DD_POLICY_PRIORITY needs pp and prio");
    if (!d_makespan || (!d_finish && g->n > 0))
        return fail(DD_EINVAL, "d_finish and d_makespan are required");
    if (var->graph_id != g->id) return fail(DD_EMISMATCH, "handles come from different graphs");
    if (g->n >= (1 << dd::kEventIdBits))
        return fail(DD_ELIMIT, "the schedule-rule path takes n < 2^%d tasks", dd::kEventIdBits);
    if (g->n_threads > dd::kEventMaxThreads)
        return fail(DD_ELIMIT, "the schedule-rule path takes at most %d threads", dd::kEventMaxThreads);
    if (g->n_cross + (int64_t)g->n >= (int64_t(1) << 31))
        return fail(DD_ELIMIT, "too many edges for the schedule-rule path");
    hipStream_t s = (hipStream_t)stream;
    dd_status st = DD_OK;
    uint8_t *d_pp = nullptr;
    int32_t *d_prio = nullptr, *ref = nullptr;
    int64_t *est = nullptr;
    uint32_t *err = nullptr;
    uint32_t h_err = 0;
    const size_t nv = (size_t)g->n * (size_t)var->V;
    {
        std::lock_guard<std::mutex> lk(g->ev_mu);
        if (!g->ev.rec) {
            hipError_t e = dd::build_event_lists(g, &g->ev, s);
            if (e != hipSuccess) {
                dd::free_event_lists(&g->ev, s);
                return hip_fail(e, "build out-edge lists");
            }
            // the lists belong to the graph and are released on its stream
            e = dd::note_use(g->uses, g->stream, s);
            if (e != hipSuccess) return hip_fail(e, "record stream use");
        }
    }
    if (policy == DD_POLICY_PRIORITY) {
        TRY(copy_in(&d_pp, pp, (size_t)g->n, s), "copy pp");
        TRY(copy_in(&d_prio, prio, (size_t)g->n, s), "copy prio");
    }
    TRY(dd::dalloc_n(&ref, nv, s), "alloc reference counts");
    TRY(dd::dalloc_n(&est, nv, s), "alloc start times");
    TRY(copy_in(&err, (const uint32_t *)nullptr, 1, s), "alloc");
    TRY(dd::launch_sim_event(g, g->ev, var, policy, d_pp, d_prio, ref, est, d_finish, d_start,
                             d_makespan, err, s), "simulate");
    {
        dd::ReadBack rb(s, sizeof(uint32_t));
        TRY(rb.add(&h_err, err, sizeof(uint32_t)), "read err");
        TRY(rb.finish(), "sync");
    }
    TRY(dd::note_use(g->uses, g->stream, s), "record stream use");
    TRY(dd::note_use(var->uses, var->stream, s), "record stream use");
    if (h_err & 2u)
        st = fail(DD_ELIMIT, "more than %d tasks were ready at once in some variant",
                  dd::kEventQueue);
    else if (h_err & 1u)
        st = fail(DD_ECYCLE, "the active dependencies and thread chains contain a cycle");
fail_out:
    dd::dfree(d_pp, s);
    dd::dfree(d_prio, s);
    dd::dfree(ref, s);
    dd::dfree(est, s);
    dd::dfree(err, s);
    return st;
}

dd_status dd_simulate_batch_noalloc(const dd_graph *g, const dd_sched *sched, const dd_variants *var,
                                    int64_t *d_finish, int64_t *d_start, int64_t *d_makespan,
                                    void *stream) {
    g_err[0] = 0;
    if (!g || !sched || !var) return fail(DD_EINVAL, "NULL handle");
    if (!d_makespan || (!d_finish && g->n > 0))
        return fail(DD_EINVAL, "d_finish and d_makespan are required");
    if (sched->graph_id != g->id || var->graph_id != g->id)
        return fail(DD_EMISMATCH, "handles come from different graphs");
    const uint64_t missing = var->used_mask & g->cross_mask & ~sched->mask;
    if (missing)
        return fail(DD_EMISMATCH, "variants switch on edge classes 0x%llx that the schedule was not built for",
                    (unsigned long long)missing);
    size_t need = 0, limit = 0;
    hipError_t e = dd::simulate_noalloc(g, sched, var, d_finish, d_start, d_makespan,
                                        (hipStream_t)stream, &need, &limit);
    if (need > limit)
        return fail(DD_EINVAL, "this batch needs %zu bytes of scratch; the allocation-free entry "
                               "point has %zu (use dd_simulate_batch)", need, limit);
    if (e != hipSuccess) return hip_fail(e, "simulate launch");
    return DD_OK;
}

dd_status dd_release_cache(void) {
    g_err[0] = 0;
    hipError_t e = dd::release_cache();
    if (e != hipSuccess) return hip_fail(e, "release cache");
    return DD_OK;
}

dd_status dd_sched_task_steps(const dd_sched *sched, int32_t *steps_out, void *stream) {
    g_err[0] = 0;
    if (!sched || !steps_out) return fail(DD_EINVAL, "NULL argument");
    hipStream_t s = (hipStream_t)stream;
    if (sched->n == 0) return DD_OK;
    hipError_t e = hipMemcpyAsync(steps_out, sched->node_step, sizeof(int32_t) * (size_t)sched->n,
                                  hipMemcpyDefault, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_fail(e, "copy steps");
    return DD_OK;
}

dd_status dd_simulate_plan(const dd_sched *sched, const dd_variants *var,
                           int32_t *variants_per_wg) {
    g_err[0] = 0;
    if (!sched || !var || !variants_per_wg) return fail(DD_EINVAL, "NULL argument");
    const int sw = dd::split_width(sched, var);
    *variants_per_wg = sw > 0 ? -sw : dd::strip_width(var->V);
    return DD_OK;
}

dd_status dd_sched_info(const dd_sched *sched, int64_t *n_steps, int64_t *n_segments,
                        int64_t *max_step_width, int64_t *n_gathers) {
    g_err[0] = 0;
    if (!sched) return fail(DD_EINVAL, "NULL schedule");
    if (n_steps) *n_steps = sched->n_steps;
    if (n_segments) *n_segments = sched->n_segments;
    if (max_step_width) *max_step_width = sched->max_width;
    if (n_gathers) *n_gathers = sched->n_gathers;
    return DD_OK;
}

void dd_graph_free(dd_graph *g) {
    if (!g) return;
    free_graph_arrays(g);
    delete g;
}

void dd_sched_free(dd_sched *x) {
    if (!x) return;
    free_sched_arrays(x);
    delete x;
}

void dd_variants_free(dd_variants *x) {
    if (!x) return;
    hipStream_t s = x->stream;
    dd::join_uses(x->uses, s);
    dd::dfree(x->table, s);
    dd::dfree(x->rm_bits, s);
    dd::dfree(x->edge_on, s);
    delete x;
}

}  // extern "C"
