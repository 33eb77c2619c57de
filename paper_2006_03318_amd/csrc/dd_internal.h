// Internal declarations shared by the HIP sources of the dd library.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>
#include <utility>
#include <vector>

#include "dd.h"

namespace dd {

// ---------------------------------------------------------------------------
// error bits raised by device-side validation (one 32-bit word per check run)
enum : uint32_t {
    ERR_THREAD_RANGE = 1u << 0,   // thread id outside [0, n_threads)       EINVAL
    ERR_PREV_RANGE = 1u << 1,     // thread_prev outside [-1, n) or == self  EINVAL
    ERR_PREV_THREAD = 1u << 2,    // thread_prev on another thread           ECHAIN
    ERR_NEG_TIME = 1u << 3,       // negative duration or gap                EINVAL
    ERR_BIG_TIME = 1u << 4,       // duration or gap >= 2^62                 ERANGE
    ERR_PTR_ORDER = 1u << 5,      // in_ptr decreasing                       EINVAL
    ERR_SRC_RANGE = 1u << 6,      // in_src outside [0, n)                   EINVAL
    ERR_SELF_LOOP = 1u << 7,      // edge u -> u                             ECYCLE
    ERR_EDGE_CLS = 1u << 8,       // edge class >= 64                        EINVAL
    ERR_SUCC = 1u << 9,           // two tasks name the same thread_prev     ECHAIN
    ERR_HEADS = 1u << 10,         // a thread with two first tasks           ECHAIN
    ERR_CHAIN_CYCLE = 1u << 11,   // thread order loops                      ECHAIN
    ERR_BACK_EDGE = 1u << 12,     // same-thread dependency points backwards ECYCLE
    ERR_KAHN_CYCLE = 1u << 13,    // Kahn rounds stall before the end        ECYCLE
    ERR_SCALE = 1u << 14,         // p < 0 or q < 1                          EINVAL
};

constexpr int64_t kTimeLimit = int64_t(1) << 62;

// Per-(class, variant) shrink/scale entry: floor(d * p / q) evaluated as
// a = d * p; q a power of two: a >> shift; otherwise the high 64 bits of
// a * magic shifted right by `shift` (Granlund & Montgomery, PLDI 1994,
// round-up method; exact for every a < 2^62).
struct alignas(16) ScaleEntry {
    uint64_t magic;   // 0 when q is a power of two
    uint32_t p;
    uint32_t shift;
};

// One schedule position as the simulation reads it: the task, its
// duration, gap and class, and up to two of its gathers inline (source task,
// the source's schedule position, edge class).  Gathers beyond two stay in
// the gather arrays (gat_ptr[q] + 2 onwards).
struct alignas(16) Rec {
    int64_t dur, gap;
    int32_t node, g0_src, g1_src, g0_spos;
    int32_t g1_spos;
    uint32_t cls;     // bits 0..15 task class, 16..23 / 24..31 edge class of gather 0 / 1
    uint32_t flags;   // bit0: first task of a thread run; bit1: last task of a run;
                      // bits 2..7: thread (graphs with at most 64 threads);
                      // bits 8..31: gathers beyond two (saturating)
    uint32_t g0_gap32;  // gap of gather 0's source, low 32 bits (whole when gaps < 2^32)
};
static_assert(sizeof(Rec) == 48, "record size");

// Schedules of at most this many steps keep a host copy of their step
// offsets: the few-variant path launches one kernel per step.
constexpr int64_t kSplitMaxSteps = 512;

// Graphs with at most this many threads keep each thread's latest release in
// LDS during the simulation instead of gathering the previous task of a run.
constexpr int kMaxCarryThreads = 64;

// Streams other than its own on which a handle's device memory was used.
// A handle's blocks go back to the cache of the stream it was created on;
// before that, its own stream waits for the last use on each other stream,
// so a later allocation there cannot overwrite memory a kernel still reads.
struct ForeignUses {
    std::mutex mu;
    std::vector<std::pair<hipStream_t, hipEvent_t>> ev;
};
// record the point after the work just queued on s (no-op when s == own)
hipError_t note_use(ForeignUses &u, hipStream_t own, hipStream_t s);
// make `own` wait for every recorded use; the events are released
void join_uses(ForeignUses &u, hipStream_t own);

// Statistics reduced on the device while loading (hi/lo split sums cannot
// overflow for n < 2^31 values below 2^62).
struct LoadStats {
    unsigned long long dsum_hi, dsum_lo, gsum_hi, gsum_lo;
    unsigned long long dmax, cls_max, cross_mask, gmax;
};

}  // namespace dd

namespace dd {
// Out-edge lists for the task-by-task simulation under a schedule rule:
// every dependency edge and every thread-order link as (child << 8 | class),
// class 255 for thread order (always present), grouped by parent.
struct EventLists {
    int4 *rec = nullptr;        // [n] {first out-edge, out-edge count, thread, task class}
    uint4 *e4 = nullptr;        // [n] the first four out-edges (0 past the count)
    uint32_t *edges = nullptr;  // [n_edges]
    int64_t n_edges = 0;
};
constexpr uint32_t kEdgeAlways = 255;
}  // namespace dd

struct dd_graph {
    int32_t n = 0, n_threads = 0;
    bool shared = false;          // threads may hold several chains (DD_LOAD_SHARED_THREADS);
                                  // then xin_* hold every dependency edge
    int64_t n_edges = 0, n_cross = 0;
    int device = 0;
    hipStream_t stream = nullptr;
    uint64_t id = 0;
    // statistics (host)
    int64_t dmax = 0, gmax = 0, gsum = 0;
    __int128 dsum = 0;
    int32_t max_cls = 0;
    uint64_t cross_mask = 0;      // edge classes present among cross-thread edges
    // device arrays
    int32_t *thread_prev = nullptr, *thread_id = nullptr;
    int64_t *dur = nullptr, *gap = nullptr;
    uint16_t *cls = nullptr;
    int32_t *rank = nullptr;      // position of each task on its thread
    int64_t *thread_base = nullptr;  // [T+1]
    int32_t *order = nullptr;     // [n] tasks thread-major in thread order
    int64_t *xin_ptr = nullptr;   // [n+1] cross-thread in-edges
    int32_t *xin_src = nullptr;
    uint8_t *xin_cls = nullptr;
    mutable dd::ForeignUses uses;
    mutable std::mutex ev_mu;     // guards ev, built on first use
    mutable dd::EventLists ev;
};

struct dd_sched {
    uint64_t graph_id = 0;
    int32_t n = 0, mode = 0;
    uint64_t mask = 0;
    int64_t n_steps = 0, n_segments = 0, max_width = 0, n_gathers = 0;
    hipStream_t stream = nullptr;
    int32_t *step_ptr = nullptr;  // [n_steps+1] position offsets
    int32_t *pos_node = nullptr;  // [n]
    uint8_t *pos_flags = nullptr; // [n] bit0: first task of a thread run
    int64_t *pos_dur = nullptr, *pos_gap = nullptr;
    uint16_t *pos_cls = nullptr;
    int64_t *gat_ptr = nullptr;   // [n+1] per position
    int32_t *gat_src = nullptr;   // source task of each gather
    int32_t *gat_pos = nullptr;   // position it feeds
    uint8_t *gat_cls = nullptr;   // edge class; 255 = always present (thread order)
    int64_t *gat_gap = nullptr;   // gap of the source task
    int32_t *gat_spos = nullptr;  // schedule position of the source task
    int32_t *node_step = nullptr; // [n]
    dd::Rec *rec = nullptr;       // [n] per position
    bool thread_carry = false;    // thread predecessors come from per-thread carries
    std::vector<int32_t> h_step_ptr;  // host copy of step_ptr (schedules of at most
                                      // kSplitMaxSteps steps; empty otherwise)
    mutable dd::ForeignUses uses;
};

struct dd_variants {
    uint64_t graph_id = 0;
    int32_t n = 0, V = 0, W = 0, n_cls = 0;
    uint64_t used_mask = 0;       // OR of edge_on over all variants
    uint64_t all_mask = 0;        // AND of edge_on over all variants
    bool any_magic = false;       // some scale has q not a power of two
    bool f64_ok = false;          // every simulated time below 2^51 and every d * p below
                                  // 2^53: the double form of the time arithmetic is exact
    hipStream_t stream = nullptr;
    dd::ScaleEntry *table = nullptr;  // [n_cls][V]
    uint32_t *rm_bits = nullptr;      // [n][W]
    uint64_t *edge_on = nullptr;      // [V]
    mutable dd::ForeignUses uses;
};

namespace dd {

// Read-backs of small results through a pinned host buffer (one per host
// thread, kept until the process ends).  A copy from the device into
// pageable memory waits for its stream by itself (about 10 us each); into
// pinned memory it is a plain DMA, so the queued copies of one read-back
// cost one synchronization.  cap = the bytes that will be queued.
class ReadBack {
public:
    ReadBack(hipStream_t s, size_t cap);
    // queue a copy of n bytes from src (device or host) into dst
    hipError_t add(void *dst, const void *src, size_t n);
    // wait for the stream, then fill every queued dst
    hipError_t finish();
private:
    struct Item { void *dst; size_t off, n; };
    hipStream_t s_;
    char *buf_ = nullptr;
    size_t cap_ = 0, used_ = 0;
    hipError_t err_ = hipSuccess;
    std::vector<Item> items_;
};

// device memory (cache of blocks kept per device and stream)
hipError_t dalloc(void **p, size_t bytes, hipStream_t s);
void dfree(void *p, hipStream_t s);
// return every cached block of the current device (waits for the device)
hipError_t release_cache();
template <class T>
hipError_t dalloc_n(T **p, size_t count, hipStream_t s) {
    return dalloc(reinterpret_cast<void **>(p), count * sizeof(T) + 16, s);
}

// exclusive prefix sum: out[i] = sum_{j<i} in[j] for i in [0, n]; in/out may alias
hipError_t scan_exclusive(const int64_t *in, int64_t *out, int64_t n, hipStream_t s);
// the same with the caller's temporaries: tmp holds scan_temp_count(n) int64
int64_t scan_temp_count(int64_t n);
hipError_t scan_exclusive_ws(const int64_t *in, int64_t *out, int64_t n, int64_t *tmp,
                             hipStream_t s);

inline int grid_for(int64_t n, int bs) {
    int64_t g = (n + bs - 1) / bs;
    if (g < 1) g = 1;
    if (g > (int64_t(1) << 30)) g = int64_t(1) << 30;
    return (int)g;
}

// graph load kernels (k_graph.hip)
hipError_t launch_validate_nodes(const dd_graph *g, const int64_t *in_ptr, int32_t *succ,
                                 int32_t *heads, uint32_t *err, LoadStats *st, hipStream_t s);
hipError_t launch_validate_edges(const dd_graph *g, const int64_t *in_ptr, const int32_t *in_src,
                                 const uint8_t *edge_cls, const int32_t *succ, uint32_t *err,
                                 hipStream_t s);
hipError_t launch_rank_chains(const dd_graph *g, const int32_t *succ, int32_t *tmp_nxt,
                              int32_t *tmp_nxt2, int32_t *tmp_rank2, uint32_t *err,
                              hipStream_t s);
hipError_t launch_build_order(const dd_graph *g, const int32_t *succ, int64_t *len_tmp,
                              hipStream_t s);
hipError_t launch_cross_edges(dd_graph *g, const int64_t *in_ptr, const int32_t *in_src,
                              const uint8_t *edge_cls, int64_t *cnt_tmp, uint32_t *err,
                              LoadStats *st, hipStream_t s);
hipError_t launch_cross_fill(dd_graph *g, const int64_t *in_ptr, const int32_t *in_src,
                             const uint8_t *edge_cls, hipStream_t s);

// levelization (k_levelize.hip)
struct LevelizeOut {
    int64_t n_steps, n_segments, max_width, n_gathers;
    uint32_t err;
};
dd_status levelize_device(const dd_graph *g, uint64_t mask, int32_t mode, dd_sched *sch,
                          hipStream_t s, char *msg, size_t msg_len);

// transforms (k_transform.hip)
hipError_t launch_build_scale_table(const dd_ratio *scale_dev, int32_t n_cls, int32_t V,
                                    ScaleEntry *table, uint32_t *err, hipStream_t s);

// few-variant simulation (k_split.hip): every step cut across several
// workgroups per variant, one launch per step.  split_width() gives the
// variants per workgroup (1, 2, 4 or 8) when the schedule and variants suit
// it, else 0; launch_split() takes that width.
int split_width(const dd_sched *sch, const dd_variants *var);
// look-back polls of one slot before a lane folds that chunk itself
// (negative: the default)
void split_set_polls(int32_t polls);
hipError_t launch_split(const dd_graph *g, const dd_sched *sch, const dd_variants *var,
                        int64_t *finish, int64_t *start, int64_t *makespan, int vg, hipStream_t s);

// variants per workgroup of the one-workgroup-per-strip kernel when the
// caller leaves it to the library: enough workgroups to cover the 256
// compute units, then the widest rows
inline int strip_width(int64_t V) {
    int vs = 1;
    while (vs < 16 && V / (vs * 2) >= 256) vs *= 2;
    return vs;
}

// simulation (k_simulate.hip)
hipError_t launch_simulate(const dd_graph *g, const dd_sched *sch, const dd_variants *var,
                           int64_t *finish, int64_t *start, int64_t *makespan, int vs_hint,
                           hipStream_t s);
// the same in the library's per-GPU scratch array, allocating nothing:
// *need = bytes this call needs, *limit = the array's size;
// hipErrorInvalidValue when need > limit (nothing launched)
hipError_t simulate_noalloc(const dd_graph *g, const dd_sched *sch, const dd_variants *var,
                            int64_t *finish, int64_t *start, int64_t *makespan, hipStream_t s,
                            size_t *need, size_t *limit);

// runtime breakdown (k_breakdown.hip): scratch [2 * V + n_cls + 1] int64,
// order [n] int32, out [V][4]
hipError_t launch_breakdown(const dd_graph *g, const dd_variants *var, const uint8_t *role_dev,
                            const int64_t *finish, const int64_t *makespan, int64_t *scratch,
                            int32_t *order, int64_t *out, hipStream_t s);

// simulation under a schedule rule (k_event.hip)
// out-edge lists of g (dependencies in xin_*, thread order in thread_prev)
hipError_t build_event_lists(const dd_graph *g, EventLists *ev, hipStream_t s);
void free_event_lists(EventLists *ev, hipStream_t s);
// ref: int32 [V][n], est: int64 [V][n] working memory; err: uint32, zeroed
// by the caller (bit 0: a cycle, bit 1: frontier capacity exceeded)
hipError_t launch_sim_event(const dd_graph *g, const EventLists &ev, const dd_variants *var,
                            int32_t policy, const uint8_t *pp, const int32_t *prio, int32_t *ref,
                            int64_t *est, int64_t *finish, int64_t *start, int64_t *makespan,
                            uint32_t *err, hipStream_t s);
constexpr int kEventQueue = 1024;      // ready tasks one variant may hold
constexpr int kEventIdBits = 22;       // tasks: n < 2^22
constexpr int kEventMaxThreads = 4096;



}  // namespace dd
