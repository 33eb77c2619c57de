// Simulation under an overridden schedule() (Sec. 4.4, "Schedule"; the P3
// model of the appendix).
//
// When a thread holds tasks with no recorded order among them (the push and
// pull slices a what-if recipe puts on a communication channel), the start
// times depend on which ready task schedule() picks, so the max-plus form of
// the batch kernel no longer applies.  This path runs Algorithm 1 task by
// task for every variant: the reference counts, the frontier Q of ready
// tasks, schedule(Q), the thread progress P and the children's start times.
//
// Design (one wavefront per variant, 64 threads per workgroup):
//  * the frontier lives in LDS (up to kEventQueue entries of 18 bytes,
//    structure of arrays): what schedule() reads -- id, push/pull and
//    removal flags, thread, priority, start so far.  The dispatched task's
//    record (out-edges, duration, gap, class) is read when it is picked;
//  * schedule(Q) is a wave reduction: the least time max(P[t], start), then
//    the least id among those (Q is in trace order, so that is Q's first),
//    then, for the priority rule when that task is a push/pull task, the
//    highest priority (least id among equals) over the push/pull tasks of
//    least time -- the task the paper's scan over Q ends with;
//  * the dispatched task's children are handled one per lane: a device
//    atomic decrement of the child's reference count and an atomic max of
//    its start (two edges from one parent, e.g. a dependency that repeats
//    the thread order, stay correct), with the child's metadata loaded at
//    the same time; children whose count reaches zero join Q;
//  * reference counts and starts are per-variant arrays [V][n] in device
//    memory; P for every thread and the variant's scale column (when it has
//    at most kLdsCls classes) sit in LDS.
// Each step is a chain of dependent latencies (LDS, reductions, the picked
// task's record, the children's atomics), so the rate is set by how many
// variants run at once: every variant is one wave of ~20 KB of LDS, eight
// per CU, so about 2,000 variants are resident together.
#include "dd_common.h"
#include "dd_internal.h"

namespace dd {
namespace {

constexpr int kBS = 256;
constexpr int kQ = kEventQueue;
constexpr int kLdsCls = 64;        // scale columns cached in LDS up to this many classes

__device__ __forceinline__ int64_t scaled(int64_t d, const ScaleEntry &se) {
    const uint64_t a = (uint64_t)d * (uint64_t)se.p;
    return (int64_t)(se.magic ? (__umul64hi(a, se.magic) >> se.shift) : (a >> se.shift));
}

// Wave-wide minima: butterflies inside each row of 16 lanes with DPP (quad
// permutations, half-row and row mirrors), then the four row results read
// into scalar registers.  All 64 lanes must be active.
template <int CTRL>
__device__ __forceinline__ uint32_t dpp32(uint32_t x) {
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, CTRL, 0xf, 0xf, false);
}
template <int CTRL>
__device__ __forceinline__ uint64_t dpp64(uint64_t x) {
    const uint32_t lo = dpp32<CTRL>((uint32_t)x);
    const uint32_t hi = dpp32<CTRL>((uint32_t)(x >> 32));
    return ((uint64_t)hi << 32) | lo;
}
__device__ __forceinline__ uint64_t readlane_u64(uint64_t x, int l) {
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)x, l);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(x >> 32), l);
    return ((uint64_t)hi << 32) | lo;
}
template <class T>
__device__ __forceinline__ T tmin(T a, T b) { return b < a ? b : a; }

__device__ __forceinline__ uint64_t wave_min_u64(uint64_t x) {
    x = tmin(x, dpp64<0xB1>(x));     // quad_perm [1,0,3,2]
    x = tmin(x, dpp64<0x4E>(x));     // quad_perm [2,3,0,1]
    x = tmin(x, dpp64<0x141>(x));    // row_half_mirror
    x = tmin(x, dpp64<0x140>(x));    // row_mirror
    return tmin(tmin(readlane_u64(x, 0), readlane_u64(x, 16)),
                tmin(readlane_u64(x, 32), readlane_u64(x, 48)));
}

__device__ __forceinline__ uint32_t wave_min_u32(uint32_t x) {
    x = tmin(x, dpp32<0xB1>(x));
    x = tmin(x, dpp32<0x4E>(x));
    x = tmin(x, dpp32<0x141>(x));
    x = tmin(x, dpp32<0x140>(x));
    const uint32_t a = (uint32_t)__builtin_amdgcn_readlane((int)x, 0);
    const uint32_t b = (uint32_t)__builtin_amdgcn_readlane((int)x, 16);
    const uint32_t c = (uint32_t)__builtin_amdgcn_readlane((int)x, 32);
    const uint32_t d = (uint32_t)__builtin_amdgcn_readlane((int)x, 48);
    return tmin(tmin(a, b), tmin(c, d));
}

__device__ __forceinline__ uint32_t pick4(const uint4 &e, int k) {
    return k == 0 ? e.x : k == 1 ? e.y : k == 2 ? e.z : e.w;
}

// ---------------------------------------------------------------------------
// out-edge lists: count per parent, scan, fill, per-task records
__global__ __launch_bounds__(kBS) void k_ev_count(int32_t n, const int64_t *__restrict__ in_ptr,
                                                  const int32_t *__restrict__ in_src,
                                                  const int32_t *__restrict__ prev,
                                                  unsigned long long *__restrict__ cnt) {
    const int64_t u = (int64_t)blockIdx.x * kBS + threadIdx.x;
    if (u >= n) return;
    for (int64_t e = in_ptr[u]; e < in_ptr[u + 1]; e++) atomicAdd(&cnt[in_src[e]], 1ull);
    if (prev[u] >= 0) atomicAdd(&cnt[prev[u]], 1ull);
}

__global__ __launch_bounds__(kBS) void k_ev_fill(int32_t n, const int64_t *__restrict__ in_ptr,
                                                 const int32_t *__restrict__ in_src,
                                                 const uint8_t *__restrict__ in_cls,
                                                 const int32_t *__restrict__ prev,
                                                 const int64_t *__restrict__ beg,
                                                 unsigned long long *__restrict__ cur,
                                                 uint32_t *__restrict__ edges) {
    const int64_t u = (int64_t)blockIdx.x * kBS + threadIdx.x;
    if (u >= n) return;
    for (int64_t e = in_ptr[u]; e < in_ptr[u + 1]; e++) {
        const int32_t s = in_src[e];
        const int64_t at = beg[s] + (int64_t)atomicAdd(&cur[s], 1ull);
        edges[at] = ((uint32_t)u << 8) | (in_cls ? (uint32_t)in_cls[e] : 0u);
    }
    const int32_t p = prev[u];
    if (p >= 0) {
        const int64_t at = beg[p] + (int64_t)atomicAdd(&cur[p], 1ull);
        edges[at] = ((uint32_t)u << 8) | kEdgeAlways;
    }
}

__global__ __launch_bounds__(kBS) void k_ev_rec(int32_t n, const int64_t *__restrict__ beg,
                                                const int32_t *__restrict__ tid,
                                                const uint16_t *__restrict__ cls,
                                                const uint32_t *__restrict__ edges,
                                                int4 *__restrict__ rec, uint4 *__restrict__ e4) {
    const int64_t u = (int64_t)blockIdx.x * kBS + threadIdx.x;
    if (u >= n) return;
    const int64_t b = beg[u];
    const int32_t k = (int32_t)(beg[u + 1] - b);
    rec[u] = make_int4((int32_t)b, k, tid[u], cls ? (int32_t)cls[u] : 0);
    e4[u] = make_uint4(k > 0 ? edges[b] : 0u, k > 1 ? edges[b + 1] : 0u,
                       k > 2 ? edges[b + 2] : 0u, k > 3 ? edges[b + 3] : 0u);
}

// ---------------------------------------------------------------------------
struct EvArgs {
    int32_t n, V, W, T, n_cls, policy;
    const int4 *__restrict__ rec;
    const uint4 *__restrict__ e4;
    const uint32_t *__restrict__ edges;
    const int64_t *__restrict__ in_ptr;    // dependency in-edges (for the first counts)
    const uint8_t *__restrict__ in_cls;
    const int32_t *__restrict__ tprev;
    const int32_t *__restrict__ tid;
    const int64_t *__restrict__ dur;
    const int64_t *__restrict__ gap;
    const ScaleEntry *__restrict__ table;  // [n_cls][V]
    const uint32_t *__restrict__ rm;       // [n][W]
    const uint64_t *__restrict__ edge_on;  // [V]
    const uint8_t *__restrict__ pp;
    const int32_t *__restrict__ prio;
    int32_t *ref;                          // [V][n]
    unsigned long long *est;               // [V][n] (times >= 0: unsigned order is the order)
    int64_t *finish, *start, *makespan;
    uint32_t *err;
};

// A frontier entry is 18 bytes: what schedule(Q) reads.  The rest of a task
// (out-edges, duration, gap, class) is read when it is dispatched.
constexpr int kSlotBits = 10;
static_assert((1 << kSlotBits) == kQ, "slot bits");
constexpr uint32_t kIdMask = (1u << kEventIdBits) - 1u;
constexpr uint32_t kPPb = 1u << kEventIdBits;          // push/pull task
constexpr uint32_t kRMb = 1u << (kEventIdBits + 1);    // removed in this variant
static_assert(kEventIdBits + kSlotBits <= 32, "id and slot share one word");

struct Frontier {
    uint32_t a[kQ];     // id | flags
    uint16_t th[kQ];    // thread
    int32_t pr[kQ];     // priority
    int64_t est[kQ];    // start so far (final once the task is ready)
};

__device__ __forceinline__ void push_entry(Frontier &q, int32_t slot, uint32_t u, bool ppf,
                                           bool rmv, int32_t th, int32_t pr, int64_t est) {
    q.a[slot] = u | (ppf ? kPPb : 0u) | (rmv ? kRMb : 0u);
    q.th[slot] = (uint16_t)th;
    q.pr[slot] = pr;
    q.est[slot] = est;
}

template <bool TLDS>
__global__ __launch_bounds__(64) void k_sim_event(EvArgs a) {
    extern __shared__ int64_t sP[];           // [T] thread progress
    __shared__ Frontier q;
    __shared__ ScaleEntry sTab[TLDS ? kLdsCls : 1];
    const int lane = threadIdx.x;
    const int v = blockIdx.x;
    const int32_t n = a.n;
    const int64_t V = a.V;
    const uint64_t on = a.edge_on[v];
    int32_t *ref = a.ref + (int64_t)v * n;
    unsigned long long *est = a.est + (int64_t)v * n;
    const uint64_t lt = (1ull << lane) - 1ull;
    const uint32_t vbit = 1u << (v & 31);
    const int vw = v >> 5;

    for (int t = lane; t < a.T; t += 64) sP[t] = 0;
    if (TLDS)
        for (int c = lane; c < a.n_cls; c += 64) sTab[c] = a.table[(int64_t)c * V + v];
    uint32_t err = 0;

    // reference counts over the active parents; tasks with none are ready
    int32_t qn = 0;
    for (int64_t base = 0; base < n; base += 64) {
        const int64_t u = base + lane;
        bool root = false;
        if (u < n) {
            int32_t r = a.tprev[u] >= 0 ? 1 : 0;
            for (int64_t e = a.in_ptr[u]; e < a.in_ptr[u + 1]; e++) {
                const uint32_t c = a.in_cls ? a.in_cls[e] : 0u;
                r += (int32_t)((on >> c) & 1ull);
            }
            ref[u] = r;
            est[u] = 0ull;
            root = r == 0;
        }
        const uint64_t b = __ballot(root);
        if (root) {
            const int32_t slot = qn + __popcll(b & lt);
            if (slot < kQ)
                push_entry(q, slot, (uint32_t)u, a.pp ? a.pp[u] != 0 : false,
                           (a.rm[u * a.W + vw] & vbit) != 0u, a.tid[u], a.prio ? a.prio[u] : 0, 0);
            else
                err |= 2u;
        }
        qn += __popcll(b);
        if (qn > kQ) qn = kQ;
    }
    __threadfence();   // the counts are in memory before the first atomic on them
    __syncthreads();

    int64_t ms = 0;
    int32_t done = 0;
    int32_t bu = 0;                 // this lane's buffered result: task, finish, start
    int64_t bf = 0, bs = 0;
    while (qn > 0) {
        // ---- schedule(Q) ----
        // One pass: per lane, the least time among its entries, the least
        // (id, slot) among its entries of that time, and the best push/pull
        // key (highest priority, then least id) among them.  Times are
        // nonnegative, so they compare as unsigned.
        uint64_t tb = ~0ull;
        uint32_t kb = 0xffffffffu;           // id << kSlotBits | slot
        uint64_t pb = ~0ull;                 // ~priority << 32 | id << kSlotBits | slot
        for (int j = 0; j * 64 < qn; j++) {
            const int i = j * 64 + lane;
            if (i < qn) {
                const int64_t p = sP[q.th[i]];
                const int64_t e = q.est[i];
                const uint64_t t = (uint64_t)(p > e ? p : e);
                const uint32_t ai = q.a[i];
                const uint32_t k = ((ai & kIdMask) << kSlotBits) | (uint32_t)i;
                const uint64_t pk = (ai & kPPb)
                    ? ((uint64_t)(~((uint32_t)q.pr[i] ^ 0x80000000u)) << 32) | k : ~0ull;
                if (t < tb) {
                    tb = t;
                    kb = k;
                    pb = pk;
                } else if (t == tb) {
                    kb = tmin(kb, k);
                    pb = tmin(pb, pk);
                }
            }
        }
        const uint64_t T0 = wave_min_u64(tb);
        const bool at = tb == T0;
        const uint32_t m1 = wave_min_u32(at ? kb : 0xffffffffu);
        int32_t ws = (int32_t)(m1 & (uint32_t)(kQ - 1));
        if (a.policy == 1 && (q.a[ws] & kPPb)) {
            // the push/pull tasks of least time: highest priority, then least id
            const uint64_t pk = wave_min_u64(at ? pb : ~0ull);
            ws = (int32_t)(pk & (uint64_t)(kQ - 1));
        }
        // ---- dispatch ----
        const uint32_t wa = __builtin_amdgcn_readfirstlane(q.a[ws]);
        const int32_t th = __builtin_amdgcn_readfirstlane((int32_t)q.th[ws]);
        const int64_t eu = q.est[ws];
        const int32_t u = (int32_t)(wa & kIdMask);
        const bool rmv = (wa & kRMb) != 0u;
        const int4 ur = a.rec[u];
        const uint4 ue4 = a.e4[u];
        const int64_t dd = a.dur[u];
        const int64_t gg = a.gap[u];
        const ScaleEntry se = TLDS ? sTab[ur.w] : a.table[(int64_t)ur.w * V + v];
        const int64_t du = rmv ? 0 : scaled(dd, se);
        const int64_t gu = rmv ? 0 : gg;
        const int64_t pt = sP[th];
        const int64_t s = pt > eu ? pt : eu;
        const int64_t f = s + du;
        const int64_t rel = f + gu;
        if (!rmv) ms = f > ms ? f : ms;
        const int32_t last = qn - 1;
        if (lane == 0) {
            // the last entry fills the dispatched one's slot
            q.a[ws] = q.a[last];
            q.th[ws] = q.th[last];
            q.pr[ws] = q.pr[last];
            q.est[ws] = q.est[last];
            sP[th] = rel;
        }
        // results go out 64 at a time, one per lane: a store in every step
        // would make each step's wait for its loads wait for the store too
        // (vector memory operations complete in order)
        if (lane == (done & 63)) {
            bu = u;
            bf = f;
            bs = s;
        }
        qn = last;
        done++;
        if ((done & 63) == 0) {
            a.finish[(int64_t)bu * V + v] = bf;
            if (a.start) a.start[(int64_t)bu * V + v] = bs;
        }
        // ---- children ----
        for (int32_t base = 0; base < ur.y; base += 64) {
            const int32_t k = base + lane;
            bool act = false;
            uint32_t pk = 0;
            if (k < ur.y) {
                pk = k < 4 ? pick4(ue4, k) : a.edges[(int64_t)ur.x + k];
                const uint32_t c = pk & 255u;
                act = c == kEdgeAlways || ((on >> c) & 1ull);
            }
            bool ready = false;
            int64_t ce = 0;
            int32_t cth = 0, cp = 0;
            bool cpp = false, crm = false;
            const int32_t c = (int32_t)(pk >> 8);
            if (act) {
                const int32_t old = atomicSub(&ref[c], 1);
                const unsigned long long oe = atomicMax(&est[c], (unsigned long long)rel);
                // what the frontier entry needs, if this was the child's last parent
                cth = a.tid[c];
                cp = a.prio ? a.prio[c] : 0;
                cpp = a.pp ? a.pp[c] != 0 : false;
                crm = (a.rm[(int64_t)c * a.W + vw] & vbit) != 0u;
                ready = old == 1;
                ce = (int64_t)oe > rel ? (int64_t)oe : rel;
            }
            const uint64_t b = __ballot(ready);
            if (ready) {
                const int32_t slot = qn + __popcll(b & lt);
                if (slot < kQ)
                    push_entry(q, slot, (uint32_t)c, cpp, crm, cth, cp, ce);
                else
                    err |= 2u;
            }
            qn += __popcll(b);
            if (qn > kQ) qn = kQ;
        }
    }
    if (lane < (done & 63)) {
        a.finish[(int64_t)bu * V + v] = bf;
        if (a.start) a.start[(int64_t)bu * V + v] = bs;
    }
    if (done != n) err |= 1u;
    for (int o = 32; o > 0; o >>= 1) err |= (uint32_t)__shfl_xor((int)err, o, 64);
    if (lane == 0) {
        a.makespan[v] = ms;
        if (err) atomicOr(a.err, err);
    }
}

}  // namespace

// ---------------------------------------------------------------------------
hipError_t build_event_lists(const dd_graph *g, EventLists *ev, hipStream_t s) {
    const int32_t n = g->n;
    hipError_t e = hipSuccess;
    unsigned long long *cnt = nullptr;
    int64_t *beg = nullptr;
    int64_t m = 0;
    const int blocks = grid_for(n, kBS);
#define EV_TRY(x)                  \
    do {                           \
        e = (x);                   \
        if (e != hipSuccess) goto out; \
    } while (0)
    EV_TRY(dalloc_n(&cnt, (size_t)n + 1, s));
    EV_TRY(dalloc_n(&beg, (size_t)n + 1, s));
    EV_TRY(hipMemsetAsync(cnt, 0, sizeof(unsigned long long) * ((size_t)n + 1), s));
    if (n > 0) {
        k_ev_count<<<blocks, kBS, 0, s>>>(n, g->xin_ptr, g->xin_src, g->thread_prev, cnt);
        EV_TRY(hipGetLastError());
    }
    EV_TRY(scan_exclusive((const int64_t *)cnt, beg, n, s));
    EV_TRY(hipMemcpyAsync(&m, beg + n, sizeof(int64_t), hipMemcpyDeviceToHost, s));
    EV_TRY(hipStreamSynchronize(s));
    EV_TRY(dalloc_n(&ev->edges, (size_t)m + 1, s));
    EV_TRY(dalloc_n(&ev->rec, (size_t)n + 1, s));
    EV_TRY(dalloc_n(&ev->e4, (size_t)n + 1, s));
    EV_TRY(hipMemsetAsync(cnt, 0, sizeof(unsigned long long) * ((size_t)n + 1), s));
    if (n > 0) {
        k_ev_fill<<<blocks, kBS, 0, s>>>(n, g->xin_ptr, g->xin_src, g->xin_cls, g->thread_prev,
                                         beg, cnt, ev->edges);
        EV_TRY(hipGetLastError());
        k_ev_rec<<<blocks, kBS, 0, s>>>(n, beg, g->thread_id, g->cls, ev->edges, ev->rec, ev->e4);
        EV_TRY(hipGetLastError());
    }
    ev->n_edges = m;
    // complete before any stream uses the lists
    EV_TRY(hipStreamSynchronize(s));
out:
#undef EV_TRY
    dfree(cnt, s);
    dfree(beg, s);
    return e;
}

void free_event_lists(EventLists *ev, hipStream_t s) {
    dfree(ev->rec, s);
    dfree(ev->e4, s);
    dfree(ev->edges, s);
    *ev = EventLists();
}

hipError_t launch_sim_event(const dd_graph *g, const EventLists &ev, const dd_variants *var,
                            int32_t policy, const uint8_t *pp, const int32_t *prio, int32_t *ref,
                            int64_t *est, int64_t *finish, int64_t *start, int64_t *makespan,
                            uint32_t *err, hipStream_t s) {
    EvArgs a;
    a.n = g->n;
    a.V = var->V;
    a.W = var->W;
    a.T = g->n_threads;
    a.n_cls = var->n_cls;
    a.policy = policy;
    a.rec = ev.rec;
    a.e4 = ev.e4;
    a.edges = ev.edges;
    a.in_ptr = g->xin_ptr;
    a.in_cls = g->xin_cls;
    a.tprev = g->thread_prev;
    a.tid = g->thread_id;
    a.dur = g->dur;
    a.gap = g->gap;
    a.table = var->table;
    a.rm = var->rm_bits;
    a.edge_on = var->edge_on;
    a.pp = pp;
    a.prio = prio;
    a.ref = ref;
    a.est = reinterpret_cast<unsigned long long *>(est);
    a.finish = finish;
    a.start = start;
    a.makespan = makespan;
    a.err = err;
    const size_t lds = sizeof(int64_t) * (size_t)(g->n_threads > 0 ? g->n_threads : 1);
    if (var->n_cls <= kLdsCls)
        k_sim_event<true><<<var->V, 64, lds, s>>>(a);
    else
        k_sim_event<false><<<var->V, 64, lds, s>>>(a);
    return hipGetLastError();
}

}  // namespace dd
