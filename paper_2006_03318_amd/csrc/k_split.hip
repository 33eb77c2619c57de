// Batched simulation for few-variant sweeps: every phase cut across several
// workgroups per variant.
//
// What is computed is what the one-workgroup-per-variant kernel computes
// (Sec. 4.1, Algorithm 1, with the transformations of Sec. 4.4 applied per
// variant): for each task u and variant v,
//     d' = removed ? 0 : floor(d * p / q),   g' = removed ? 0 : g
//     start  = max(0, release of every parent present in v)
//     finish = start + d',   release = finish + g'
//     makespan[v] = max finish over tasks not removed in v.
//
// How.  With few variants, one workgroup per variant leaves most compute
// units idle and walks each long phase alone.  Here each phase is one
// launch.  Its positions are cut into chunks of L consecutive positions and
// each workgroup takes one (variant group, chunk) pair.  Inside a run of one
// thread the releases follow R_i = max(R_{i-1}, X_i) + w_i, so a chunk folds
// its positions into one map c -> max(c + A, B) per variant; a run's first
// task ignores its input (A = kHead).  A chunk
//   1. gathers its parents' releases (all in earlier phases, so written by
//      earlier launches) and folds its maps: lane, wave, workgroup;
//   2. publishes its aggregate map, or, when it starts a run, its final
//      release at once;
//   3. finds its carry-in by looking back over the chunks before it in the
//      phase: every thread reads one (chunk, variant) slot, so a pass covers
//      256 / VG chunks, composed in the wave and then across waves; it stops
//      at the first chunk that starts a run or has published its final
//      release (chunk 0 always starts a run);
//   4. publishes its final release, then writes finish (and start) of every
//      position.
// A chunk never depends on another workgroup running: every input of a
// chunk's aggregate comes from earlier launches, so a lane that has polled
// an earlier chunk's slot for long enough (that chunk's workgroup may not
// have started yet) folds that chunk itself and goes on.  No assumption on
// how many workgroups are resident or in which order they start.

#include "dd_common.h"
#include "dd_internal.h"

#include <algorithm>
#include <atomic>

namespace dd {
namespace {

constexpr int kSpNT = 256;                              // threads per workgroup
constexpr int64_t kHead = -(int64_t(1) << 62);          // a map that ignores its input
constexpr int64_t kHeadMaxWg = 1024;    // a one-chunk step rides on a next launch of at most
                                        // this many workgroups
constexpr int32_t kPolls = 1 << 12;                     // look-back polls before a lane folds
                                                        // the chunk itself

// The look-back slot of one (step, variant group, chunk, variant).  Every
// slot is written at most once per call and cleared before the first step,
// so each word is its own flag: a value x is stored as x with the sign bit
// flipped, which is never 0 for the values stored here (they lie in
// [kHead, 2^62)), and 0 means "not yet".  Readers need no ordering between
// the words, hence relaxed device-scope atomics only (no cache write-back
// or invalidation, which at device scope would touch the whole L2).
struct alignas(8) LookSlot {
    uint64_t a, b;      // aggregate map
    uint64_t inc;       // release at the chunk's end
};
__device__ __forceinline__ uint64_t enc(int64_t x) { return (uint64_t)x ^ (1ull << 63); }
__device__ __forceinline__ int64_t dec(uint64_t w) { return (int64_t)(w ^ (1ull << 63)); }

struct SplitArgs {
    const Rec *rec;
    const int64_t *gat_ptr;       // [n+1] gathers of each position
    const int32_t *gat_src;       // (gathers beyond two of a position)
    const uint8_t *gat_cls;
    const int32_t *thread_prev;   // [n] previous task on the thread
    const int64_t *gap;           // [n] gap of every task
    const ScaleEntry *table;      // [n_cls][V]
    const uint32_t *rm;           // [n][W] removal bits
    const uint64_t *edge_on;      // [V]
    int32_t V, W, thread_carry, ngrp;
    int32_t polls;                // look-back polls of one slot before the lane folds the chunk
    int64_t *finish, *start;
    unsigned long long *makespan; // [V], zero before the first phase
    LookSlot *look;               // [chunks of all steps][ngrp][VG], zero before the first phase
};

__device__ __forceinline__ int64_t scale_dur(int64_t d, const ScaleEntry &se) {
    const uint64_t x = (uint64_t)d * (uint64_t)se.p;
    return (int64_t)(se.magic ? (__umul64hi(x, se.magic) >> se.shift) : (x >> se.shift));
}

// (a, b) := (a, b) followed by (a2, b2)
__device__ __forceinline__ void then(int64_t &a, int64_t &b, int64_t a2, int64_t b2) {
    const int64_t t = b + a2;
    b = t > b2 ? t : b2;
    a = (a == kHead || a2 == kHead) ? kHead : a + a2;
}

// the map applied to a carry
__device__ __forceinline__ int64_t apply(int64_t a, int64_t b, int64_t c) {
    if (a == kHead) return b;
    const int64_t t = c + a;
    return t > b ? t : b;
}

__device__ __forceinline__ int64_t max64(int64_t x, int64_t y) { return x > y ? x : y; }

__device__ __forceinline__ bool cls_on(uint64_t eon, uint32_t c) {
    return c == 255u || ((eon >> c) & 1ull);
}

__device__ __forceinline__ uint64_t ld_relaxed(const uint64_t *p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_relaxed(uint64_t *p, uint64_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// One phase [ps0, ps1): pnch chunks of L = (kSpNT / VG) * K positions per
// variant group; lane = (slot, variant), each slot K consecutive positions,
// whose loads go out S positions at a time (S = K: every load of a lane in
// flight together, for launches of few workgroups; S = K / 2: fewer
// registers and more resident waves, for launches of many).  When the
// phase before it is a single chunk [h0, h1) (h1 > h0), every workgroup
// first computes that phase itself and writes its results (the same
// values from every workgroup of a group), so it needs no launch of its
// own: its parents lie in earlier launches, and a workgroup barrier makes
// the workgroup's own writes visible to its loads.
template <int VG, int K, int S>
__global__ __launch_bounds__(kSpNT) void k_sim_phase(int32_t p, int32_t ps0, int32_t ps1,
                                                     int32_t pnch, int64_t pcoff, int32_t h0,
                                                     int32_t h1, SplitArgs a) {
    constexpr int NSL = kSpNT / VG;
    constexpr int L = NSL * K;
    constexpr int NWV = kSpNT / 64;
    __shared__ int sFirst;
    __shared__ int64_t sWA[NWV][VG], sWB[NWV][VG];
    __shared__ int64_t sLA[NWV][VG], sLB[NWV][VG];
    __shared__ int64_t sCarry[VG];
    __shared__ unsigned long long sMs[VG];

    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int j = tid % VG, slot = tid / VG;
    const int g = blockIdx.x % a.ngrp;
    const int v = g * VG + j;
    const bool vok = v < a.V;
    const int vv = vok ? v : 0;
    const int64_t V = a.V, W = a.W;
    const int vw = vv >> 5;
    const uint32_t vbit = 1u << (vv & 31);
    const uint64_t eon = a.edge_on[vv];

    // chunk c of the phase [s0, s1) of nch chunks, whose look-back slots
    // start at chunk offset coff; keep = add to the makespan
    auto run_chunk = [&](const int32_t s0, const int32_t s1, const int32_t nch, const int c,
                         const int64_t coff, const bool keep) {
    // this step's slots: [nch][ngrp][VG] from chunk offset coff
    LookSlot *const look = a.look + coff * a.ngrp * VG;
    auto slot_of = [&](int ch) { return look + ((int64_t)ch * a.ngrp + g) * VG + j; };
    auto chunk_end = [&](int ch) {
        const int64_t e = (int64_t)s0 + (int64_t)(ch + 1) * L;
        return e < (int64_t)s1 ? e : (int64_t)s1;
    };
    const int64_t q0 = (int64_t)s0 + (int64_t)c * L;
    const int64_t q1 = chunk_end(c);
    if (tid < VG) sMs[tid] = 0ull;

    // release of a parent: its finish plus its gap when it is kept
    auto rel = [&](int64_t s) -> int64_t {
        const int64_t f = a.finish[s * V + vv];
        const bool rs = a.rm[s * W + vw] & vbit;
        return f + (rs ? 0 : a.gap[s]);
    };

    // one position for this lane's variant: latest parent release x,
    // duration dp and gap gp as transformed, run start, kept.  In three
    // stages, so that a lane issues the loads of all its positions before
    // it waits for any: the record; what the record points at (the task's
    // removal word and scale entry, each inline parent's finish, removal
    // word and gap); the arithmetic, with the rare loads (parents beyond
    // two, a run's thread predecessor).
    struct Pos {
        int64_t x, dp, gp;
        int32_t u;
        bool head, live;
    };
    struct Deps {
        ScaleEntry se;
        int64_t f0, g0, f1, g1;
        uint32_t rmw, r0w, r1w;
    };
    auto deps_of = [&](const Rec &r) -> Deps {
        const int64_t u = r.node;
        Deps d{};
        d.rmw = a.rm[u * W + vw];
        d.se = a.table[(int64_t)(r.cls & 0xffffu) * V + vv];
        if (r.g0_src >= 0) {
            const int64_t s0i = r.g0_src;
            d.f0 = a.finish[s0i * V + vv];
            d.r0w = a.rm[s0i * W + vw];
            d.g0 = a.gap[s0i];
        }
        if (r.g1_src >= 0) {
            const int64_t s1i = r.g1_src;
            d.f1 = a.finish[s1i * V + vv];
            d.r1w = a.rm[s1i * W + vw];
            d.g1 = a.gap[s1i];
        }
        return d;
    };
    auto position_of = [&](int64_t q, const Rec &r, const Deps &d) -> Pos {
        const int64_t u = r.node;
        const bool live = !(d.rmw & vbit);
        const int64_t dp = live ? scale_dur(r.dur, d.se) : 0;
        const int64_t gp = live ? r.gap : 0;
        int64_t x = 0;
        if (r.g0_src >= 0 && cls_on(eon, (r.cls >> 16) & 0xffu))
            x = max64(x, d.f0 + ((d.r0w & vbit) ? 0 : d.g0));
        if (r.g1_src >= 0 && cls_on(eon, r.cls >> 24))
            x = max64(x, d.f1 + ((d.r1w & vbit) ? 0 : d.g1));
        if (r.flags >> 8) {                    // gathers beyond two
            const int64_t e1 = a.gat_ptr[q + 1];
            for (int64_t e = a.gat_ptr[q] + 2; e < e1; e++)
                if (cls_on(eon, a.gat_cls[e])) x = max64(x, rel(a.gat_src[e]));
        }
        const bool head = r.flags & 1u;
        if (head && a.thread_carry) {          // the run's thread predecessor
            const int32_t tp = a.thread_prev[u];
            if (tp >= 0) x = max64(x, rel(tp));
        }
        return Pos{x, dp, gp, (int32_t)u, head, live};
    };
    auto position = [&](int64_t q) -> Pos {
        const Rec r = a.rec[q];
        return position_of(q, r, deps_of(r));
    };

    // 1. gather and fold
    int64_t X[K], DP[K], GP[K];
    int32_t ND[K];
    uint32_t hd = 0, ok = 0, lv = 0;
    int64_t la = 0, lb = kHead;               // identity
    static_assert(K % S == 0, "stages of whole positions");
#pragma unroll
    for (int h = 0; h < K; h += S) {
        Rec R[S];
        Deps D[S];
#pragma unroll
        for (int i = 0; i < S; i++) {          // positions past the chunk read its last one
            const int64_t q = q0 + (int64_t)slot * K + h + i;
            R[i] = a.rec[q < q1 ? q : q1 - 1];
        }
#pragma unroll
        for (int i = 0; i < S; i++) D[i] = deps_of(R[i]);
#pragma unroll
        for (int i = 0; i < S; i++) {
            const int k = h + i;
            const int64_t q = q0 + (int64_t)slot * K + k;
            X[k] = 0; DP[k] = 0; GP[k] = 0; ND[k] = 0;
            if (q < q1) {
                const Pos ps = position_of(q, R[i], D[i]);
                X[k] = ps.x; DP[k] = ps.dp; GP[k] = ps.gp; ND[k] = ps.u;
                ok |= 1u << k;
                hd |= (ps.head ? 1u : 0u) << k;
                lv |= (ps.live ? 1u : 0u) << k;
                then(la, lb, ps.head ? kHead : ps.dp + ps.gp, ps.x + ps.dp + ps.gp);
            }
        }
    }
    // inclusive scan over the slots of one variant: inside the wave (lanes
    // VG apart), then across waves
    int64_t ia = la, ib = lb;
#pragma unroll
    for (int o = VG; o < 64; o <<= 1) {
        const int64_t pa = shfl_up64(ia, o), pb = shfl_up64(ib, o);
        if (lane >= o) {
            int64_t na = pa, nb = pb;
            then(na, nb, ia, ib);
            ia = na; ib = nb;
        }
    }
    if (lane >= 64 - VG) { sWA[wv][j] = ia; sWB[wv][j] = ib; }
    if (tid == 0) sFirst = c == 0 || (hd & 1u);
    const int64_t xa = shfl_up64(ia, VG), xb = shfl_up64(ib, VG);
    __syncthreads();
    int64_t ea = 0, eb = kHead;               // exclusive map of this slot
    for (int w2 = 0; w2 < wv; w2++) then(ea, eb, sWA[w2][j], sWB[w2][j]);
    if (lane >= VG) then(ea, eb, xa, xb);

    // 2.-3. publish, look back, publish the chunk's final release
    int64_t ga = 0, gb = kHead;               // the chunk's aggregate
    for (int w2 = 0; w2 < NWV; w2++) then(ga, gb, sWA[w2][j], sWB[w2][j]);
    const bool later = c + 1 < nch;           // a chunk after this one reads the slot
    LookSlot *const own = slot_of(c);
    // the carry-in is needed unless the chunk's first position starts a run
    const bool first_head = sFirst != 0;
    if (later && !first_head && tid < VG) {
        st_relaxed(&own->a, enc(ga));
        st_relaxed(&own->b, enc(gb));
    }
    int64_t cin = kHead;
    if (!first_head) {
        // every thread reads chunk dtop - slot for its variant, so one pass
        // covers NSL chunks; acc composes the chunks after the current
        // window up to c - 1 (the same in every thread of one variant)
        int64_t acc_a = 0, acc_b = kHead;
        bool done = false;
        int dtop = c - 1;
        for (;;) {
            const int d = dtop - slot;
            int64_t ta = 0, tb = kHead;       // identity past chunk 0
            if (!done && d >= 0) {
                LookSlot *const ls = slot_of(d);
                for (int32_t n = 0;; n++) {
                    if (n >= a.polls) {       // fold chunk d here
                        const int64_t e = chunk_end(d);
                        for (int64_t q = (int64_t)s0 + (int64_t)d * L; q < e; q++) {
                            const Pos ps = position(q);
                            then(ta, tb, ps.head ? kHead : ps.dp + ps.gp, ps.x + ps.dp + ps.gp);
                        }
                        break;
                    }
                    const uint64_t wi = ld_relaxed(&ls->inc);
                    if (wi) { ta = kHead; tb = dec(wi); break; }
                    const uint64_t wa = ld_relaxed(&ls->a), wb = ld_relaxed(&ls->b);
                    if (wa && wb) { ta = dec(wa); tb = dec(wb); break; }
                    __builtin_amdgcn_s_sleep(2);
                }
            }
            // in the wave: (earlier chunk) followed by (later chunks)
#pragma unroll
            for (int o = VG; o < 64; o <<= 1) {
                const int64_t pa = shfl_up64(ta, o), pb = shfl_up64(tb, o);
                if (lane >= o) then(ta, tb, pa, pb);
            }
            if (lane >= 64 - VG) { sLA[wv][j] = ta; sLB[wv][j] = tb; }
            __syncthreads();
            if (!done) {
                int64_t na = 0, nb = kHead;   // the last wave holds the earliest chunks
                for (int w2 = NWV - 1; w2 >= 0; w2--) then(na, nb, sLA[w2][j], sLB[w2][j]);
                then(na, nb, acc_a, acc_b);
                acc_a = na; acc_b = nb;
                dtop -= NSL;
                done = acc_a == kHead || dtop < 0;
            }
            if (!__syncthreads_or(done ? 0 : 1)) break;
        }
        cin = apply(acc_a, acc_b, kHead);
    }
    if (tid < VG) {
        sCarry[j] = cin;
        if (later) st_relaxed(&own->inc, enc(apply(ga, gb, cin)));
    }
    __syncthreads();

    // 4. results
    int64_t cr = apply(ea, eb, sCarry[j]);
    unsigned long long ms = 0ull;
#pragma unroll
    for (int k = 0; k < K; k++) {
        if (ok & (1u << k)) {
            const int64_t st = (hd & (1u << k)) ? X[k] : max64(cr, X[k]);
            const int64_t f = st + DP[k];
            cr = f + GP[k];
            if (vok) {
                a.finish[(int64_t)ND[k] * V + v] = f;
                if (a.start) a.start[(int64_t)ND[k] * V + v] = st;
                if ((lv >> k) & 1u) ms = ms > (unsigned long long)f ? ms : (unsigned long long)f;
            }
        }
    }
    if (ms) atomicMax(&sMs[j], ms);
    __syncthreads();
    if (keep && tid < VG && vok && sMs[tid]) atomicMax(&a.makespan[v], sMs[tid]);
    };

    const int c = (int)(blockIdx.x / a.ngrp);
    if (h1 > h0) {
        // the one-chunk phase before this one (only chunk 0 adds it to the
        // makespan); the barrier orders its writes before this phase's loads
        run_chunk(h0, h1, 1, 0, 0, c == 0);
        __syncthreads();
    }
    run_chunk(ps0, ps1, pnch, c, pcoff, true);
}

__global__ __launch_bounds__(256) void k_split_zero(uint64_t *look, int64_t nl, int64_t *makespan,
                                                   int64_t V) {
    const int64_t stride = (int64_t)gridDim.x * 256;
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < nl + V; i += stride) {
        if (i < nl) look[i] = 0ull;
        else makespan[i - nl] = 0;
    }
}

std::atomic<int32_t> g_polls{kPolls};

template <int VG, int K, int S>
hipError_t run_phases(const dd_graph *g, const dd_sched *sch, const dd_variants *var,
                      int64_t *finish, int64_t *start, int64_t *makespan, hipStream_t s) {
    constexpr int L = (kSpNT / VG) * K;
    const std::vector<int32_t> &sp = sch->h_step_ptr;
    const int64_t ns = sch->n_steps;
    if ((int64_t)sp.size() != ns + 1) return hipErrorInvalidValue;
    int64_t nchunks = 0;               // chunks of all steps
    for (int64_t p = 0; p < ns; p++) nchunks += (sp[p + 1] - sp[p] + L - 1) / L;
    const int ngrp = (var->V + VG - 1) / VG;
    const int64_t nslot = nchunks * ngrp * VG;
    const int64_t nl = nslot * (int64_t)(sizeof(LookSlot) / 8);
    LookSlot *look = nullptr;
    hipError_t e = dalloc_n(&look, (size_t)nslot + 1, s);
    if (e == hipSuccess) {
        const int zg = grid_for(nl + var->V, 256);
        k_split_zero<<<zg < 1024 ? zg : 1024, 256, 0, s>>>(reinterpret_cast<uint64_t *>(look), nl,
                                                          makespan, var->V);
        e = hipGetLastError();
    }
    SplitArgs args{sch->rec, sch->gat_ptr, sch->gat_src, sch->gat_cls, g->thread_prev, g->gap,
                   var->table, var->rm_bits, var->edge_on, var->V, var->W,
                   sch->thread_carry ? 1 : 0, ngrp, g_polls.load(), finish, start,
                   reinterpret_cast<unsigned long long *>(makespan), look};
    int64_t coff = 0;
    int32_t h0 = 0, h1 = 0;                  // a pending one-chunk step
    for (int64_t p = 0; p < ns && e == hipSuccess; p++) {
        const int64_t len = sp[p + 1] - sp[p];
        if (len <= 0) continue;
        const int32_t nch = (int32_t)((len + L - 1) / L);
        if ((int64_t)nch * ngrp > INT32_MAX) {   // more workgroups than one launch takes
            e = hipErrorInvalidConfiguration;
            break;
        }
        // a one-chunk step waits to ride on the next step's launch (unless
        // one is already waiting, it is the last step, or that launch has
        // more than kHeadMaxWg workgroups, each of which would redo it)
        int64_t pn = p + 1;
        while (pn < ns && sp[pn + 1] == sp[pn]) pn++;
        const int64_t wg_next = pn < ns ? (sp[pn + 1] - sp[pn] + L - 1) / L * ngrp : 0;
        if (nch == 1 && h1 == h0 && pn < ns && wg_next <= kHeadMaxWg) {
            h0 = sp[p];
            h1 = sp[p + 1];
            coff += nch;
            continue;
        }
        k_sim_phase<VG, K, S><<<nch * ngrp, kSpNT, 0, s>>>((int32_t)p, sp[p], sp[p + 1], nch, coff,
                                                           h0, h1, args);
        e = hipGetLastError();
        coff += nch;
        h0 = h1 = 0;
    }
    dfree(look, s);
    return e;
}

}  // namespace

void split_set_polls(int32_t polls) { g_polls.store(polls < 0 ? kPolls : polls); }

int split_width(const dd_sched *sch, const dd_variants *var) {
    if (sch->n <= 0 || var->V <= 0 || (int64_t)sch->h_step_ptr.size() != sch->n_steps + 1)
        return 0;
    // Fewer than 1,024 variants only: below that the one-workgroup-per-strip
    // kernel either leaves compute units idle or runs its workgroups in two
    // passes (one variant per workgroup up to 511 variants, two up to
    // 1,023).  Then by measured cost: that kernel takes about 1.8 us per round
    // of 512 positions, this path about 8 us per step (a launch and its
    // chain of memory trips), so this one wins when steps hold more than
    // about 4.4 rounds on average.
    if (var->V >= 1024) return 0;
    const std::vector<int32_t> &sp = sch->h_step_ptr;
    int64_t rounds = 0, wmax = 0;
    for (int64_t p = 0; p < sch->n_steps; p++) {
        const int64_t len = sp[p + 1] - sp[p];
        rounds += (len + 511) / 512;
        wmax = std::max<int64_t>(wmax, len);
    }
    if (rounds * 9 <= sch->n_steps * 40) return 0;
    // 8 variants per workgroup when the widest step then still gives about
    // 1.5 workgroups per compute unit, else 4 (more, smaller workgroups)
    const int64_t wg8 = (int64_t)((var->V + 7) / 8) * ((wmax + 255) / 256);
    if (var->V >= 8 && wg8 >= 384) return 8;
    return var->V >= 4 ? 4 : var->V >= 2 ? 2 : 1;
}

hipError_t launch_split(const dd_graph *g, const dd_sched *sch, const dd_variants *var,
                        int64_t *finish, int64_t *start, int64_t *makespan, int vg, hipStream_t s) {
    switch (vg) {
        case 1: return run_phases<1, 1, 1>(g, sch, var, finish, start, makespan, s);
        case 2: return run_phases<2, 2, 2>(g, sch, var, finish, start, makespan, s);
        case 4: return run_phases<4, 4, 4>(g, sch, var, finish, start, makespan, s);
        case 8: {
            // half the loads in flight when the widest step needs 1,024 or
            // more workgroups (occupancy then matters more than one lane's
            // overlap: 768 variants 1.66 against 1.85 ms, 64 variants 0.33
            // against 0.31 ms)
            int64_t wmax = 0;
            const std::vector<int32_t> &sp = sch->h_step_ptr;
            for (size_t p = 0; p + 1 < sp.size(); p++) wmax = std::max<int64_t>(wmax, sp[p + 1] - sp[p]);
            if ((int64_t)((var->V + 7) / 8) * ((wmax + 255) / 256) >= 1024)
                return run_phases<8, 8, 4>(g, sch, var, finish, start, makespan, s);
            return run_phases<8, 8, 8>(g, sch, var, finish, start, makespan, s);
        }
        default: return hipErrorInvalidValue;
    }
}

}  // namespace dd
