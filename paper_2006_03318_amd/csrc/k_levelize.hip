// Levelization on the GPU: Kahn's algorithm over the task graph (the
// reference counts and ready frontier of Sec. 4.1, Algorithm 1), taken one
// whole frontier per round.
//
// Phases.  Because tasks on one thread run in their recorded order
// (Sec. 4.2.2), the graph is a set of thread chains plus cross-thread
// dependencies.  A round advances the front of every thread past all tasks
// whose cross-thread parents lie behind the fronts of their own threads at
// the start of the round; the tasks passed in round r form phase r, one
// contiguous run ("segment") per thread.  This is Kahn's algorithm where
// "parent done" is read off the parent thread's front instead of a
// decremented counter.  Phase = longest path counting 1 per cross-thread
// edge and 0 per thread-order edge.  A round that advances no thread while
// tasks remain means a cycle.
//
// Levels.  Kahn level = longest path counting 1 per edge.  Inside a
// segment, level_i = max(level_{i-1} + 1, X_i) with X_i = 1 + the largest
// level of a cross-thread parent; with the phases known, every segment is a
// segmented prefix maximum of X_j - j.
//
// The schedule handed to the simulation lists tasks by step (phase or
// level); within a phase step, thread runs are contiguous and in thread
// order.  Each position carries its "gathers": the cross-thread parents,
// plus the previous task on the thread for the first task of a run.

#include "dd_common.h"
#include "dd_internal.h"

#include <stdio.h>

namespace dd {
namespace {

constexpr int kBS = 256;
constexpr int kWG = 1024;   // the single workgroup running the rounds

struct Req {
    const int64_t *base;      // [T+1] thread start in order space
    const int32_t *order;
    const int32_t *rank;
    const int32_t *tid;
    const int64_t *xin_ptr;
    const int32_t *xin_src;
    const uint8_t *xin_cls;
};

__device__ __forceinline__ bool on(uint64_t mask, uint8_t c) { return (mask >> c) & 1ull; }

// per order position: number of active cross-thread parents
__global__ __launch_bounds__(kBS) void k_req_count(int32_t n, Req r, uint64_t mask,
                                                   int64_t *__restrict__ cnt,
                                                   int64_t *__restrict__ flag) {
    const int64_t p = (int64_t)blockIdx.x * kBS + threadIdx.x;
    if (p >= n) return;
    const int32_t u = r.order[p];
    int64_t c = 0;
    for (int64_t k = r.xin_ptr[u]; k < r.xin_ptr[u + 1]; k++) c += on(mask, r.xin_cls[k]);
    cnt[p] = c;
    flag[p] = c > 0;
}

constexpr int kWinT = 16;               // graph threads of the windowed rounds at most

// A candidate packed for the windowed rounds: its order position and, for
// the first two parent threads (by id) among its requirements, the largest
// requirement position on each (order space); meta = first thread | second
// thread << 8 | number of distinct parent threads << 16.  It is blocked when
// one of those maxima lies at or past its thread's front; only a candidate
// with parents on three or more threads needs its full requirement list.
struct alignas(16) CandEnt {
    int32_t pos, g0, g1;
    uint32_t meta;
};

// candidates (positions with a cross-thread parent) and their requirements;
// with pent, the packed entries too (T <= kWinT: the first two parent
// threads by id; T <= kEntT: the first two met in the list, which serves
// the same test)
constexpr int kEntT = 255;              // graph threads a packed entry can name (8 bits)
__global__ __launch_bounds__(kBS) void k_req_fill(int32_t n, int32_t T, Req r, uint64_t mask,
                                                  const int64_t *__restrict__ cidx,
                                                  const int64_t *__restrict__ rptr_by_pos,
                                                  int64_t *__restrict__ cand_pos,
                                                  int64_t *__restrict__ req_ptr,
                                                  int32_t *__restrict__ req_chain,
                                                  int64_t *__restrict__ req_gpos,
                                                  CandEnt *__restrict__ pent) {
    const int64_t p = (int64_t)blockIdx.x * kBS + threadIdx.x;
    if (p >= n) return;
    if (cidx[p + 1] == cidx[p]) return;
    const int64_t i = cidx[p];
    cand_pos[i] = p;
    int64_t o = rptr_by_pos[p];
    req_ptr[i] = o;
    const int32_t u = r.order[p];
    int32_t mx[kWinT];                  // largest requirement per parent thread (-1: none)
#pragma unroll
    for (int z = 0; z < kWinT; z++) mx[z] = -1;
    int32_t t0 = -1, t1 = -1, m0 = -1, m1 = -1;   // T > kWinT: the first two threads met
    bool many = false;                            // a third parent thread
    for (int64_t k = r.xin_ptr[u]; k < r.xin_ptr[u + 1]; k++) {
        if (!on(mask, r.xin_cls[k])) continue;
        const int32_t s = r.xin_src[k];
        const int32_t ts = r.tid[s];
        const int64_t gp = r.base[ts] + r.rank[s];
        req_chain[o] = ts;
        req_gpos[o] = gp;
#pragma unroll
        for (int z = 0; z < kWinT; z++)
            if (z == ts && (int32_t)gp > mx[z]) mx[z] = (int32_t)gp;
        if (ts == t0) m0 = (int32_t)gp > m0 ? (int32_t)gp : m0;
        else if (ts == t1) m1 = (int32_t)gp > m1 ? (int32_t)gp : m1;
        else if (t0 < 0) { t0 = ts; m0 = (int32_t)gp; }
        else if (t1 < 0) { t1 = ts; m1 = (int32_t)gp; }
        else many = true;
        o++;
    }
    if (!pent) return;                  // (more than kEntT threads: no packed entries)
    if (T > kWinT) {
        const uint32_t nd = (t0 >= 0 ? 1u : 0u) + (t1 >= 0 ? 1u : 0u) + (many ? 1u : 0u);
        pent[i] = CandEnt{(int32_t)p, m0 < 0 ? 0 : m0, m1 < 0 ? 0 : m1,
                          (uint32_t)(t0 < 0 ? 0 : t0) | ((uint32_t)(t1 < 0 ? 0 : t1) << 8) | (nd << 16)};
        return;
    }
    CandEnt ce{(int32_t)p, 0, 0, 0u};
    uint32_t nd = 0;
#pragma unroll
    for (int z = 0; z < kWinT; z++) {
        if (mx[z] < 0) continue;
        if (nd == 0) { ce.g0 = mx[z]; ce.meta |= (uint32_t)z; }
        if (nd == 1) { ce.g1 = mx[z]; ce.meta |= (uint32_t)z << 8; }
        nd++;
    }
    ce.meta |= nd << 16;
    pent[i] = ce;
}

// (also closes the requirement lists: req_ptr[C] = R, from the scan totals)
__global__ __launch_bounds__(kBS) void k_cand_base(int32_t T, int64_t n, const int64_t *__restrict__ base,
                                                   const int64_t *__restrict__ cidx,
                                                   const int64_t *__restrict__ rptr,
                                                   int64_t *__restrict__ req_ptr,
                                                   int64_t *__restrict__ cbase,
                                                   int64_t *__restrict__ front,
                                                   int64_t *__restrict__ ci) {
    const int64_t t = (int64_t)blockIdx.x * kBS + threadIdx.x;
    if (t == 0) req_ptr[cidx[n]] = rptr[n];
    if (t > T) return;
    cbase[t] = cidx[base[t]];
    if (t < T) {
        front[t] = base[t];
        ci[t] = cidx[base[t]];
    }
}

struct KahnArgs {
    const CandEnt *pent;      // [C] packed entries (T <= kEntT), else null
    int32_t T;
    int64_t n;
    const int64_t *base;      // [T+1]
    const int64_t *cand_pos;  // [C]
    const int64_t *cbase;     // [T+1]
    const int64_t *req_ptr;   // [C+1]
    const int32_t *req_chain;
    const int64_t *req_gpos;
    int64_t *front, *cidx, *nfront, *ncidx;   // [T]
    int32_t *long_list;       // [T]
    int64_t *seg_start;       // [n] order position of each segment's first task
    int64_t *seg_len;         // [n]
    int32_t *seg_step;        // [n]
    int64_t *step_seg;        // [n+1] first segment of each step
    int64_t *result;          // [0] steps, [1] segments
    uint32_t *err;
};

// Round state of the generic rounds: with at most kLdsT graph threads the
// fronts, candidate cursors and thread bounds live in LDS (a requirement
// check then reads its parent thread's front from LDS, not from global
// memory); beyond that they stay in the global arrays.
constexpr int kLdsT = 2048;
constexpr int kProbe = 128;     // candidates a round probes per thread before the long-run scan

template <bool L>
__global__ __launch_bounds__(kWG) void k_kahn_rounds(KahnArgs a) {
    __shared__ int s_nlong;
    __shared__ int s_unfinished;
    __shared__ unsigned long long s_first;
    __shared__ int64_t s_carry_cnt;
    __shared__ int64_t s_st[L ? 6 * (kLdsT + 1) : 1];
    const int lane = threadIdx.x & 63;
    int64_t *const front = L ? s_st : a.front;
    int64_t *const cidx = L ? s_st + (kLdsT + 1) : a.cidx;
    int64_t *const nfront = L ? s_st + 2 * (kLdsT + 1) : a.nfront;
    int64_t *const ncidx = L ? s_st + 3 * (kLdsT + 1) : a.ncidx;
    const int64_t *const base = L ? s_st + 4 * (kLdsT + 1) : a.base;
    const int64_t *const cbase = L ? s_st + 5 * (kLdsT + 1) : a.cbase;
    if (L) {
        for (int t = threadIdx.x; t <= a.T; t += kWG) {
            if (t < a.T) {
                s_st[t] = a.front[t];
                s_st[(kLdsT + 1) + t] = a.cidx[t];
            }
            s_st[4 * (kLdsT + 1) + t] = a.base[t];
            s_st[5 * (kLdsT + 1) + t] = a.cbase[t];
        }
        __syncthreads();
    }
    // lanes per graph thread in step A: all threads in one pass when they fit
    int gsh = 6;
    while (gsh > 0 && ((int64_t)a.T << gsh) > kWG) gsh--;
    const int G = 1 << gsh;
    const unsigned long long gmask = G == 64 ? ~0ull : ((1ull << G) - 1ull);
    // a candidate is blocked while a requirement lies at or past the front
    // of its thread
    auto blocked_list = [&](int64_t j) {
        for (int64_t k = a.req_ptr[j]; k < a.req_ptr[j + 1]; k++)
            if (a.req_gpos[k] >= front[a.req_chain[k]]) return true;
        return false;
    };
    // with packed entries: one 16-byte load; only a candidate with parents
    // on three or more threads reads its requirement list
    auto blocked_ent = [&](const CandEnt &e, int64_t j) {
        const uint32_t nd = e.meta >> 16;
        if (e.g0 >= front[e.meta & 0xff]) return true;
        if (nd > 1 && e.g1 >= front[(e.meta >> 8) & 0xff]) return true;
        if (nd > 2) return blocked_list(j);
        return false;
    };
    auto blocked = [&](int64_t j) {
        if (a.pent) return blocked_ent(a.pent[j], j);
        return blocked_list(j);
    };
    int64_t nseg = 0;
    int64_t round = 0;
    for (;;) {
        if (threadIdx.x == 0) {
            s_nlong = 0;
            s_unfinished = 0;
        }
        __syncthreads();
        // A: a group of G lanes per graph thread (G = 64 when few threads,
        // fewer when there are more, so that every thread is probed in one
        // pass) scans up to kProbe candidates of its thread, G at a time
        for (int t0 = 0; t0 < a.T; t0 += kWG >> gsh) {
            const int t = t0 + (int)(threadIdx.x >> gsh);        // uniform within a group
            const int gl = (int)threadIdx.x & (G - 1);
            const bool act = t < a.T;
            const int64_t f = act ? front[t] : 0, end = act ? base[t + 1] : 0;
            int64_t ci = act ? cidx[t] : 0;
            const int64_t ce = act ? cbase[t + 1] : 0;
            const bool fin = !act || f >= end;
            if (act && fin && gl == 0) { nfront[t] = f; ncidx[t] = ci; }
            if (!fin && gl == 0) s_unfinished = 1;   // a flag: every writer stores 1
            bool done = fin;
            int64_t cnew = ce;
            int32_t npos = 0;                 // order position of candidate cnew (packed entries)
            for (int w = 0; w < (kProbe >> gsh); w++) {
                if (__all(done)) break;                           // wave-uniform
                const int64_t j = ci + gl;
                bool b = false;
                int32_t pj = 0;
                if (!done && j < ce) {
                    if (a.pent) {
                        const CandEnt e = a.pent[j];
                        pj = e.pos;
                        b = blocked_ent(e, j);
                    } else {
                        b = blocked_list(j);
                    }
                }
                const unsigned long long bal = __ballot(b);
                const unsigned long long gb = (bal >> (lane & ~(G - 1))) & gmask;
                const int fl = gb ? __ffsll((long long)gb) - 1 : 0;
                const int32_t pf = __shfl(pj, (lane & ~(G - 1)) + fl, 64);   // the finder's position
                if (!done) {
                    if (gb) {
                        cnew = ci + fl;
                        npos = pf;
                        done = true;
                    } else if (ci + G >= ce) {
                        cnew = ce;
                        done = true;
                    } else {
                        ci += G;
                    }
                }
            }
            if (!fin && gl == 0) {
                if (done) {
                    ncidx[t] = cnew;
                    nfront[t] = cnew < ce ? (a.pent ? (int64_t)npos : a.cand_pos[cnew]) : end;
                } else {
                    ncidx[t] = ci;
                    a.long_list[atomicAdd(&s_nlong, 1)] = t;
                }
            }
        }
        __syncthreads();
        // B: threads with long ready runs, scanned by the whole workgroup
        const int nlong = s_nlong;
        for (int i = 0; i < nlong; i++) {
            const int t = a.long_list[i];
            int64_t ci = ncidx[t];
            const int64_t ce = cbase[t + 1];
            int64_t cnew = ce;
            for (;;) {
                if (threadIdx.x == 0) s_first = ~0ull;
                __syncthreads();
                const int64_t j = ci + threadIdx.x;
                if (j < ce && blocked(j)) atomicMin(&s_first, (unsigned long long)j);
                __syncthreads();
                const unsigned long long fb = s_first;
                __syncthreads();
                if (fb != ~0ull) { cnew = (int64_t)fb; break; }
                if (ci + kWG >= ce) { cnew = ce; break; }
                ci += kWG;
            }
            if (threadIdx.x == 0) {
                ncidx[t] = cnew;
                nfront[t] = cnew < ce ? a.cand_pos[cnew] : base[t + 1];
            }
        }
        __syncthreads();
        if (s_unfinished == 0) break;                 // every thread at its end
        // C: emit one segment per advanced thread.  Up to 64 threads: one
        // wave ranks them with a ballot; else a workgroup scan of packed
        // count<<32 | length per block of kWG threads.
        if (a.T <= 64) {
            if (threadIdx.x < 64) {
                const int t = (int)threadIdx.x;
                const int64_t len = t < a.T ? nfront[t] - front[t] : 0;
                const unsigned long long bal = __ballot(len > 0);
                if (len > 0) {
                    const int64_t sg = nseg + __popcll(bal & ((1ull << t) - 1ull));
                    a.seg_start[sg] = front[t];
                    a.seg_len[sg] = len;
                    a.seg_step[sg] = (int32_t)round;
                }
                if (t == 0) s_carry_cnt = __popcll(bal);
            }
            __syncthreads();
        } else {
            if (threadIdx.x == 0) s_carry_cnt = 0;
            __syncthreads();
            for (int b0 = 0; b0 < a.T; b0 += kWG) {
                const int t = b0 + threadIdx.x;
                int64_t len = 0;
                if (t < a.T) len = nfront[t] - front[t];
                const int64_t packed = len > 0 ? ((int64_t(1) << 32) | len) : 0;
                int64_t tot;
                const int64_t ex = block_excl_scan<kWG>(packed, &tot);
                if (len > 0) {
                    const int64_t sg = nseg + s_carry_cnt + (ex >> 32);
                    a.seg_start[sg] = front[t];
                    a.seg_len[sg] = len;
                    a.seg_step[sg] = (int32_t)round;
                }
                __syncthreads();
                if (threadIdx.x == 0) s_carry_cnt += tot >> 32;
                __syncthreads();
            }
        }
        const int64_t adv = s_carry_cnt;
        if (adv == 0) {                               // stalled: cycle
            if (threadIdx.x == 0) atomicOr(a.err, ERR_KAHN_CYCLE);
            break;
        }
        if (threadIdx.x == 0) a.step_seg[round] = nseg;
        nseg += adv;
        // D: advance the fronts
        for (int t = threadIdx.x; t < a.T; t += kWG) {
            front[t] = nfront[t];
            cidx[t] = ncidx[t];
        }
        round++;
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        a.step_seg[round] = nseg;
        a.result[0] = round;
        a.result[1] = nseg;
    }
}

// Windowed rounds for graphs with at most kWinT threads: the same rounds as
// above, with each thread's next candidates staged in LDS (a wave per thread,
// waves taking threads w, w + waves, ...) so that a round reads no global
// memory except to refill a window that is less than half full, to cross a
// ready run longer than the window, or for a requirement past the first two
// of a candidate.
//
// A long ready run is crossed with tile maxima: for tiles of 64 and of 4096
// consecutive candidates (global candidate order), the largest requirement
// position on each parent thread.  A tile whose maxima all lie behind the
// round's fronts holds no blocked candidate.  Candidates before the search
// start are ready already, so only a tile that also holds another thread's
// candidates can look blocked without being so; the search then simply goes
// on after it.
constexpr int kWinBytes = 6144 * 16;    // LDS window of candidate entries, shared by all threads
constexpr int kRefill = 16;             // window entries loaded per lane at once

// tile maxima over candidates: tm1[k * T + s] = largest requirement position
// on thread s among candidates [64k, 64k + 64) (-1 if none); one wave per tile
__global__ __launch_bounds__(kBS) void k_tile_max1(const int64_t *__restrict__ pC, int32_t T,
                                                   const int64_t *__restrict__ req_ptr,
                                                   const int32_t *__restrict__ req_chain,
                                                   const int64_t *__restrict__ req_gpos,
                                                   int32_t *__restrict__ tm1) {
    const int64_t C = *pC;                // candidates (the grid covers every position)
    const int64_t j = (int64_t)blockIdx.x * kBS + threadIdx.x;
    const int64_t k = j >> 6;
    if ((k << 6) >= C) return;           // whole waves past the last tile
    const bool ok = j < C;
    const int64_t q0 = ok ? req_ptr[j] : 0, q1 = ok ? req_ptr[j + 1] : 0;
    for (int32_t ts = 0; ts < T; ts++) {
        int64_t r = -1;
        for (int64_t q = q0; q < q1; q++)
            if (req_chain[q] == ts && req_gpos[q] > r) r = req_gpos[q];
        r = wave_max64(r);
        if ((threadIdx.x & 63) == 0 && (k << 6) < C) tm1[k * T + ts] = (int32_t)r;
    }
}

// tm2[m * T + s] = maximum of tm1 over tiles [64m, 64m + 64)
__global__ __launch_bounds__(kBS) void k_tile_max2(const int64_t *__restrict__ pC, int32_t T,
                                                   const int32_t *__restrict__ tm1,
                                                   int32_t *__restrict__ tm2) {
    const int64_t C1 = (*pC + 63) / 64;   // tiles of 64 candidates
    const int64_t k = (int64_t)blockIdx.x * kBS + threadIdx.x;
    const int64_t m = k >> 6;
    if ((m << 6) >= C1) return;          // whole waves past the last tile
    for (int32_t ts = 0; ts < T; ts++) {
        int64_t r = k < C1 ? tm1[k * T + ts] : -1;
        r = wave_max64(r);
        if ((threadIdx.x & 63) == 0 && (m << 6) < C1) tm2[m * T + ts] = (int32_t)r;
    }
}

struct WinArgs {
    int32_t T, wlog;                    // window of 2^wlog entries per thread
    const int64_t *base;                // [T+1]
    const int64_t *cbase;               // [T+1]
    const CandEnt *pent;                // [C]
    const int64_t *req_ptr;             // [C+1]
    const int32_t *req_chain;
    const int64_t *req_gpos;
    const int32_t *tm1, *tm2;           // tile maxima (tiles of 64 and 4096 candidates)
    int32_t *ftab;                      // [(n+1) x T] fronts at the start of each round
    int64_t *result;                    // [0] steps
    uint32_t *err;
};

__device__ __forceinline__ bool win_blocked(const WinArgs &a, const CandEnt &e, int64_t j,
                                            const int32_t *front) {
    const uint32_t nd = e.meta >> 16;
    if (e.g0 >= front[e.meta & 0xff]) return true;
    if (nd > 1 && e.g1 >= front[(e.meta >> 8) & 0xff]) return true;
    if (nd > 2) {                        // parents on three or more threads
        for (int64_t k = a.req_ptr[j]; k < a.req_ptr[j + 1]; k++)
            if (a.req_gpos[k] >= front[a.req_chain[k]]) return true;
    }
    return false;
}

// One barrier per round: round r reads the fronts of buffer r & 1 and writes
// the advanced fronts, plus one flag per thread (advanced, unfinished), into
// buffer (r + 1) & 1 and r & 1; a buffer is rewritten only two rounds later,
// after the next barrier.  The fronts of every round go to a table from which
// the segments are cut afterwards (k_win_seg_*).
__global__ __launch_bounds__(kWG) void k_kahn_win(WinArgs a) {
    static_assert(kWG / 64 >= kWinT, "a wave per graph thread");
    constexpr int kWinE = kWinBytes / (int)sizeof(CandEnt);
    __shared__ CandEnt s_win[kWinE + 64];
    __shared__ __align__(16) int32_t s_front[2][kWinT];
    __shared__ __align__(16) uint8_t s_adv[2][16], s_unf[2][16];   // flags of graph threads
    const int lane = threadIdx.x & 63;
    // wave t walks graph thread t (uniform: the wave's state stays scalar)
    const int t = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const int W = 1 << a.wlog;
    const int T = a.T;
    const bool mine = t < T;
    CandEnt *const win = s_win + (mine ? t : 0) * W;
    // the wave's own thread: front end, candidate range and window in registers
    const int end = mine ? (int)a.base[t + 1] : 0;
    const int ce = mine ? (int)a.cbase[t + 1] : 0;
    int ci = mine ? (int)a.cbase[t] : 0;
    int wend = ci;
    int f = mine ? (int)a.base[t] : 0;             // the wave's own front (also in LDS for the others)
    if (threadIdx.x < 32) reinterpret_cast<uint8_t *>(s_adv)[threadIdx.x] = 0;
    if (threadIdx.x < 32) reinterpret_cast<uint8_t *>(s_unf)[threadIdx.x] = 0;
    if (threadIdx.x < 2 * kWinT) s_front[0][threadIdx.x] = 0;   // fronts past T stay 0
    __syncthreads();
    if (threadIdx.x < T) {
        s_front[0][threadIdx.x] = (int32_t)a.base[threadIdx.x];
        a.ftab[threadIdx.x] = (int32_t)a.base[threadIdx.x];
    }
    __syncthreads();
    int64_t round = 0;
    int32_t frow = 0;                             // front table rows of the current batch
    for (;;) {
        const int cur = (int)(round & 1);
        // refill this thread's window when less than half of it lies ahead
        if (mine && wend < ce && wend - ci < (W >> 1)) {
            // all loads of a refill are in flight together (one memory latency)
            const int nend = ci + W < ce ? ci + W : ce;
            const int from = wend > ci ? wend : ci;     // entries behind ci are spent
            for (int j0 = from; j0 < nend; j0 += kRefill * 64) {
                CandEnt v[kRefill];
#pragma unroll
                for (int r = 0; r < kRefill; r++) {
                    const int j = j0 + r * 64 + lane;
                    v[r] = a.pent[j < nend ? j : from];
                }
#pragma unroll
                for (int r = 0; r < kRefill; r++) {   // past the end: a spare slot
                    const int j = j0 + r * 64 + lane;
                    CandEnt *dst = j < nend ? &win[j & (W - 1)] : &s_win[kWinE + lane];
                    *dst = v[r];
                }
            }
            wend = nend;
        }
        // advance this thread's front past its ready candidates
        if (mine) {
            int cnew = ce;
            int npos = end;                        // order position of candidate cnew (end if none)
            const int32_t *front = s_front[cur];
            if (f < end) {
                for (;;) {
                    if (ci >= ce) { cnew = ce; break; }
                    if (ci < wend) {
                        const int lim = wend < ce ? wend : ce;
                        const int j = ci + lane;
                        const CandEnt e = win[j & (W - 1)];
                        const bool bl = j < lim && win_blocked(a, e, j, front);
                        const unsigned long long bal = __ballot(bl);
                        if (bal) {
                            const int L = __ffsll((long long)bal) - 1;
                            cnew = ci + L;
                            npos = __builtin_amdgcn_readlane(e.pos, L);   // the finder's entry
                            break;
                        }
                        ci = ci + 64 < lim ? ci + 64 : lim;
                    } else {
                        // past the window (a long ready run): tiles of 4096,
                        // then of 64, then single candidates, 64 per probe
                        int32_t fr[kWinT];         // the round's fronts (wave-uniform)
#pragma unroll
                        for (int q = 0; q < kWinT / 4; q++) {
                            const int4 v = reinterpret_cast<const int4 *>(front)[q];
                            fr[4 * q] = v.x; fr[4 * q + 1] = v.y; fr[4 * q + 2] = v.z; fr[4 * q + 3] = v.w;
                        }
                        auto tile_blocked = [&](const int32_t *row) {
                            bool b = false;
#pragma unroll
                            for (int ts = 0; ts < kWinT; ts++)
                                if (ts < T && row[ts] >= fr[ts]) b = true;
                            return b;
                        };
                        int64_t pos = ci;          // every candidate before pos is ready
                        cnew = ce;
                        while (pos < ce) {
                            const int64_t k2 = pos >> 12, t2 = k2 + lane;
                            const bool b2 = (t2 << 12) < ce && tile_blocked(a.tm2 + t2 * T);
                            const unsigned long long bal2 = __ballot(b2);
                            if (!bal2) { pos = (k2 + 64) << 12; continue; }
                            const int64_t L2 = k2 + __ffsll((long long)bal2) - 1;
                            pos = pos > (L2 << 12) ? pos : (L2 << 12);
                            const int64_t end2 = ce < ((L2 + 1) << 12) ? ce : ((L2 + 1) << 12);
                            const int64_t k1 = pos >> 6, t1 = k1 + lane;
                            const bool b1 = (t1 << 6) < end2 && tile_blocked(a.tm1 + t1 * T);
                            const unsigned long long bal1 = __ballot(b1);
                            if (!bal1) { pos = end2; continue; }
                            const int64_t L1 = k1 + __ffsll((long long)bal1) - 1;
                            pos = pos > (L1 << 6) ? pos : (L1 << 6);
                            const int64_t end1 = ce < ((L1 + 1) << 6) ? ce : ((L1 + 1) << 6);
                            const int64_t j = pos + lane;
                            const CandEnt e1 = a.pent[j < end1 ? j : pos];
                            const bool b0 = j < end1 && win_blocked(a, e1, j, front);
                            const unsigned long long bal0 = __ballot(b0);
                            if (bal0) {
                                const int L = __ffsll((long long)bal0) - 1;
                                cnew = (int)(pos + L);
                                npos = __builtin_amdgcn_readlane(e1.pos, L);
                                break;
                            }
                            pos = end1;
                        }
                        break;
                    }
                }
            } else {
                cnew = ci;
            }
            const int nf = f >= end ? f : (cnew < ce ? npos : end);
            if (lane == 0) {
                s_front[cur ^ 1][t] = nf;
                s_adv[cur][t] = nf > f;
                s_unf[cur][t] = f < end;
            }
            // front table row round + 1: lane (round & 63) keeps it until a
            // batch of 64 rows goes out in one store (a store each round would
            // make the next round wait for it)
            const int slotr = (int)(round & 63);
            frow = lane == slotr ? nf : frow;
            if (slotr == 63) a.ftab[(round - 63 + lane + 1) * T + t] = frow;
            ci = cnew;
            f = nf;
        }
        __syncthreads();
        // every wave reads the same flags: all threads done, or a stall (cycle)
        const uint4 uf = *reinterpret_cast<const uint4 *>(s_unf[cur]);
        const uint4 av = *reinterpret_cast<const uint4 *>(s_adv[cur]);
        const bool unf = (uf.x | uf.y | uf.z | uf.w) != 0;
        const bool adv = (av.x | av.y | av.z | av.w) != 0;
        if (!unf || !adv) {
            if (!unf) {
                // rows of the last, partial batch
                const int slotr = (int)(round & 63);
                if (mine && slotr != 63 && lane <= slotr)
                    a.ftab[(round - slotr + lane + 1) * T + t] = frow;
            } else if (threadIdx.x == 0) {
                atomicOr(a.err, ERR_KAHN_CYCLE);
            }
            break;
        }
        round++;
    }
    if (threadIdx.x == 0) a.result[0] = round;
}

// segments from the front table: thread t advanced in round r when its front
// moved; segments are numbered in (round, thread) order
__global__ __launch_bounds__(kBS) void k_win_seg_count(int64_t R, int32_t T,
                                                       const int32_t *__restrict__ ftab,
                                                       int64_t *__restrict__ cnt) {
    const int64_t i = (int64_t)blockIdx.x * kBS + threadIdx.x;
    if (i < R * T) cnt[i] = ftab[i + T] > ftab[i];
}

// The position offset of segment (r, t) comes straight from the front table:
// every thread's advance before round r, plus the advances of lower threads
// in round r.  nseg[0] receives the segment count; seg_off[nseg] = n.
__global__ __launch_bounds__(kBS) void k_win_seg_fill(int64_t R, int32_t T,
                                                      const int32_t *__restrict__ ftab,
                                                      const int64_t *__restrict__ off,
                                                      int64_t *__restrict__ seg_start,
                                                      int64_t *__restrict__ seg_len,
                                                      int64_t *__restrict__ seg_off,
                                                      int32_t *__restrict__ seg_step,
                                                      int64_t *__restrict__ step_seg,
                                                      int64_t *__restrict__ nseg) {
    const int64_t i = (int64_t)blockIdx.x * kBS + threadIdx.x;
    if (i > R * T) return;
    if (i % T == 0) step_seg[i / T] = off[i];          // i == R*T gives the total
    const int64_t r = i / T;
    const int t = (int)(i % T);
    if (i == R * T) {
        nseg[0] = off[i];
        int64_t done = 0;
        for (int z = 0; z < T; z++) done += ftab[R * T + z] - ftab[z];
        seg_off[off[i]] = done;
        return;
    }
    const int32_t f0 = ftab[i], f1 = ftab[i + T];
    if (f1 > f0) {
        int64_t o = 0;
        for (int z = 0; z < T; z++) o += ftab[r * T + z] - ftab[z];
        for (int z = 0; z < t; z++) o += ftab[(r + 1) * T + z] - ftab[r * T + z];
        const int64_t sidx = off[i];
        seg_start[sidx] = f0;
        seg_len[sidx] = f1 - f0;
        seg_off[sidx] = o;
        seg_step[sidx] = (int32_t)r;
    }
}

// positions in step order: segment of each position by binary search
__global__ __launch_bounds__(kBS) void k_positions(
    int64_t n, const int64_t *__restrict__ pnseg, const int64_t *__restrict__ seg_off,
    const int64_t *__restrict__ seg_start,
    const int32_t *__restrict__ seg_step, const int32_t *__restrict__ order,
    const int64_t *__restrict__ dur, const int64_t *__restrict__ gap,
    const uint16_t *__restrict__ cls, int32_t *__restrict__ pos_node,
    uint8_t *__restrict__ pos_flags, int64_t *__restrict__ pos_dur,
    int64_t *__restrict__ pos_gap, uint16_t *__restrict__ pos_cls,
    int32_t *__restrict__ node_step) {
    const int64_t q = (int64_t)blockIdx.x * kBS + threadIdx.x;
    if (q >= n) return;
    const int64_t nseg = *pnseg;
    int64_t lo = 0, hi = nseg - 1;          // last segment with seg_off <= q
    while (lo < hi) {
        const int64_t mid = (lo + hi + 1) >> 1;
        if (seg_off[mid] <= q) lo = mid; else hi = mid - 1;
    }
    const int64_t p = seg_start[lo] + (q - seg_off[lo]);
    const int32_t u = order[p];
    pos_node[q] = u;
    pos_flags[q] = (q == seg_off[lo]) ? 1 : 0;
    pos_dur[q] = dur[u];
    pos_gap[q] = gap[u];
    pos_cls[q] = cls ? cls[u] : 0;
    node_step[u] = seg_step[lo];
}

__global__ __launch_bounds__(kBS) void k_step_ptr(int64_t nsteps, const int64_t *__restrict__ step_seg,
                                                  const int64_t *__restrict__ seg_off,
                                                  int32_t *__restrict__ step_ptr) {
    const int64_t r = (int64_t)blockIdx.x * kBS + threadIdx.x;
    if (r <= nsteps) step_ptr[r] = (int32_t)seg_off[step_seg[r]];
}

// gathers per position: thread predecessor for run heads + active cross parents
__global__ __launch_bounds__(kBS) void k_gather_count(int64_t n, const int32_t *__restrict__ pos_node,
                                                      const uint8_t *__restrict__ pos_flags,
                                                      const int32_t *__restrict__ prev,
                                                      const int64_t *__restrict__ xin_ptr,
                                                      const uint8_t *__restrict__ xin_cls,
                                                      uint64_t mask, bool with_prev,
                                                      int64_t *__restrict__ cnt) {
    const int64_t q = (int64_t)blockIdx.x * kBS + threadIdx.x;
    if (q >= n) return;
    const int32_t u = pos_node[q];
    int64_t c = (with_prev && (pos_flags[q] & 1) && prev[u] >= 0) ? 1 : 0;
    for (int64_t k = xin_ptr[u]; k < xin_ptr[u + 1]; k++) c += on(mask, xin_cls[k]);
    cnt[q] = c;
}

__global__ __launch_bounds__(kBS) void k_gather_fill(
    int64_t n, const int32_t *__restrict__ pos_node, const uint8_t *__restrict__ pos_flags,
    const int32_t *__restrict__ prev, const int64_t *__restrict__ xin_ptr,
    const int32_t *__restrict__ xin_src, const uint8_t *__restrict__ xin_cls, uint64_t mask,
    bool with_prev, const int64_t *__restrict__ gap, const int64_t *__restrict__ gptr,
    int32_t *__restrict__ gsrc, int32_t *__restrict__ gpos, uint8_t *__restrict__ gcls,
    int64_t *__restrict__ ggap) {
    const int64_t q = (int64_t)blockIdx.x * kBS + threadIdx.x;
    if (q >= n) return;
    const int32_t u = pos_node[q];
    int64_t o = gptr[q];
    if (with_prev && (pos_flags[q] & 1) && prev[u] >= 0) {
        gsrc[o] = prev[u]; gpos[o] = (int32_t)q; gcls[o] = 255; ggap[o] = gap[prev[u]];
        o++;
    }
    for (int64_t k = xin_ptr[u]; k < xin_ptr[u + 1]; k++) {
        if (!on(mask, xin_cls[k])) continue;
        const int32_t s = xin_src[k];
        gsrc[o] = s; gpos[o] = (int32_t)q; gcls[o] = xin_cls[k]; ggap[o] = gap[s];
        o++;
    }
}

__global__ __launch_bounds__(kBS) void k_inverse(int64_t n, const int32_t *__restrict__ pos_node,
                                                 int32_t *__restrict__ pos_of) {
    const int64_t q = (int64_t)blockIdx.x * kBS + threadIdx.x;
    if (q < n) pos_of[pos_node[q]] = (int32_t)q;
}

__global__ __launch_bounds__(kBS) void k_gather_spos(const int64_t *__restrict__ pG,
                                                     const int32_t *__restrict__ gsrc,
                                                     const int32_t *__restrict__ pos_of,
                                                     int32_t *__restrict__ gspos) {
    const int64_t e = (int64_t)blockIdx.x * kBS + threadIdx.x;
    if (e < *pG) gspos[e] = pos_of[gsrc[e]];
}

// the per-position record the simulation streams through LDS
__global__ __launch_bounds__(kBS) void k_records(
    int64_t n, const int32_t *__restrict__ tid, const int32_t *__restrict__ pos_node,
    const uint8_t *__restrict__ pos_flags,
    const int64_t *__restrict__ pos_dur, const int64_t *__restrict__ pos_gap,
    const uint16_t *__restrict__ pos_cls, const int64_t *__restrict__ gptr,
    const int32_t *__restrict__ gsrc, const int32_t *__restrict__ gspos,
    const uint8_t *__restrict__ gcls, const int64_t *__restrict__ ggap, Rec *__restrict__ rec) {
    const int64_t q = (int64_t)blockIdx.x * kBS + threadIdx.x;
    if (q >= n) return;
    Rec r;
    r.dur = pos_dur[q];
    r.gap = pos_gap[q];
    r.node = pos_node[q];
    const int32_t t = tid[r.node];
    const int64_t e0 = gptr[q], e1 = gptr[q + 1];
    const int64_t ng = e1 - e0;
    uint32_t c0 = 0, c1 = 0;
    r.g0_src = -1; r.g1_src = -1; r.g0_spos = 0; r.g1_spos = 0;
    r.g0_gap32 = 0;
    if (ng > 0) {
        r.g0_src = gsrc[e0]; r.g0_spos = gspos[e0]; c0 = gcls[e0];
        r.g0_gap32 = (uint32_t)ggap[e0];
    }
    if (ng > 1) { r.g1_src = gsrc[e0 + 1]; r.g1_spos = gspos[e0 + 1]; c1 = gcls[e0 + 1]; }
    r.cls = (uint32_t)pos_cls[q] | (c0 << 16) | (c1 << 24);
    int64_t extra = ng > 2 ? ng - 2 : 0;   // count saturates; the gather pointers are exact
    if (extra > 0xFFFFFF) extra = 0xFFFFFF;
    // last task of a run: the next position starts a run (or the schedule ends)
    const bool last = (q + 1 == n) || (pos_flags[q + 1] & 1);
    r.flags = (uint32_t)(pos_flags[q] & 1) | (last ? 2u : 0u) |
              ((uint32_t)(t < kMaxCarryThreads ? t : 0) << 2) | ((uint32_t)extra << 8);
    rec[q] = r;
}

__global__ __launch_bounds__(kBS) void k_step_width(int64_t nsteps, const int32_t *__restrict__ step_ptr,
                                                    unsigned long long *__restrict__ wmax) {
    const int64_t r = (int64_t)blockIdx.x * kBS + threadIdx.x;
    int64_t w = r < nsteps ? (int64_t)(step_ptr[r + 1] - step_ptr[r]) : 0;
    w = wave_max64(w);
    if ((threadIdx.x & 63) == 0) atomic_max_hot(wmax, (unsigned long long)w);
}

// Kahn levels from the phase schedule (one workgroup, phases in order)
struct LevelArgs {
    int64_t nsteps;
    const int32_t *step_ptr;
    const int32_t *pos_node;
    const uint8_t *pos_flags;
    const int32_t *prev;
    const int64_t *xin_ptr;
    const int32_t *xin_src;
    const uint8_t *xin_cls;
    uint64_t mask;
    int32_t *level;          // [n] by task
    unsigned long long *max_level;
};

__global__ __launch_bounds__(kWG) void k_levels(LevelArgs a) {
    __shared__ int64_t s_val[kWG];
    __shared__ uint8_t s_head[kWG];
    __shared__ int64_t s_tmp[kWG];
    __shared__ uint8_t s_htmp[kWG];
    __shared__ int64_t s_carry;
    int64_t lmax = 0;
    for (int64_t r = 0; r < a.nsteps; r++) {
        const int64_t p0 = a.step_ptr[r], p1 = a.step_ptr[r + 1];
        if (threadIdx.x == 0) s_carry = INT64_MIN / 4;
        __syncthreads();
        for (int64_t w0 = p0; w0 < p1; w0 += kWG) {
            const int64_t q = w0 + threadIdx.x;
            int64_t x = INT64_MIN / 4;
            uint8_t h = 1;
            int32_t u = -1;
            if (q < p1) {
                u = a.pos_node[q];
                h = a.pos_flags[q] & 1;
                int64_t best = 0;
                if (h && a.prev[u] >= 0) best = (int64_t)a.level[a.prev[u]] + 1;
                for (int64_t k = a.xin_ptr[u]; k < a.xin_ptr[u + 1]; k++)
                    if (on(a.mask, a.xin_cls[k])) {
                        const int64_t l = (int64_t)a.level[a.xin_src[k]] + 1;
                        best = l > best ? l : best;
                    }
                x = best - q;          // level_q - q is a running max inside a run
            }
            if (threadIdx.x == 0 && !h) {   // run continues from the previous window
                x = x > s_carry ? x : s_carry;
            }
            s_val[threadIdx.x] = x;
            s_head[threadIdx.x] = h;
            __syncthreads();
            // segmented inclusive max-scan (Hillis-Steele with head flags)
            for (int d = 1; d < kWG; d <<= 1) {
                int64_t v = s_val[threadIdx.x];
                uint8_t hh = s_head[threadIdx.x];
                if ((int)threadIdx.x >= d && !hh) {
                    const int64_t o = s_val[threadIdx.x - d];
                    v = o > v ? o : v;
                    hh = s_head[threadIdx.x - d];
                }
                s_tmp[threadIdx.x] = v;
                s_htmp[threadIdx.x] = hh;
                __syncthreads();
                s_val[threadIdx.x] = s_tmp[threadIdx.x];
                s_head[threadIdx.x] = s_htmp[threadIdx.x];
                __syncthreads();
            }
            if (q < p1) {
                const int64_t lv = s_val[threadIdx.x] + q;
                a.level[u] = (int32_t)lv;
                lmax = lv > lmax ? lv : lmax;
            }
            __syncthreads();
            if (threadIdx.x == kWG - 1) s_carry = s_val[kWG - 1];
            __syncthreads();
        }
    }
    lmax = wave_max64(lmax);
    if ((threadIdx.x & 63) == 0) atomic_max_hot(a.max_level, (unsigned long long)lmax);
}

__global__ __launch_bounds__(kBS) void k_level_count(int32_t n, const int32_t *__restrict__ level,
                                                     int64_t *__restrict__ cnt) {
    const int64_t u = (int64_t)blockIdx.x * kBS + threadIdx.x;
    if (u < n) atomicAdd((unsigned long long *)&cnt[level[u]], 1ull);
}

__global__ __launch_bounds__(kBS) void k_level_scatter(int32_t n, const int32_t *__restrict__ level,
                                                       int64_t *__restrict__ fill,
                                                       const int64_t *__restrict__ dur,
                                                       const int64_t *__restrict__ gap,
                                                       const uint16_t *__restrict__ cls,
                                                       int32_t *__restrict__ pos_node,
                                                       uint8_t *__restrict__ pos_flags,
                                                       int64_t *__restrict__ pos_dur,
                                                       int64_t *__restrict__ pos_gap,
                                                       uint16_t *__restrict__ pos_cls,
                                                       int32_t *__restrict__ node_step) {
    const int64_t u = (int64_t)blockIdx.x * kBS + threadIdx.x;
    if (u >= n) return;
    const int32_t l = level[u];
    const int64_t q = (int64_t)atomicAdd((unsigned long long *)&fill[l], 1ull);
    pos_node[q] = (int32_t)u;
    pos_flags[q] = 1;            // every task is its own run: thread predecessor gathered
    pos_dur[q] = dur[u];
    pos_gap[q] = gap[u];
    pos_cls[q] = cls ? cls[u] : 0;
    node_step[u] = l;
}

__global__ __launch_bounds__(kBS) void k_i64_to_i32(int64_t n, const int64_t *__restrict__ in,
                                                    int32_t *__restrict__ out) {
    const int64_t i = (int64_t)blockIdx.x * kBS + threadIdx.x;
    if (i < n) out[i] = (int32_t)in[i];
}

}  // namespace

#define CK(x)                                                              \
    do {                                                                   \
        hipError_t e_ = (x);                                               \
        if (e_ != hipSuccess) {                                            \
            snprintf(msg, msg_len, "%s: %s", #x, hipGetErrorString(e_));   \
            st = e_ == hipErrorOutOfMemory ? DD_ENOMEM : DD_EHIP;          \
            goto done;                                                     \
        }                                                                  \
    } while (0)

dd_status levelize_device(const dd_graph *g, uint64_t mask, int32_t mode, dd_sched *sch,
                          hipStream_t s, char *msg, size_t msg_len) {
    dd_status st = DD_OK;
    const int64_t n = g->n;
    const int32_t T = g->n_threads;
    const int64_t N1 = n + 1;
    const int64_t Cmax = n;                  // candidates <= tasks
    const int64_t Rmax = g->n_cross;         // requirements <= cross edges
    int64_t *cnt = nullptr, *flag = nullptr, *cidx = nullptr, *rptr = nullptr, *cand_pos = nullptr,
            *req_ptr = nullptr, *req_gpos = nullptr, *cbase = nullptr, *front = nullptr,
            *ci = nullptr, *nfront = nullptr, *nci = nullptr, *seg_start = nullptr,
            *seg_len = nullptr, *seg_off = nullptr, *step_seg = nullptr, *result = nullptr,
            *gcnt = nullptr, *lvl_cnt = nullptr;
    int32_t *req_chain = nullptr, *long_list = nullptr, *seg_step = nullptr, *level = nullptr;
    CandEnt *pent = nullptr;
    int32_t *ftab = nullptr, *tm1 = nullptr, *tm2 = nullptr;
    int64_t *seg_cnt = nullptr;
    const bool windowed = T <= kWinT;
    uint32_t *err = nullptr;
    unsigned long long *wmax = nullptr;
    int64_t h_res[2] = {0, 0};
    uint32_t h_err = 0;
    unsigned long long h_w = 0;
    Req rq{g->thread_base, g->order, g->rank, g->thread_id, g->xin_ptr, g->xin_src, g->xin_cls};
    const int gN = grid_for(n, kBS);

    sch->n = (int32_t)n;
    sch->mode = mode;
    sch->mask = mask;
    sch->thread_carry = T <= kMaxCarryThreads;
    CK(dalloc_n(&cnt, N1, s));
    CK(dalloc_n(&flag, N1, s));
    CK(dalloc_n(&cidx, N1, s));
    CK(dalloc_n(&rptr, N1, s));
    CK(dalloc_n(&err, 1, s));
    CK(dalloc_n(&result, 4, s));
    CK(dalloc_n(&wmax, 1, s));
    CK(hipMemsetAsync(err, 0, sizeof(uint32_t), s));
    CK(hipMemsetAsync(result, 0, 4 * sizeof(int64_t), s));
    CK(hipMemsetAsync(wmax, 0, sizeof(unsigned long long), s));
    if (n > 0) {
        k_req_count<<<gN, kBS, 0, s>>>((int32_t)n, rq, mask, cnt, flag);
        CK(hipGetLastError());
    }
    CK(scan_exclusive(flag, cidx, n, s));
    CK(scan_exclusive(cnt, rptr, n, s));
    // sized by their bounds, so no count has to come back to the host first
    CK(dalloc_n(&cand_pos, (size_t)Cmax + 1, s));
    CK(dalloc_n(&req_ptr, (size_t)Cmax + 1, s));
    CK(dalloc_n(&req_chain, (size_t)Rmax + 1, s));
    CK(dalloc_n(&req_gpos, (size_t)Rmax + 1, s));
    if (T <= kEntT) CK(dalloc_n(&pent, (size_t)Cmax + 1, s));
    CK(dalloc_n(&cbase, (size_t)T + 1, s));
    CK(dalloc_n(&front, (size_t)T, s));
    CK(dalloc_n(&ci, (size_t)T, s));
    CK(dalloc_n(&nfront, (size_t)T, s));
    CK(dalloc_n(&nci, (size_t)T, s));
    CK(dalloc_n(&long_list, (size_t)T, s));
    CK(dalloc_n(&seg_start, N1, s));
    CK(dalloc_n(&seg_len, N1, s));
    CK(dalloc_n(&seg_step, N1, s));
    CK(dalloc_n(&seg_off, N1 + 1, s));
    CK(dalloc_n(&step_seg, N1 + 1, s));
    if (n > 0) {
        k_req_fill<<<gN, kBS, 0, s>>>((int32_t)n, T, rq, mask, cidx, rptr, cand_pos, req_ptr,
                                      req_chain, req_gpos, pent);
        CK(hipGetLastError());
    }
    k_cand_base<<<grid_for((int64_t)T + 1, kBS), kBS, 0, s>>>(T, n, g->thread_base, cidx, rptr,
                                                               req_ptr, cbase, front, ci);
    CK(hipGetLastError());
    if (windowed) {
        int wlog = 6;                                  // 2^wlog entries per thread
        while ((int64_t)T << (wlog + 1) <= kWinBytes / (int64_t)sizeof(CandEnt)) wlog++;
        CK(dalloc_n(&ftab, (size_t)(n + 2) * T, s));
        const int64_t C1 = (Cmax + 63) / 64, C2 = (C1 + 63) / 64;   // tiles at most
        CK(dalloc_n(&tm1, (size_t)(C1 > 0 ? C1 : 1) * T, s));
        CK(dalloc_n(&tm2, (size_t)(C2 > 0 ? C2 : 1) * T, s));
        if (n > 0) {
            k_tile_max1<<<grid_for(C1 * 64, kBS), kBS, 0, s>>>(cidx + n, T, req_ptr, req_chain,
                                                               req_gpos, tm1);
            CK(hipGetLastError());
            k_tile_max2<<<grid_for(C2 * 64, kBS), kBS, 0, s>>>(cidx + n, T, tm1, tm2);
            CK(hipGetLastError());
        }
        WinArgs wa{T, wlog, g->thread_base, cbase, pent, req_ptr, req_chain, req_gpos,
                   tm1, tm2, ftab, result, err};
        k_kahn_win<<<1, kWG, 0, s>>>(wa);
        CK(hipGetLastError());
    } else {
        KahnArgs ka{pent, T, n, g->thread_base, cand_pos, cbase, req_ptr, req_chain, req_gpos,
                    front, ci, nfront, nci, long_list, seg_start, seg_len, seg_step, step_seg,
                    result, err};
        if (T <= kLdsT) k_kahn_rounds<true><<<1, kWG, 0, s>>>(ka);
        else k_kahn_rounds<false><<<1, kWG, 0, s>>>(ka);
        CK(hipGetLastError());
    }
    {
        ReadBack rb(s, 2 * sizeof(int64_t) + sizeof(uint32_t));
        CK(rb.add(h_res, result, 2 * sizeof(int64_t)));
        CK(rb.add(&h_err, err, sizeof(uint32_t)));
        CK(rb.finish());
    }
    if (h_err & ERR_KAHN_CYCLE) {
        snprintf(msg, msg_len, "dependencies plus thread order contain a cycle "
                               "(Kahn rounds stalled after %lld steps)", (long long)h_res[0]);
        st = DD_ECYCLE;
        goto done;
    }
    if (windowed) {                                    // cut the segments from the fronts
        const int64_t R = h_res[0], RT = R * T;
        CK(dalloc_n(&seg_cnt, (size_t)RT + 1, s));
        if (RT > 0) {
            k_win_seg_count<<<grid_for(RT, kBS), kBS, 0, s>>>(R, T, ftab, seg_cnt);
            CK(hipGetLastError());
        }
        CK(scan_exclusive(seg_cnt, seg_cnt, RT, s));
        k_win_seg_fill<<<grid_for(RT + 1, kBS), kBS, 0, s>>>(R, T, ftab, seg_cnt, seg_start,
                                                             seg_len, seg_off, seg_step, step_seg,
                                                             result + 1);
        CK(hipGetLastError());
    }
    {
        // (the windowed rounds leave the segment count on the device; it
        // comes back with the gather count below)
        const int64_t nph = h_res[0];
        if (!windowed) CK(scan_exclusive(seg_len, seg_off, h_res[1], s));
        CK(dalloc_n(&sch->pos_node, N1, s));
        CK(dalloc_n(&sch->pos_flags, N1, s));
        CK(dalloc_n(&sch->pos_dur, N1, s));
        CK(dalloc_n(&sch->pos_gap, N1, s));
        CK(dalloc_n(&sch->pos_cls, N1, s));
        CK(dalloc_n(&sch->node_step, N1, s));
        CK(dalloc_n(&sch->gat_ptr, N1, s));
        if (n > 0) {
            k_positions<<<gN, kBS, 0, s>>>(n, result + 1, seg_off, seg_start, seg_step, g->order, g->dur,
                                           g->gap, g->cls, sch->pos_node, sch->pos_flags,
                                           sch->pos_dur, sch->pos_gap, sch->pos_cls,
                                           sch->node_step);
            CK(hipGetLastError());
        }
        if (mode == DD_PHASES) {
            sch->n_steps = nph;
            CK(dalloc_n(&sch->step_ptr, (size_t)nph + 1, s));
            k_step_ptr<<<grid_for(nph + 1, kBS), kBS, 0, s>>>(nph, step_seg, seg_off, sch->step_ptr);
            CK(hipGetLastError());
        } else {
            // levels from phases, then tasks sorted by level
            int32_t *tmp_ptr = nullptr;
            unsigned long long *lmax = nullptr;
            unsigned long long h_lmax = 0;
            CK(dalloc_n(&level, N1, s));
            CK(dalloc_n(&tmp_ptr, (size_t)nph + 1, s));
            CK(dalloc_n(&lmax, 1, s));
            CK(hipMemsetAsync(lmax, 0, sizeof(unsigned long long), s));
            k_step_ptr<<<grid_for(nph + 1, kBS), kBS, 0, s>>>(nph, step_seg, seg_off, tmp_ptr);
            LevelArgs la{nph, tmp_ptr, sch->pos_node, sch->pos_flags, g->thread_prev, g->xin_ptr,
                         g->xin_src, g->xin_cls, mask, level, lmax};
            k_levels<<<1, kWG, 0, s>>>(la);
            CK(hipGetLastError());
            {
                ReadBack rb(s, sizeof(h_lmax));
                CK(rb.add(&h_lmax, lmax, sizeof(h_lmax)));
                CK(rb.finish());
            }
            dfree(tmp_ptr, s);
            dfree(lmax, s);
            const int64_t nl = n > 0 ? (int64_t)h_lmax + 1 : 0;
            CK(dalloc_n(&lvl_cnt, (size_t)nl + 1, s));
            CK(hipMemsetAsync(lvl_cnt, 0, sizeof(int64_t) * ((size_t)nl + 1), s));
            if (n > 0) {
                k_level_count<<<gN, kBS, 0, s>>>((int32_t)n, level, lvl_cnt);
                CK(hipGetLastError());
            }
            CK(scan_exclusive(lvl_cnt, lvl_cnt, nl, s));
            CK(dalloc_n(&sch->step_ptr, (size_t)nl + 1, s));
            k_i64_to_i32<<<grid_for(nl + 1, kBS), kBS, 0, s>>>(nl + 1, lvl_cnt, sch->step_ptr);
            CK(hipGetLastError());
            if (n > 0) {
                k_level_scatter<<<gN, kBS, 0, s>>>((int32_t)n, level, lvl_cnt, g->dur, g->gap,
                                                   g->cls, sch->pos_node, sch->pos_flags,
                                                   sch->pos_dur, sch->pos_gap, sch->pos_cls,
                                                   sch->node_step);
                CK(hipGetLastError());
            }
            sch->n_steps = nl;
            sch->n_segments = n;
        }
        // gathers
        CK(dalloc_n(&gcnt, N1, s));
        if (n > 0) {
            k_gather_count<<<gN, kBS, 0, s>>>(n, sch->pos_node, sch->pos_flags, g->thread_prev,
                                              g->xin_ptr, g->xin_cls, mask, !sch->thread_carry,
                                              gcnt);
            CK(hipGetLastError());
        }
        CK(scan_exclusive(gcnt, sch->gat_ptr, n, s));
        // gather lists sized by their bound (cross edges, plus one thread
        // predecessor per run head without thread carries); the count comes
        // back with the last read-back
        const int64_t Gmax = g->n_cross + (sch->thread_carry ? 0 : n);
        CK(dalloc_n(&sch->gat_src, (size_t)Gmax + 1, s));
        CK(dalloc_n(&sch->gat_pos, (size_t)Gmax + 1, s));
        CK(dalloc_n(&sch->gat_cls, (size_t)Gmax + 1, s));
        CK(dalloc_n(&sch->gat_gap, (size_t)Gmax + 1, s));
        if (n > 0) {
            k_gather_fill<<<gN, kBS, 0, s>>>(n, sch->pos_node, sch->pos_flags, g->thread_prev,
                                             g->xin_ptr, g->xin_src, g->xin_cls, mask,
                                             !sch->thread_carry, g->gap,
                                             sch->gat_ptr, sch->gat_src, sch->gat_pos,
                                             sch->gat_cls, sch->gat_gap);
            CK(hipGetLastError());
        }
        {
            int32_t *pos_of = nullptr;
            CK(dalloc_n(&pos_of, N1, s));
            CK(dalloc_n(&sch->gat_spos, (size_t)Gmax + 1, s));
            CK(dalloc_n(&sch->rec, N1, s));
            if (n > 0) {
                k_inverse<<<gN, kBS, 0, s>>>(n, sch->pos_node, pos_of);
                if (Gmax > 0)
                    k_gather_spos<<<grid_for(Gmax, kBS), kBS, 0, s>>>(sch->gat_ptr + n, sch->gat_src,
                                                                     pos_of, sch->gat_spos);
                k_records<<<gN, kBS, 0, s>>>(n, g->thread_id, sch->pos_node, sch->pos_flags, sch->pos_dur,
                                             sch->pos_gap, sch->pos_cls, sch->gat_ptr, sch->gat_src,
                                             sch->gat_spos, sch->gat_cls, sch->gat_gap, sch->rec);
                CK(hipGetLastError());
            }
            dfree(pos_of, s);
        }
        k_step_width<<<grid_for(sch->n_steps, kBS), kBS, 0, s>>>(sch->n_steps, sch->step_ptr, wmax);
        CK(hipGetLastError());
        int64_t h_G = 0;
        const bool keep_steps = sch->n_steps <= kSplitMaxSteps;
        if (keep_steps) sch->h_step_ptr.resize((size_t)sch->n_steps + 1);
        ReadBack rb(s, sizeof(h_w) + 2 * sizeof(int64_t) +
                           (keep_steps ? sizeof(int32_t) * ((size_t)sch->n_steps + 1) : 0));
        CK(rb.add(&h_w, wmax, sizeof(h_w)));
        CK(rb.add(&h_G, sch->gat_ptr + n, sizeof(int64_t)));
        if (mode == DD_PHASES) CK(rb.add(&h_res[1], result + 1, sizeof(int64_t)));
        if (keep_steps)
            CK(rb.add(sch->h_step_ptr.data(), sch->step_ptr,
                      sizeof(int32_t) * ((size_t)sch->n_steps + 1)));
        CK(rb.finish());
        sch->max_width = (int64_t)h_w;
        sch->n_gathers = h_G;
        if (mode == DD_PHASES) sch->n_segments = h_res[1];
    }
done:
    dfree(cnt, s); dfree(flag, s); dfree(cidx, s); dfree(rptr, s); dfree(err, s);
    dfree(result, s); dfree(wmax, s); dfree(cand_pos, s); dfree(req_ptr, s);
    dfree(req_chain, s); dfree(req_gpos, s); dfree(cbase, s); dfree(front, s); dfree(ci, s);
    dfree(nfront, s); dfree(nci, s); dfree(long_list, s); dfree(seg_start, s);
    dfree(seg_len, s); dfree(seg_off, s); dfree(seg_step, s); dfree(step_seg, s);
    dfree(gcnt, s); dfree(lvl_cnt, s); dfree(level, s); dfree(pent, s);
    dfree(ftab, s); dfree(tm1, s); dfree(tm2, s); dfree(seg_cnt, s);
    return st;
}

}  // namespace dd
