// Batched simulation: every variant of the transformed graph at once (the
// hot path).
//
// What is computed (Sec. 4.1, Algorithm 1, with the transformations of
// Sec. 4.4 applied per variant): for each task u in topological order and
// each variant v,
//     d' = removed ? 0 : floor(d * p / q),   g' = removed ? 0 : g
//     start  = max(0, release of every parent present in v)
//     finish = start + d',   release = finish + g'
//     makespan[v] = max finish over tasks not removed in v.
// Parents are cross-thread dependencies plus the previous task on the
// thread.  The result is unique; Algorithm 1's frontier order does not
// change it when each thread runs its tasks in recorded order.
//
// How.  One workgroup owns VS consecutive variants for the whole graph:
// variants never interact, so the grid needs no synchronization at all
// (no grid barrier, no cross-XCD flags).  The workgroup walks the schedule
// step by step (phases: one run of consecutive tasks per thread).  Inside
// a run, releases follow a max-plus recurrence
//     R_i = max(R_{i-1}, X_i) + w_i      (X_i = max over cross parents)
// whose steps compose associatively:  c -> max(c + A, B).  A round covers
// NS*K positions: NS slots x VS variants (lane = slot*VS + variant, so the
// VS lanes of a slot touch VS consecutive int64 of one task row: finish is
// task-major / variant-minor).  Per round:
//   1. gathers: every (cross parent, variant) pair of the round is read in
//      parallel and max-reduced into LDS (ds_max_i64);
//   2. each lane walks its K positions and keeps local results in registers;
//   3. the (A, B) summaries of the slots are scanned across slots in LDS;
//   4. each lane fixes its K results with its carry-in and stores them.
// Run boundaries inside a round reset the recurrence (segmented scan).

#include "dd_common.cuh"
#include "dd_internal.h"

#include <stdlib.h>

namespace dd {
namespace {

constexpr int kNT = 512;   // threads per workgroup (8 waves)

struct SimArgs {
    int64_t n_steps;
    const int32_t *step_ptr;
    const int32_t *pos_node;
    const uint8_t *pos_flags;
    const int64_t *pos_dur;
    const int64_t *pos_gap;
    const uint16_t *pos_cls;
    const int64_t *gat_ptr;
    const int32_t *gat_src;
    const int32_t *gat_pos;
    const uint8_t *gat_cls;
    const int64_t *gat_gap;
    const ScaleEntry *table;
    const uint32_t *rm;
    const uint64_t *edge_on;
    int32_t V, W;
    int64_t *finish;
    int64_t *start;
    int64_t *makespan;
};

__device__ __forceinline__ int64_t scaled(int64_t d, const ScaleEntry &se) {
    const uint64_t a = (uint64_t)d * (uint64_t)se.p;
    const uint64_t hi = __umul64hi(a, se.magic) >> se.shift;
    const uint64_t lo = a >> se.shift;
    return (int64_t)(se.magic ? hi : lo);
}

__device__ __forceinline__ int64_t max64(int64_t a, int64_t b) { return a > b ? a : b; }

template <int VS, int K>
__global__ __launch_bounds__(kNT) void k_simulate(SimArgs a) {
    constexpr int NS = kNT / VS;       // slots
    constexpr int RP = NS * K;         // positions per round
    constexpr int NE = NS * VS;        // == kNT scan elements
    __shared__ int64_t sX[RP * VS];
    __shared__ int64_t sA[2][NE];
    __shared__ int64_t sB[2][NE];
    __shared__ uint8_t sH[2][NE];
    __shared__ int64_t sCarry[VS];
    __shared__ unsigned long long sMs[VS];

    const int tid = threadIdx.x;
    const int vo = tid % VS;
    const int slot = tid / VS;
    const int v = blockIdx.x * VS + vo;
    const bool vok = v < a.V;
    const int vv = vok ? v : 0;
    const uint64_t eon = a.edge_on[vv];
    const uint32_t vbit = 1u << (vv & 31);
    const int vw = vv >> 5;
    const int64_t V = a.V;
    const int64_t W = a.W;

    if (tid < VS) {
        sMs[tid] = 0;
        sCarry[tid] = 0;
    }
    int64_t ms = 0;
    __syncthreads();

    for (int64_t r = 0; r < a.n_steps; r++) {
        const int p0 = a.step_ptr[r], p1 = a.step_ptr[r + 1];
        for (int r0 = p0; r0 < p1; r0 += RP) {
            const int rn = (p1 - r0) < RP ? (p1 - r0) : RP;
            for (int i = tid; i < rn * VS; i += kNT) sX[i] = 0;
            __syncthreads();
            // 1. gathers: release of each present parent, max-reduced per position
            const int64_t e0 = a.gat_ptr[r0], e1 = a.gat_ptr[r0 + rn];
            for (int64_t e = e0 + slot; e < e1; e += NS) {
                const uint8_t c = a.gat_cls[e];
                if (c == 255 || ((eon >> c) & 1ull)) {
                    const int64_t s = a.gat_src[e];
                    const int64_t f = a.finish[s * V + vv];
                    const bool rmv = (a.rm[s * W + vw] & vbit) != 0;
                    const int64_t rel = f + (rmv ? 0 : a.gat_gap[e]);
                    atomicMax((long long *)&sX[(a.gat_pos[e] - r0) * VS + vo], (long long)rel);
                }
            }
            __syncthreads();
            // 2. local walk over K positions
            int64_t Fl[K], Dp[K], Dd[K];
            int32_t U[K];
            uint32_t valid = 0, before = 0, rmk = 0;
            int64_t A = 0, B = 0;
            bool hh = false;
            const int pb = r0 + slot * K;
#pragma unroll
            for (int k = 0; k < K; k++) {
                const int q = pb + k;
                Fl[k] = 0; Dp[k] = 0; Dd[k] = 0; U[k] = 0;
                if (q < r0 + rn) {
                    valid |= 1u << k;
                    const int32_t u = a.pos_node[q];
                    U[k] = u;
                    const bool head = (a.pos_flags[q] & 1) != 0;
                    const int64_t d = a.pos_dur[q], g = a.pos_gap[q];
                    const ScaleEntry se = a.table[(int64_t)a.pos_cls[q] * V + vv];
                    const bool rmv = (a.rm[(int64_t)u * W + vw] & vbit) != 0;
                    const int64_t dp = rmv ? 0 : scaled(d, se);
                    const int64_t gp = rmv ? 0 : g;
                    const int64_t X = sX[(q - r0) * VS + vo];
                    if (head) { hh = true; A = 0; B = 0; }
                    const int64_t S = max64(B, X);
                    const int64_t F = S + dp;
                    Dp[k] = A + dp;
                    A += dp + gp;
                    B = F + gp;
                    Fl[k] = F;
                    Dd[k] = dp;
                    if (!hh) before |= 1u << k;
                    if (rmv) rmk |= 1u << k;
                }
            }
            // 3. slot summaries; slot 0 absorbs the carry from the previous round
            {
                int64_t Bs = B;
                bool Hs = hh;
                if (slot == 0 && !hh) {
                    Bs = max64(sCarry[vo] + A, B);
                    Hs = true;
                }
                sA[0][tid] = A;
                sB[0][tid] = Bs;
                sH[0][tid] = Hs;
            }
            __syncthreads();
            int cur = 0;
#pragma unroll
            for (int d = 1; d < NS; d <<= 1) {
                int64_t a1 = sA[cur][tid], b1 = sB[cur][tid];
                uint8_t h1 = sH[cur][tid];
                if (slot >= d && !h1) {
                    const int j = tid - d * VS;
                    const int64_t a0 = sA[cur][j], b0 = sB[cur][j];
                    b1 = max64(b0 + a1, b1);
                    a1 = a0 + a1;
                    h1 = sH[cur][j];
                }
                sA[cur ^ 1][tid] = a1;
                sB[cur ^ 1][tid] = b1;
                sH[cur ^ 1][tid] = h1;
                cur ^= 1;
                __syncthreads();
            }
            // 4. finalize with the carry-in of this slot
            const int64_t cin = slot == 0 ? sCarry[vo] : sB[cur][tid - VS];
#pragma unroll
            for (int k = 0; k < K; k++) {
                if (!((valid >> k) & 1u)) continue;
                const int64_t F = ((before >> k) & 1u) ? max64(cin + Dp[k], Fl[k]) : Fl[k];
                if (vok) {
                    const int64_t o = (int64_t)U[k] * V + v;
                    a.finish[o] = F;
                    if (a.start) a.start[o] = F - Dd[k];
                    if (!((rmk >> k) & 1u)) ms = max64(ms, F);
                }
            }
            const int64_t carry_out = sB[cur][(NS - 1) * VS + vo];
            __syncthreads();
            if (slot == 0) sCarry[vo] = carry_out;
        }
    }
    atomicMax(&sMs[vo], (unsigned long long)ms);
    __syncthreads();
    if (slot == 0 && vok) a.makespan[v] = (int64_t)sMs[vo];
}

// ---------------------------------------------------------------------------
// Pipelined form.  A round = up to RP consecutive positions of one step.
// Everything a round reads from global memory is requested one or two
// rounds earlier, so no global round trip sits between two rounds:
//   * schedule records (static) are copied into an LDS ring two rounds
//     ahead (one coalesced 64 B record per position);
//   * the task's removal word and the release of every gather source that
//     finished at least two rounds back ("old") are loaded into registers
//     one round ahead;
//   * a gather source that finished in the previous round ("recent") is
//     read from an LDS copy of that round's releases.
// Per round: walk (registers + LDS) | B1 | issue next loads, scan slot
// summaries per variant with wave shuffles | B2 | finalize, store, refill
// LDS | B3.
struct PipeArgs {
    const int32_t *gat_src;       // gathers beyond two per position
    const int32_t *gat_spos;
    const uint8_t *gat_cls;
    const int64_t *gat_gap;
    const ScaleEntry *table;      // [n_cls][V]
    int32_t n_cls;
    const uint32_t *rm;           // [n][W]
    const uint64_t *edge_on;      // [V]
    int32_t V, W;
    int64_t *finish, *start, *makespan;
    int64_t *dummy;               // [2 * kNT] target of stores from idle lanes
};

constexpr int kTabLds = 2560;     // table entries kept in LDS (40 KB)

typedef __attribute__((address_space(1))) int64_t gi64;   // global-memory int64

// VPL consecutive int64 of one task row (one load or store per lane)
template <int VPL> struct alignas(8) Vals { int64_t x[VPL]; };
typedef long long i64x2 __attribute__((ext_vector_type(2), aligned(8)));
typedef __attribute__((address_space(1))) i64x2 gi64x2;

__device__ __forceinline__ void store_vals(gi64 *o, const Vals<1> &v) { *o = v.x[0]; }
__device__ __forceinline__ void store_vals(gi64 *o, const Vals<2> &v) {
    i64x2 t;
    t.x = v.x[0];
    t.y = v.x[1];
    *(gi64x2 *)o = t;
}

template <int K, int VPL>
struct Dyn {                      // per-lane loads for the next round
    uint32_t rmw[K];              // removal word of the task
    Vals<VPL> f0[K], f1[K];       // finish of old gather sources
    uint32_t r0w[K], r1w[K];      // removal words of those sources
};

__device__ __forceinline__ bool cls_on(uint64_t eon, uint8_t c) {
    return c == 255 || ((eon >> c) & 1ull);
}

// Lane layout: slot = tid / LPS handles K consecutive positions; the LPS
// lanes of a slot each own VPL consecutive variants (VS = LPS * VPL per
// workgroup), so one 8*VPL-byte load or store serves every variant of the
// lane and the per-position bookkeeping is paid once per VPL variants.
// Idle lanes keep issuing the same prefetch loads (clamped addresses) and
// stores (to a dummy target), so the count of memory operations in flight
// is the same on every path and the wait for the next round's data never
// includes this round's stores.
template <int LPS, int VPL, int K, bool TLDS, bool START>
__global__ __launch_bounds__(kNT) void k_sim_pipe(const int32_t *__restrict__ round_r0,
                                                  const int32_t *__restrict__ round_rn,
                                                  const int64_t *__restrict__ n_rounds,
                                                  const Rec *__restrict__ rec, PipeArgs a) {
    constexpr int VS = LPS * VPL;
    constexpr int NS = kNT / LPS;
    constexpr int RP = NS * K;
    constexpr int NE = NS * VS;           // slot summaries (= kNT * VPL)
    static_assert(RP <= kNT, "one record per thread and round");
    static_assert(NE / 64 <= 16, "chunk totals");
    __shared__ Rec sRec[2][RP];
    __shared__ int64_t sR[RP * VS];
    __shared__ int64_t sA[NE], sB[NE];
    __shared__ uint8_t sH[NE];
    __shared__ int64_t sTA[16], sTB[16];
    __shared__ uint8_t sTH[16];
    __shared__ ScaleEntry sT[TLDS ? kTabLds : 1];
    __shared__ unsigned long long sMs[VS];
    __shared__ uint64_t sEon[VS];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int lis = tid % LPS;
    const int slot = tid / LPS;
    const int nwg = gridDim.x;
    // XCD-aware: workgroups dispatched to one XCD (b % 8) own one contiguous
    // block of variants, so neighbouring variant strips of a task row are
    // written through the same L2.
    int wg = blockIdx.x;
    if ((nwg & 7) == 0) wg = (blockIdx.x & 7) * (nwg >> 3) + (blockIdx.x >> 3);
    const int v0 = wg * VS;
    const int vf = v0 + lis * VPL;            // first variant of this lane
    const bool lok = vf < a.V;                // VPL == 2 implies V even: vf + 1 < V too
    const int vvf = lok ? vf : 0;
    const uint32_t vsh = (uint32_t)(vvf & 31);
    const int vw = vvf >> 5;
    const int64_t V = a.V, W = a.W;
    const int64_t nr = *n_rounds;
    const int o0 = lis * VPL;                 // variant offset inside the workgroup
    gi64 *const dummy = (gi64 *)(a.dummy + tid * VPL);

    if (TLDS) {
        for (int i = tid; i < a.n_cls * VS; i += kNT) {
            const int c = i / VS, o = i % VS;
            const int vx = v0 + o < a.V ? v0 + o : 0;
            sT[i] = a.table[(int64_t)c * V + vx];
        }
    }
    if (tid < VS) {
        sMs[tid] = 0;
        // per-variant values read inside the loop live in LDS: a register
        // loaded before the loop would make every round wait for all traffic
        sEon[tid] = a.edge_on[v0 + tid < a.V ? v0 + tid : 0];
    }
    for (int rr = 0; rr < 2; rr++) {          // prologue: records of rounds 0 and 1
        if (rr < nr) {
            const int r0 = round_r0[rr], rn = round_rn[rr];
            for (int i = tid; i < rn; i += kNT) sRec[rr][i] = rec[r0 + i];
        }
    }
    __syncthreads();

    // loads of round kk (records in sRec[kk & 1]); a gather is old when its
    // source position precedes prev_r0 (its round finished two rounds ago)
    auto issue = [&](int64_t kk, int prev_r0, Dyn<K, VPL> &d) {
        const int rn = round_rn[kk];
        const Rec *R = sRec[kk & 1];
#pragma unroll
        for (int i = 0; i < K; i++) {
            const int q = slot * K + i;
            const bool ok = q < rn;
            const int4 w1 = reinterpret_cast<const int4 *>(&R[q])[2];   // node, g0_src, g1_src, g0_spos
            const int g1_spos = reinterpret_cast<const int4 *>(&R[q])[3].x;
            const int32_t node = ok ? w1.x : 0;
            const bool n0 = ok && w1.y >= 0 && w1.w < prev_r0;
            const bool n1 = ok && w1.z >= 0 && g1_spos < prev_r0;
            const int64_t a0 = n0 ? w1.y : 0, a1 = n1 ? w1.z : 0;
            d.rmw[i] = a.rm[(int64_t)node * W + vw];
            if (__any(n0)) {
                d.f0[i] = *reinterpret_cast<const Vals<VPL> *>(a.finish + a0 * V + vvf);
                d.r0w[i] = a.rm[a0 * W + vw];
            }
            if (__any(n1)) {
                d.f1[i] = *reinterpret_cast<const Vals<VPL> *>(a.finish + a1 * V + vvf);
                d.r1w[i] = a.rm[a1 * W + vw];
            }
        }
    };
    Dyn<K, VPL> D;
    if (nr > 0) issue(0, 0, D);

    int64_t carry[VPL], ms[VPL];
#pragma unroll
    for (int j = 0; j < VPL; j++) { carry[j] = 0; ms[j] = 0; }
    int prev_r0 = 0;
    for (int64_t k = 0; k < nr; k++) {
        const int r0 = round_r0[k], rn = round_rn[k];
        const Rec *R = sRec[k & 1];
        uint64_t eon[VPL];
#pragma unroll
        for (int j = 0; j < VPL; j++) eon[j] = sEon[o0 + j];
        // next round's loads, issued before this round's walk so they have a
        // whole round to arrive (records of k+1 are in LDS since round k-1)
        Dyn<K, VPL> DN;
        const int64_t k1 = k + 1 < nr ? k + 1 : k;
        issue(k1, r0, DN);
        // records of round k+2: global -> registers now, -> LDS after finalize
        const int64_t k2 = k + 2 < nr ? k + 2 : k;
        const int r0b = round_r0[k2];
        const int nxt_rn = k + 2 < nr ? round_rn[k2] : 0;
        const uint4 *nsrc = reinterpret_cast<const uint4 *>(rec + r0b + (tid < nxt_rn ? tid : 0));
        const uint4 nx0 = nsrc[0], nx1 = nsrc[1], nx2 = nsrc[2], nx3 = nsrc[3];

        // walk: local max-plus recurrence over this slot's K positions
        int64_t Fl[K][VPL], Dp[K][VPL], Dd[K][VPL];
        int32_t U[K];
        int64_t A[VPL], B[VPL];
#pragma unroll
        for (int j = 0; j < VPL; j++) { A[j] = 0; B[j] = 0; }
        uint32_t before = 0, rmk[VPL];
#pragma unroll
        for (int j = 0; j < VPL; j++) rmk[j] = 0;
        bool hh = false;
#pragma unroll
        for (int i = 0; i < K; i++) {
            const int q = slot * K + i;
            const bool ok = q < rn;
            const int4 *r4 = reinterpret_cast<const int4 *>(&R[q]);
            const int4 w0 = r4[0], w1 = r4[1], w2 = r4[2], w3 = r4[3];
            const int64_t dur = ((int64_t)(uint32_t)w0.y << 32) | (uint32_t)w0.x;
            const int64_t gap = ((int64_t)(uint32_t)w0.w << 32) | (uint32_t)w0.z;
            const int64_t g0gap = ((int64_t)(uint32_t)w1.y << 32) | (uint32_t)w1.x;
            const int64_t g1gap = ((int64_t)(uint32_t)w1.w << 32) | (uint32_t)w1.z;
            const int32_t node = w2.x, s0 = w2.y, s1 = w2.z, p0 = w2.w, p1 = w3.x;
            const uint32_t cl = (uint32_t)w3.y;
            const int cls = cl & 0xffff;
            const uint8_t c0 = (cl >> 16) & 0xff, c1 = cl >> 24;
            const uint32_t flags = (uint32_t)w3.z;
            const int32_t ovf = w3.w;
            const bool head = ok && (flags & 1u);
            U[i] = node;
            const bool old0 = p0 < prev_r0, old1 = p1 < prev_r0;
            int i0 = p0 - prev_r0, i1 = p1 - prev_r0;
            i0 = i0 < 0 ? 0 : (i0 >= RP ? RP - 1 : i0);
            i1 = i1 < 0 ? 0 : (i1 >= RP ? RP - 1 : i1);
            const uint32_t extra = ok ? (flags >> 8) : 0u;
#pragma unroll
            for (int j = 0; j < VPL; j++) {
                const uint32_t bit = vsh + j;
                const bool rmv = (D.rmw[i] >> bit) & 1u;
                int64_t X = 0;
                {
                    const int64_t ro = D.f0[i].x[j] + (((D.r0w[i] >> bit) & 1u) ? 0 : g0gap);
                    const int64_t rn0 = sR[i0 * VS + o0 + j];
                    const int64_t rel = old0 ? ro : rn0;
                    const bool on = ok && s0 >= 0 && cls_on(eon[j], c0);
                    X = on ? max64(X, rel) : X;
                }
                {
                    const int64_t ro = D.f1[i].x[j] + (((D.r1w[i] >> bit) & 1u) ? 0 : g1gap);
                    const int64_t rn1 = sR[i1 * VS + o0 + j];
                    const int64_t rel = old1 ? ro : rn1;
                    const bool on = ok && s1 >= 0 && cls_on(eon[j], c1);
                    X = on ? max64(X, rel) : X;
                }
                if (extra) {                                   // rare: wide fan-in
                    for (uint32_t e2 = 0; e2 < extra; e2++) {
                        const int64_t e = (int64_t)ovf + e2;
                        const uint8_t c = a.gat_cls[e];
                        if (!cls_on(eon[j], c)) continue;
                        const int32_t sp = a.gat_spos[e];
                        int64_t rel;
                        if (sp < prev_r0) {
                            const int64_t sx = a.gat_src[e];
                            const bool rs = (a.rm[sx * W + vw] >> bit) & 1u;
                            rel = a.finish[sx * V + vvf + j] + (rs ? 0 : a.gat_gap[e]);
                        } else {
                            rel = sR[(sp - prev_r0) * VS + o0 + j];
                        }
                        X = max64(X, rel);
                    }
                }
                const ScaleEntry se = TLDS ? sT[cls * VS + o0 + j]
                                           : a.table[(int64_t)cls * V + vvf + j];
                const bool live = ok && !rmv;
                const int64_t dp = live ? scaled(dur, se) : 0;
                const int64_t gp = live ? gap : 0;
                A[j] = head ? 0 : A[j];
                B[j] = head ? 0 : B[j];
                const int64_t S = max64(B[j], X);
                const int64_t F = S + dp;
                Dp[i][j] = A[j] + dp;
                A[j] += dp + gp;
                B[j] = F + gp;
                Fl[i][j] = F;
                Dd[i][j] = dp;
                if (rmv) rmk[j] |= 1u << i;
            }
            hh = hh || head;
            if (!hh) before |= 1u << i;
        }
        // slot summaries (variant-major); slot 0 absorbs the carry
#pragma unroll
        for (int j = 0; j < VPL; j++) {
            const int e = (o0 + j) * NS + slot;
            const bool fold = slot == 0 && !hh;
            sA[e] = A[j];
            sB[e] = fold ? max64(carry[j] + A[j], B[j]) : B[j];
            sH[e] = hh || slot == 0;
        }
        __syncthreads();                                     // B1
        // inclusive scan of slot summaries per variant: wave shuffles, then
        // earlier 64-slot chunks of the same variant
        int64_t xa[VPL], xb[VPL];
        uint8_t xh[VPL];
#pragma unroll
        for (int j = 0; j < VPL; j++) {
            const int e = tid + j * kNT;
            xa[j] = sA[e]; xb[j] = sB[e]; xh[j] = sH[e];
#pragma unroll
            for (int d = 1; d < 64; d <<= 1) {
                const int64_t la = shfl_up64(xa[j], d), lb = shfl_up64(xb[j], d);
                const uint8_t lh = (uint8_t)__shfl_up((int)xh[j], d, 64);
                if (lane >= d && !xh[j]) {
                    xb[j] = max64(lb + xa[j], xb[j]); xa[j] = la + xa[j]; xh[j] = lh;
                }
            }
        }
        if (NS > 64) {
#pragma unroll
            for (int j = 0; j < VPL; j++) {
                const int e = tid + j * kNT;
                if (lane == 63) { sTA[e >> 6] = xa[j]; sTB[e >> 6] = xb[j]; sTH[e >> 6] = xh[j]; }
            }
            __syncthreads();
#pragma unroll
            for (int j = 0; j < VPL; j++) {
                const int e = tid + j * kNT;
                const int chunk = (e % NS) >> 6;
                const int first = (e / NS) * (NS >> 6);
                if (chunk > 0 && !xh[j]) {
                    int64_t pa = sTA[first], pb = sTB[first];
                    uint8_t ph = sTH[first];
                    for (int c = 1; c < chunk; c++) {
                        const int64_t ca = sTA[first + c], cb = sTB[first + c];
                        const uint8_t ch = sTH[first + c];
                        if (!ch) { pb = max64(pb + ca, cb); pa = pa + ca; }
                        else { pa = ca; pb = cb; ph = ch; }
                    }
                    xb[j] = max64(pb + xa[j], xb[j]); xa[j] = pa + xa[j]; xh[j] = ph;
                }
            }
        }
#pragma unroll
        for (int j = 0; j < VPL; j++) {
            const int e = tid + j * kNT;
            sB[e] = xb[j];
        }
        __syncthreads();                                     // B2
        // finalize: carry-in, results, stores, releases for the next round
        int64_t cin[VPL];
#pragma unroll
        for (int j = 0; j < VPL; j++)
            cin[j] = slot == 0 ? carry[j] : sB[(o0 + j) * NS + slot - 1];
#pragma unroll
        for (int i = 0; i < K; i++) {
            const int q = slot * K + i;
            const bool ok = q < rn;
            const int64_t gap = R[q].gap;
            Vals<VPL> fv, sv;
#pragma unroll
            for (int j = 0; j < VPL; j++) {
                const int64_t F = ((before >> i) & 1u) ? max64(cin[j] + Dp[i][j], Fl[i][j]) : Fl[i][j];
                const bool rmv = (rmk[j] >> i) & 1u;
                if (ok) sR[q * VS + o0 + j] = F + (rmv ? 0 : gap);
                fv.x[j] = F;
                sv.x[j] = F - Dd[i][j];
                if (ok && lok && !rmv) ms[j] = max64(ms[j], F);
            }
            const bool st = ok && lok;
            gi64 *o = st ? (gi64 *)(a.finish + ((int64_t)U[i] * V + vf)) : dummy;
            asm volatile("" : "+v"(o));      // keep one unconditional global store
            store_vals(o, fv);
            if (START) {
                gi64 *os = st ? (gi64 *)(a.start + ((int64_t)U[i] * V + vf)) : dummy;
                asm volatile("" : "+v"(os));
                store_vals(os, sv);
            }
        }
#pragma unroll
        for (int j = 0; j < VPL; j++) carry[j] = sB[(o0 + j) * NS + NS - 1];
        if (tid < nxt_rn) {
            uint4 *dst = reinterpret_cast<uint4 *>(&sRec[k & 1][tid]);
            dst[0] = nx0; dst[1] = nx1; dst[2] = nx2; dst[3] = nx3;
        }
        prev_r0 = r0;
        D = DN;
        __syncthreads();                                     // B3
    }
#pragma unroll
    for (int j = 0; j < VPL; j++) atomicMax(&sMs[o0 + j], (unsigned long long)ms[j]);
    __syncthreads();
    if (tid < VS && v0 + tid < a.V) a.makespan[v0 + tid] = (int64_t)sMs[tid];
}

__global__ __launch_bounds__(256) void k_round_count(int64_t nsteps, const int32_t *__restrict__ step_ptr,
                                                     int32_t rp, int64_t *__restrict__ cnt) {
    const int64_t r = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (r < nsteps) cnt[r] = (step_ptr[r + 1] - step_ptr[r] + rp - 1) / rp;
}

__global__ __launch_bounds__(256) void k_round_fill(int64_t nsteps, const int32_t *__restrict__ step_ptr,
                                                    const int64_t *__restrict__ off, int32_t rp,
                                                    int32_t *__restrict__ r0, int32_t *__restrict__ rn) {
    const int64_t r = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (r >= nsteps) return;
    const int32_t p0 = step_ptr[r], p1 = step_ptr[r + 1];
    int64_t k = off[r];
    for (int32_t q = p0; q < p1; q += rp, k++) {
        r0[k] = q;
        rn[k] = (p1 - q) < rp ? (p1 - q) : rp;
    }
}

template <int LPS, int VPL, int K>
hipError_t launch_pipe(const dd_graph *g, const dd_sched *sch, const dd_variants *var,
                       int64_t *finish, int64_t *start, int64_t *makespan, hipStream_t s) {
    (void)g;
    constexpr int VS = LPS * VPL;
    constexpr int RP = (kNT / LPS) * K;
    const int64_t ns = sch->n_steps;
    const int64_t max_rounds = ns + (sch->n + RP - 1) / RP + 1;
    int64_t *cnt = nullptr, *dummy = nullptr;
    int32_t *r0 = nullptr, *rn = nullptr;
    hipError_t e = dalloc_n(&cnt, (size_t)ns + 2, s);
    if (e == hipSuccess) e = dalloc_n(&r0, (size_t)max_rounds, s);
    if (e == hipSuccess) e = dalloc_n(&rn, (size_t)max_rounds, s);
    if (e == hipSuccess) e = dalloc_n(&dummy, 2 * kNT, s);
    if (e != hipSuccess) { dfree(cnt, s); dfree(r0, s); dfree(rn, s); dfree(dummy, s); return e; }
    if (ns > 0) k_round_count<<<grid_for(ns, 256), 256, 0, s>>>(ns, sch->step_ptr, RP, cnt);
    e = scan_exclusive(cnt, cnt, ns, s);
    if (e == hipSuccess && ns > 0)
        k_round_fill<<<grid_for(ns, 256), 256, 0, s>>>(ns, sch->step_ptr, cnt, RP, r0, rn);
    PipeArgs args{sch->gat_src, sch->gat_spos, sch->gat_cls, sch->gat_gap, var->table,
                  var->n_cls, var->rm_bits, var->edge_on, var->V, var->W, finish, start,
                  makespan, dummy};
    const int grid = (var->V + VS - 1) / VS;
    const int64_t *nrp = cnt + ns;
    const bool tl = (int64_t)var->n_cls * VS <= kTabLds;
    if (e == hipSuccess) {
        if (tl && start)
            k_sim_pipe<LPS, VPL, K, true, true><<<grid, kNT, 0, s>>>(r0, rn, nrp, sch->rec, args);
        else if (tl)
            k_sim_pipe<LPS, VPL, K, true, false><<<grid, kNT, 0, s>>>(r0, rn, nrp, sch->rec, args);
        else if (start)
            k_sim_pipe<LPS, VPL, K, false, true><<<grid, kNT, 0, s>>>(r0, rn, nrp, sch->rec, args);
        else
            k_sim_pipe<LPS, VPL, K, false, false><<<grid, kNT, 0, s>>>(r0, rn, nrp, sch->rec, args);
        e = hipGetLastError();
    }
    dfree(cnt, s); dfree(r0, s); dfree(rn, s); dfree(dummy, s);
    return e;
}

template <int VS>
void launch_vs(const SimArgs &args, int V, hipStream_t s) {
    const int grid = (V + VS - 1) / VS;
    k_simulate<VS, 8><<<grid, kNT, 0, s>>>(args);
}

}  // namespace

hipError_t launch_simulate(const dd_graph *g, const dd_sched *sch, const dd_variants *var,
                           int64_t *finish, int64_t *start, int64_t *makespan, int vs_hint,
                           hipStream_t s) {
    SimArgs args{sch->n_steps, sch->step_ptr, sch->pos_node, sch->pos_flags, sch->pos_dur,
                 sch->pos_gap, sch->pos_cls, sch->gat_ptr, sch->gat_src, sch->gat_pos,
                 sch->gat_cls, sch->gat_gap, var->table, var->rm_bits, var->edge_on,
                 var->V, var->W, finish, start, makespan};
    (void)g;
    int vs = vs_hint;
    if (vs <= 0) {
        // enough workgroups to cover the 256 compute units, then widest rows
        vs = 1;
        while (vs < 16 && (int64_t)var->V / (vs * 2) >= 256) vs *= 2;
    }
    const char *kv = getenv("DD_KERNEL");
    if (!(kv && kv[0] == '1')) {
        // <lanes per slot, variants per lane, positions per slot>: a round
        // holds at most 512 positions (LDS record ring); two variants per
        // lane when V is even (16 B loads and stores stay inside a row)
        const bool pair = (var->V % 2) == 0 && !(kv && kv[0] == '3');
        switch (vs) {
            case 1: return launch_pipe<1, 1, 1>(g, sch, var, finish, start, makespan, s);
            case 2: return pair ? launch_pipe<1, 2, 1>(g, sch, var, finish, start, makespan, s)
                                : launch_pipe<2, 1, 2>(g, sch, var, finish, start, makespan, s);
            case 4: return pair ? launch_pipe<2, 2, 2>(g, sch, var, finish, start, makespan, s)
                                : launch_pipe<4, 1, 4>(g, sch, var, finish, start, makespan, s);
            case 8: return pair ? launch_pipe<4, 2, 4>(g, sch, var, finish, start, makespan, s)
                                : launch_pipe<8, 1, 8>(g, sch, var, finish, start, makespan, s);
            default: return pair ? launch_pipe<8, 2, 4>(g, sch, var, finish, start, makespan, s)
                                 : launch_pipe<16, 1, 8>(g, sch, var, finish, start, makespan, s);
        }
    }
    switch (vs) {
        case 1: launch_vs<1>(args, var->V, s); break;
        case 2: launch_vs<2>(args, var->V, s); break;
        case 4: launch_vs<4>(args, var->V, s); break;
        case 8: launch_vs<8>(args, var->V, s); break;
        default: launch_vs<16>(args, var->V, s); break;
    }
    return hipGetLastError();
}

}  // namespace dd
