// Batched simulation: every variant of the transformed graph at once (the
// hot path).
//
// What is computed (Sec. 3.1, Algorithm 1, with the transformations of
// Sec. 3.4 applied per variant): for each task u in topological order and
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
