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
// step by step (a phase holds at most one run of consecutive tasks per
// thread), in rounds of at most 512 positions.  Inside a run, releases
// follow a max-plus recurrence
//     R_i = max(R_{i-1}, X_i) + w_i      (X_i = max over cross parents)
// whose steps compose associatively:  c -> max(c + A, B).  Per round:
//   walk      each slot folds its K positions into registers (cross-parent
//             releases come from HBM when the parent finished two or more
//             rounds ago, else from the LDS copy of the last round);
//   scan      the (A, B) slot summaries are scanned per variant, with DPP
//             moves inside a wave and a chunk pass across waves;
//   finalize  each lane applies its carry-in, stores finish (and start),
//             and keeps the round's releases in LDS for the next round.
// The records of round k+2 and the HBM loads of round k+1 are issued while
// round k computes.  For graphs with at most kMaxCarryThreads threads the
// release of each thread's latest task sits in LDS, so a run's first task
// reads its thread predecessor there instead of gathering it.

#include "dd_common.h"
#include "dd_internal.h"

#include <stdlib.h>

#include <mutex>
#include <type_traits>

namespace dd {
namespace {

constexpr int kNT = 512;   // threads per workgroup (8 waves)

__device__ __forceinline__ int64_t scaled(int64_t d, const ScaleEntry &se) {
    const uint64_t a = (uint64_t)d * (uint64_t)se.p;
    const uint64_t hi = __umul64hi(a, se.magic) >> se.shift;
    const uint64_t lo = a >> se.shift;
    return (int64_t)(se.magic ? hi : lo);
}

__device__ __forceinline__ int64_t max64(int64_t a, int64_t b) { return a > b ? a : b; }

// 64-bit value from its two 32-bit halves, as one register pair (left
// visible as shift-or, the compiler adds the halves to a sum one at a time)
__device__ __forceinline__ int64_t join64(int lo, int hi) {
    int64_t r = (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
    asm("" : "+v"(r));
    return r;
}

struct PipeArgs {
    const int64_t *gat_ptr;       // [n+1] gathers of each position
    const int32_t *gat_src;       // gathers beyond two per position
    const int32_t *gat_spos;
    const uint8_t *gat_cls;
    const int64_t *gat_gap;
    const int64_t *gap;           // [n] gap of every task (second inline gather)
    const ScaleEntry *table;      // [n_cls][V]
    int32_t n_cls;
    const uint32_t *rm;           // [n][W]
    const void *rmp;              // [workgroups][rmp_stride] removal bits of the workgroup's
                                  // variants per schedule position (u8 for VS <= 8, else u16)
    int64_t rmp_stride;           // positions rounded up to 16 bytes of row
    const uint64_t *edge_on;      // [V]
    uint64_t cls_mask;            // edge classes present in the schedule's gathers
    int32_t thread_carry;         // previous task of a run comes from LDS carries
    int32_t V, W;
    int64_t *finish, *start, *makespan;
    int64_t *dummy;               // [2 * threads] target of stores from idle lanes
};

constexpr int kTabLds = 4096;     // scale entries kept in LDS at most (8 B each)
constexpr size_t kLdsBytes = 160 * 1024;   // LDS of one compute unit (gfx950)
constexpr int kSmall = 64;        // rounds of at most this many positions: one wave per variant
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

// per-lane values indexed by variant: vector types stay in registers where
// a conditional read of an array element could turn into a pointer select
template <int N> struct I64V { typedef long long T __attribute__((ext_vector_type(N))); };
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Loads prefetched a round ahead: for the first gather when its source
// finished two or more rounds earlier, the source's finish, removal word and
// gap.  (The task's own removal bits come with the records.)  A second gather (rare: a task waiting on
// two other threads) loads its old source when the round needs it.
template <int K, int VPL>
struct Dyn {
    Vals<VPL> f0[K];              // finish of the first gather's source
    uint32_t r0w[K];              // removal word of that source
    int64_t g0gap[K];             // gap of that source
};

__device__ __forceinline__ bool cls_on(uint64_t eon, uint8_t c) {
    return c == 255 || ((eon >> c) & 1ull);
}

// LDS scale entry: p (bits 0..31), shift (32..39), bit 40 = multiply-high
// needed (q not a power of two; the 64-bit magic is then read from the table)
__device__ __forceinline__ int64_t scaled8(int64_t d, uint64_t e, const ScaleEntry *tab,
                                           int64_t idx) {
    const uint64_t a = (uint64_t)d * (uint32_t)e;
    const uint32_t sh = (uint32_t)(e >> 32) & 0xff;
    if (e & (1ull << 40)) return (int64_t)(__umul64hi(a, tab[idx].magic) >> sh);
    return (int64_t)(a >> sh);
}

// Run heads without flags.  A range of positions maps the release entering
// it to c -> max(c + a, b), with b >= a.  A range that holds the first task of
// a run ignores c; it is written with a = kHead + (its weights after the
// head), so c + a < 0 <= b for every c that occurs: every simulated time is
// below 2^62 (the graph and transform checks reject anything larger), and c
// plus the weights of later positions is itself such a time.  Composing keeps
// a >= kHead, so no sum overflows.
constexpr int64_t kHead = -(int64_t(1) << 62);

// Time arithmetic.  Tm<false>: plain int64.  Tm<true>: every value is an
// integer held in a double, which the hardware adds and compares in one
// full-rate instruction each (int64 takes two to three).  Times are biased
// by 2^52: the double of time t (0 <= t < 2^52) has the bit pattern
// 0x4330000000000000 + t, so moving a time between HBM (int64) and a
// register is one operation on its high word, and the bit patterns of
// nonnegative doubles order as integers do.  Weights (durations, gaps and
// their sums) stay unbiased, and a range holding a run head carries -inf,
// which any sum keeps (c + -inf = -inf loses to every b in a max).  All of
// it is exact while every simulated time stays below 2^51 and every
// duration times the scale numerator below 2^53 (checked on the host; the
// int64 form serves every other launch).  Values travel as int64 bit
// patterns either way.
template <bool FP> struct Tm;
template <> struct Tm<false> {
    static constexpr int64_t zero = 0;          // time 0
    static constexpr int64_t head = kHead;      // weight sum of a range holding a run head
    __device__ static __forceinline__ int64_t add(int64_t x, int64_t y) { return x + y; }
    __device__ static __forceinline__ int64_t sub(int64_t x, int64_t y) { return x - y; }
    __device__ static __forceinline__ int64_t mx(int64_t x, int64_t y) { return max64(x, y); }
    __device__ static __forceinline__ int64_t from_time(int64_t t) { return t; }
    __device__ static __forceinline__ int64_t to_time(int64_t x) { return x; }
    __device__ static __forceinline__ int64_t w32(uint32_t w) { return (int64_t)w; }
    __device__ static __forceinline__ double d(int64_t x) { return __longlong_as_double(x); }
    __device__ static __forceinline__ int64_t i(double x) { return __double_as_longlong(x); }
};
template <> struct Tm<true> {
    static constexpr int64_t zero = 0x4330000000000000ll;                    // 2^52
    static constexpr int64_t head = (int64_t)0xFFF0000000000000ull;          // -inf
    __device__ static __forceinline__ double d(int64_t x) { return __longlong_as_double(x); }
    __device__ static __forceinline__ int64_t i(double x) { return __double_as_longlong(x); }
    __device__ static __forceinline__ int64_t add(int64_t x, int64_t y) { return i(d(x) + d(y)); }
    __device__ static __forceinline__ int64_t sub(int64_t x, int64_t y) { return i(d(x) - d(y)); }
    __device__ static __forceinline__ int64_t mx(int64_t x, int64_t y) {
        return i(__builtin_fmax(d(x), d(y)));
    }
    __device__ static __forceinline__ int64_t from_time(int64_t t) { return t | zero; }
    __device__ static __forceinline__ int64_t to_time(int64_t x) { return x ^ zero; }
    __device__ static __forceinline__ int64_t w32(uint32_t w) { return i((double)w); }
};

// (la, lb) then (a, b)
template <bool FP = false>
__device__ __forceinline__ void compose(int64_t la, int64_t lb, int64_t &a, int64_t &b) {
    b = Tm<FP>::mx(Tm<FP>::add(lb, a), b);
    if (FP) a = Tm<FP>::add(la, a);
    else a = a < 0 ? a : la + a;
}

// one Kogge-Stone step of the max-plus scan across the wave, the left
// operand taken with a DPP lane shift (lanes without one see the identity
// (0, 0), as b >= a; in the double form the bits 0 are 0.0, below every
// biased time).  Row shifts write every lane (bound control: 0 where the
// source lies outside the row), so no lane needs its old value.
template <int CTRL, int RMASK, bool FP = false>
__device__ __forceinline__ void scan_step(int64_t &a, int64_t &b) {
    constexpr bool BC = RMASK == 0xf;
    const int alo = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)a, CTRL, RMASK, 0xf, BC);
    const int ahi = __builtin_amdgcn_update_dpp(0, (int)((uint64_t)a >> 32), CTRL, RMASK, 0xf, BC);
    const int blo = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)b, CTRL, RMASK, 0xf, BC);
    const int bhi = __builtin_amdgcn_update_dpp(0, (int)((uint64_t)b >> 32), CTRL, RMASK, 0xf, BC);
    const int64_t la = join64(alo, ahi);
    const int64_t lb = join64(blo, bhi);
    compose<FP>(la, lb, a, b);
}

__device__ __forceinline__ int64_t readlane64(int64_t x, int l) {
    const int lo = __builtin_amdgcn_readlane((int)(uint32_t)x, l);
    const int hi = __builtin_amdgcn_readlane((int)((uint64_t)x >> 32), l);
    return join64(lo, hi);
}

// inclusive scan over the 64 lanes of a wave
template <bool FP = false>
__device__ __forceinline__ void wave_scan(int64_t &a, int64_t &b) {
    scan_step<0x111, 0xf, FP>(a, b);   // row_shr:1
    scan_step<0x112, 0xf, FP>(a, b);   // row_shr:2
    scan_step<0x114, 0xf, FP>(a, b);   // row_shr:4
    scan_step<0x118, 0xf, FP>(a, b);   // row_shr:8
    scan_step<0x142, 0xa, FP>(a, b);   // row_bcast:15 into rows 1 and 3
    scan_step<0x143, 0xc, FP>(a, b);   // row_bcast:31 into rows 2 and 3
}

// Lane layout: slot = tid / LPS handles K consecutive positions; the LPS
// lanes of a slot each own VPL consecutive variants (VS = LPS * VPL per
// workgroup), so one 8*VPL-byte load or store serves every variant of the
// lane and the per-position bookkeeping is paid once per VPL variants.
// Idle lanes keep issuing the same prefetch loads (clamped addresses) and
// stores (to a dummy target), so within each kind of round the count of
// memory operations in flight is the same on every path and the wait for
// the next round's data never includes this round's stores.  Waves whose
// slots all lie past the end of a round skip the arithmetic (rounds at the
// end of a phase are ragged).
//
// UNI: every variant of the launch enables every edge class that the
// schedule's gathers use, every scale is a power of two, every duration
// and gap is below 2^32 (a gather source's gap comes from the record) and
// the launch passes the bounds of the double form of the time arithmetic
// (Tm<true>): the scaled duration is the floor of the duration times the
// scale held as a double, and every sum and maximum of the walk, the scans
// and the finalize is one double instruction.
template <int LPS, int VPL, int K, bool TLDS, bool START, bool UNI, int NT>
__global__ __launch_bounds__(NT) void k_sim_pipe(const int32_t *__restrict__ round_r0,
                                                  const int32_t *__restrict__ round_rn,
                                                  const int64_t *__restrict__ n_rounds,
                                                  const Rec *__restrict__ rec, PipeArgs a) {
    constexpr int VS = LPS * VPL;
    constexpr int NS = NT / LPS;
    constexpr int RP = NS * K;
    typedef Tm<UNI> TM;
    // a gap read from memory as a weight (below 2^32 on the uniform path)
    auto wt = [](int64_t g) -> int64_t {
        if constexpr (UNI) return TM::w32((uint32_t)g);
        else return g;
    };
    // slot summaries, variant-major with a row stride of NSP: when a wave
    // scans whole variants, 4 entries of padding put the rows written by
    // one wave on different banks
    constexpr int NSP = NS == 64 * VPL ? NS + 4 : NS;
    constexpr int NE = NSP * VS;
    constexpr int RW = RP * 3;            // 16-byte words of one ring buffer
    constexpr int PF = (RW + NT - 1) / NT;
    static_assert(sizeof(Rec) == 48, "record layout");
    static_assert(RP <= NT, "positions per round");
    static_assert(PF <= 3, "record prefetch words per lane");
    constexpr int NCH = NE / 64 > 0 ? NE / 64 : 1;   // 64-entry chunks of summaries
    static_assert(!UNI || TLDS, "uniform path keeps the table in LDS");
    // small rounds (at most 64 positions): wave w alone handles variants
    // w, w + NW, ... for every position of the round (one per lane), so the
    // round needs no slot scan across waves and only the ring barrier
    constexpr int NW = NT / 64;           // waves per workgroup
    constexpr int PS = (VS + NW - 1) / NW;  // variants per wave in a small round
    static_assert(PS <= K && PS <= 2, "load slots for small rounds");
    // records of rounds k, k+1 (read) and k+2 (being filled): a ring of three;
    // beside them the removal bits of the workgroup's variants per position
    typedef typename std::conditional<(VS <= 8), uint8_t, uint16_t>::type RmT;
    static_assert(VS <= 16, "removal bits per position");
    __shared__ uint4 sRec[3][RW];
    __shared__ RmT sRm[3][RP];
    __shared__ int64_t sR[RP * VS];
    __shared__ int64_t sA[NE], sB[NE];
    __shared__ int64_t sTA[NCH], sTB[NCH];
    extern __shared__ uint64_t sT[];      // scale table (n_cls x VS), sized at launch
    __shared__ int64_t sTC[kMaxCarryThreads * VS];
    __shared__ unsigned long long sMs[VS];
    __shared__ int64_t sCarry[VS];        // release at the end of a big round
    __shared__ uint64_t sEon[VS];
    __shared__ int sFlags;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wv = tid >> 6;
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
    const bool lok = vf < a.V;                // V is a multiple of VPL: vf + VPL - 1 < V too
    const int vvf = lok ? vf : 0;
    const uint32_t vsh = (uint32_t)(vvf & 31);
    const int vw = vvf >> 5;
    const int64_t V = a.V, W = a.W;
    const uint32_t nr = (uint32_t)*n_rounds;   // rounds < 2^32 (at most tasks + tasks / RP + 1)
    const int o0 = lis * VPL;                 // variant offset inside the workgroup
    // stores that must not land go to one 16-byte spot per wave (one line)
    gi64 *const dummy = (gi64 *)(a.dummy + (tid >> 6) * 2);
    const bool tcar = a.thread_carry != 0;
    const RmT *const rmrow = reinterpret_cast<const RmT *>(a.rmp) + (int64_t)wg * a.rmp_stride;

    if (tid == 0) sFlags = 0;
    {   // the record ring starts zeroed (no stale fields past a round's end)
        uint4 *z = &sRec[0][0];
        for (int i = tid; i < 3 * RW; i += NT) z[i] = make_uint4(0u, 0u, 0u, 0u);
    }
    __syncthreads();
    bool any_magic = false;
    if (TLDS) {
        for (int i = tid; i < a.n_cls * VS; i += NT) {
            const int c = i / VS, o = i % VS;
            const int vx = v0 + o < a.V ? v0 + o : 0;
            const ScaleEntry e = a.table[(int64_t)c * V + vx];
            const bool mg = e.magic != 0;
            any_magic |= mg;
            if (UNI)   // the scale p / 2^shift as a double (exact: p < 2^32)
                sT[i] = (uint64_t)__double_as_longlong(__builtin_ldexp((double)e.p, -(int)(e.shift & 0xff)));
            else
                sT[i] = (uint64_t)e.p | ((uint64_t)(e.shift & 0xff) << 32) | (mg ? (1ull << 40) : 0ull);
        }
    }
    for (int i = tid; i < kMaxCarryThreads * VS; i += NT) sTC[i] = TM::zero;
    if (tid < VS) {
        sMs[tid] = 0;
        sCarry[tid] = TM::zero;   // read by a first round that is small (finite, so heads ignore it)
        // per-variant values read inside the loop live in LDS: a register
        // loaded before the loop would make every round wait for all traffic
        sEon[tid] = a.edge_on[v0 + tid < a.V ? v0 + tid : 0];
    }
    if (any_magic) atomicOr(&sFlags, 1);
    for (uint32_t rr = 0; rr < 2; rr++) {     // prologue: records of rounds 0 and 1
        if (rr < nr) {
            const int r0 = round_r0[rr], rn = round_rn[rr];
            const uint4 *src = reinterpret_cast<const uint4 *>(rec + r0);
            for (int i = tid; i < rn * 3; i += NT) sRec[rr][i] = src[i];
            for (int i = tid; i < rn; i += NT) sRm[rr][i] = rmrow[r0 + i];
        }
    }
    __syncthreads();
    // uniform fast paths: every edge class of the schedule on in all of the
    // workgroup's variants; every scale a power of two (shift only)
    uint64_t eall = ~0ull;
#pragma unroll
    for (int o = 0; o < VS; o++) eall &= sEon[o];
    const bool all_on = UNI || (eall & a.cls_mask) == a.cls_mask;
    const bool shift_only = UNI || (TLDS && !(sFlags & 1));

    // positions per slot in a round of rn positions: small rounds spread
    // over all waves, one position per slot, instead of filling the first
    // wave with K positions per slot
    auto per_slot = [&](int rn) { return rn <= NS ? 1 : (rn + NS - 1) / NS; };

    // loads of a round of rn positions (records in ring buffer b); a gather
    // is old when its source position precedes prev_r0 (its round has ended
    // before the round that issues these loads)
    // (the layout is a compile-time choice: with a run-time branch between the
    // two layouts, the compiler would make each wait for the other's loads)
    // word k of the record of position q in ring buffer b: the address is
    // formed in 32 bits, and the masks (q < RP, b < 3) let the compiler use
    // full-rate 24-bit multiplies; as pointer arithmetic it became a
    // quarter-rate 64-bit multiply-add
    typedef __attribute__((address_space(3))) const u32x4 lds_u4;
    lds_u4 *const ring = (lds_u4 *)&sRec[0][0];
    auto rec_w = [&](int b, int q, int k) -> int4 {
        const uint32_t idx = ((uint32_t)b & 3u) * (uint32_t)RW + ((uint32_t)q & 0xffffu) * 3u + (uint32_t)k;
        const u32x4 u = ring[idx];
        return make_int4((int)u.x, (int)u.y, (int)u.z, (int)u.w);
    };
    // offset of row `row` (nonnegative, 32 bits) of a row-major array
    // `width` wide: one 32x32 -> 64 multiply
    auto rowoff = [](int64_t row, int64_t width) -> int64_t {
        return (int64_t)((uint64_t)(uint32_t)row * (uint64_t)(uint32_t)width);
    };
    auto issue = [&](auto small_tag, int rn, int b, int prev_r0, Dyn<K, VPL> &d) {
        constexpr bool SMALL_LAYOUT = decltype(small_tag)::value;
        const int ke = per_slot(rn);
        if constexpr (SMALL_LAYOUT) {
            // small layout: position = lane; slot jj of the load registers
            // holds variant w + 8 jj of this wave
            const int q = lane;
            const bool ok = q < rn;
            const int4 w1 = rec_w(b, q, 1);
            const bool n0 = ok & (w1.y >= 0) & (w1.w < prev_r0);
            const int64_t a0 = n0 ? w1.y : 0;
#pragma unroll
            for (int jj = 0; jj < K; jj++) {
                const int os = wv + NW * jj;
                const bool vv = jj < PS && os < VS && v0 + os < a.V;
                const int64_t vs_ = vv ? v0 + os : 0;
                const int64_t vwj = vs_ >> 5;
                // every field is written on every path: stores that differ
                // between paths get merged through a selected address, which
                // would keep the whole struct in scratch
                Vals<VPL> f{};
                uint32_t r0 = 0;
                int64_t gg = 0;
                if (jj < PS) {
                    // issued on every path (row 0 when unused): with a known
                    // count of loads, the ring refill waits for the record
                    // loads only
                    f.x[0] = a.finish[rowoff(a0, V) + vs_];
                    r0 = a.rm[rowoff(a0, W) + vwj];
                    if (!UNI) gg = a.gap[a0];
                }
                d.f0[jj] = f;
                d.r0w[jj] = r0;
                d.g0gap[jj] = gg;
            }
        } else {
#pragma unroll
            for (int i = 0; i < K; i++) {
                const int q = slot * ke + i;
                const bool ok = i < ke && q < rn;
                const int4 w1 = rec_w(b, q, 1);   // node, g0_src, g1_src, g0_spos
                const bool n0 = ok & (w1.y >= 0) & (w1.w < prev_r0);
                const int64_t a0 = n0 ? w1.y : 0;
                // issued on every path (row 0 when unused), like the small layout
                const Vals<VPL> f = *reinterpret_cast<const Vals<VPL> *>(a.finish + rowoff(a0, V) + vvf);
                const uint32_t r0 = a.rm[rowoff(a0, W) + vw];
                const int64_t gg = UNI ? 0 : a.gap[a0];
                d.f0[i] = f;
                d.r0w[i] = r0;
                d.g0gap[i] = gg;
            }
        }
    };
    // one position of the big layout (issue() does all K of them)
    // (qs = slot * positions per slot of that round)
    auto issue_big_at = [&](int rn, int ke, int qs, int b, int prev_r0, Dyn<K, VPL> &d, int i) {
        const int q = qs + i;
        const bool ok = i < ke && q < rn;
        const int4 w1 = rec_w(b, q, 1);
        const bool n0 = ok & (w1.y >= 0) & (w1.w < prev_r0);
        const int64_t a0 = n0 ? w1.y : 0;
        const Vals<VPL> f = *reinterpret_cast<const Vals<VPL> *>(a.finish + rowoff(a0, V) + vvf);
        const uint32_t r0 = a.rm[rowoff(a0, W) + vw];
        const int64_t gg = UNI ? 0 : a.gap[a0];
        d.f0[i] = f;
        d.r0w[i] = r0;
        d.g0gap[i] = gg;
    };
    // (start, size) of rounds k .. k+3, the last clamped to the final round:
    // each round loads the entry three rounds ahead, so no round waits for
    // a scalar load of its own bounds
    auto rmeta = [&](uint32_t i, int &r0_, int &rn_) {
        const uint32_t c = i < nr ? i : nr - 1;
        r0_ = round_r0[c];
        rn_ = round_rn[c];
    };
    int m0r0 = 0, m0rn = 0, m1r0 = 0, m1rn = 0, m2r0 = 0, m2rn = 0, m3r0 = 0, m3rn = 0;
    if (nr > 0) {
        rmeta(0, m0r0, m0rn);
        rmeta(1, m1r0, m1rn);
        rmeta(2, m2r0, m2rn);
        rmeta(3, m3r0, m3rn);
    }
    Dyn<K, VPL> D;
    if (nr > 0) {
        if (m0rn <= kSmall) issue(std::true_type{}, m0rn, 0, 0, D);
        else issue(std::false_type{}, m0rn, 0, 0, D);
    }
    // Consume the first round's loads here: the loop's registers then hold
    // no load in flight on entry, and the wait-count bookkeeping does not
    // make every round's walk wait for part of the next round's loads.
#pragma unroll
    for (int i = 0; i < K; i++) {
        asm volatile("" ::"v"(D.r0w[i]));
        if (!UNI) asm volatile("" ::"v"(D.g0gap[i]));
#pragma unroll
        for (int j = 0; j < VPL; j++) asm volatile("" ::"v"(D.f0[i].x[j]));
    }

    typename I64V<VPL>::T carry = TM::zero, ms = TM::zero;
    int64_t msS0 = TM::zero, msS1 = TM::zero;   // small rounds: variants w and w + NW
    int prev_r0 = 0;
    int b0 = 0, b1 = 1, b2 = 2;               // ring buffers of rounds k, k+1, k+2
    // Small and big rounds run as two inner loops rather than one loop with
    // an if/else: the compiler then sees no path through an iteration that
    // skips both bodies, so it never makes a round wait for loads of the
    // previous round, or for its stores, that were in fact consumed already.
    uint32_t k = 0;
    auto round = [&](auto small_tag, auto next_small_tag) {
        constexpr bool SMALL_ROUND = decltype(small_tag)::value;
        const int r0 = m0r0, rn = m0rn;
        int m4r0, m4rn;                           // round k+4, used from the next round on
        if (nr > 0) rmeta(k + 4, m4r0, m4rn);
        uint64_t eon[VPL];
#pragma unroll
        for (int j = 0; j < VPL; j++) eon[j] = sEon[o0 + j];
        // next round's loads (records of k+1 are in LDS since round k-1): a
        // small round issues them first; a big round during or right after
        // its walk (a big next round's loads for position i go out after the
        // walk's position i, whose prefetched registers they then reuse), so
        // their record reads and address work fill the walk's stalls and the
        // wait at the round's first barrier
        Dyn<K, VPL> DN;
        const int rn1 = m1rn;                     // round k+1 (this round if last)
        const int bN = k + 1 < nr ? b1 : b0;
        // records of round k+2: global -> registers, -> LDS before the stores
        const int nxt_w = k + 2 < nr ? m2rn * 3 : 0;
        const u32x4 *nsrc = reinterpret_cast<const u32x4 *>(rec + m2r0);
        u32x4 nx0, nx1, nx2;
        RmT nrm;
        auto load_next = [&]() {
            nx0 = nsrc[tid < nxt_w ? tid : 0];
            nrm = rmrow[m2r0 + (tid < nxt_w / 3 ? tid : 0)];
            if (PF > 1) nx1 = nsrc[tid + NT < nxt_w ? tid + NT : 0];
            if (PF > 2) nx2 = nsrc[tid + 2 * NT < nxt_w ? tid + 2 * NT : 0];
        };
        // Round k+2 goes into the buffer that round k-1 used (every wave
        // finished reading it before the previous round's last barrier).  It
        // is written before this round's result stores: vector memory
        // operations complete in order, so a later write would also wait for
        // the stores to land.
        auto put_next = [&]() {
            // the loads land here on every path (a lane that skips its write
            // would otherwise leave them pending into the next round)
            asm volatile("" ::"v"(nx0), "v"((uint32_t)nrm));
            if (PF > 1) asm volatile("" ::"v"(nx1));
            if (PF > 2) asm volatile("" ::"v"(nx2));
            u32x4 *dst = reinterpret_cast<u32x4 *>(sRec[b2]);
            if (tid < nxt_w) dst[tid] = nx0;
            if (tid < nxt_w / 3) sRm[b2][tid] = nrm;
            if (PF > 1 && tid + NT < nxt_w) dst[tid + NT] = nx1;
            if (PF > 2 && tid + 2 * NT < nxt_w) dst[tid + 2 * NT] = nx2;
        };

        if constexpr (SMALL_ROUND) {
            // ---- small round: one position per lane, variants per wave ----
            load_next();
            Dyn<K, VPL> DNs;
            issue(next_small_tag, rn1, bN, r0, DNs);
            const int q = lane;
            const bool ok = q < rn;
            const int4 w0 = rec_w(b0, q, 0), w1 = rec_w(b0, q, 1), w2 = rec_w(b0, q, 2);
            const int64_t dur = ((int64_t)(uint32_t)w0.y << 32) | (uint32_t)w0.x;
            const int64_t gap = UNI ? TM::w32((uint32_t)w0.z)
                                    : (((int64_t)(uint32_t)w0.w << 32) | (uint32_t)w0.z);
            const int32_t node = w1.x, s0 = w1.y, s1 = w1.z, p0 = w1.w, p1 = w2.x;
            const uint32_t cl = (uint32_t)w2.y;
            const int cls = ok ? (int)(cl & 0xffff) : 0;
            const uint8_t c0 = (cl >> 16) & 0xff, c1 = cl >> 24;
            const uint32_t flags = ok ? (uint32_t)w2.z : 0u;
            uint32_t rbq = sRm[b0][q];            // read on every lane: a select, not a masked read
            asm volatile("" : "+v"(rbq));
            const uint32_t rb = ok ? rbq : 0u;    // removal bits of the task
            const bool head = flags & 1u;
            const bool old0 = p0 < prev_r0, old1 = p1 < prev_r0;
            int i0 = p0 - prev_r0, i1 = p1 - prev_r0;
            i0 = i0 < 0 ? 0 : (i0 >= RP ? RP - 1 : i0);
            i1 = i1 < 0 ? 0 : (i1 >= RP ? RP - 1 : i1);
            const bool has0 = ok && s0 >= 0;
            const bool has1 = ok && s1 >= 0;
            const bool any1 = __any(has1);
            const uint32_t extra = flags >> 8;
            const int tcx = ((flags >> 2) & 63u) * VS;
            const int64_t g0w = UNI ? TM::w32((uint32_t)w2.w) : 0;   // first source's gap
            int64_t Fs[K], Ss[K];
            bool sts[K];
#pragma unroll
            for (int jj = 0; jj < K; jj++) {
                const int os = wv + NW * jj;
                const bool vw_ok = jj < PS && os < VS && v0 + os < a.V;   // wave-uniform
                const int64_t vs_ = vw_ok ? v0 + os : 0;
                int64_t F = 0, S = 0;
                bool st = false;
                if (vw_ok) {
                    const uint32_t bit = (uint32_t)(vs_ & 31);
                    const int64_t vwj = vs_ >> 5;
                    const uint64_t eo = sEon[os];
                    const bool rmv = (rb >> os) & 1u;
                    // the LDS reads that depend on the record, issued together
                    int64_t yn = sR[i0 * VS + os];
                    int64_t tcv = sTC[tcx + os];
                    uint64_t tev = TLDS ? sT[cls * VS + os] : 0ull;
                    int64_t crv = sCarry[os];
                    asm volatile("" : "+v"(yn), "+v"(tcv), "+v"(tev), "+v"(crv));
                    int64_t X;
                    {
                        const int64_t g0g = UNI ? g0w : D.g0gap[jj];
                        const int64_t ro = TM::add(TM::from_time(D.f0[jj].x[0]),
                                                   ((D.r0w[jj] >> bit) & 1u) ? 0 : g0g);
                        const int64_t rel = old0 ? ro : yn;
                        const bool on = has0 && (all_on || cls_on(eo, c0));
                        X = on ? rel : TM::zero;
                    }
                    if (any1) {
                        int64_t ro = 0;
                        if (__any(has1 && old1)) {       // rare: loaded on demand
                            const int64_t a1 = has1 && old1 ? s1 : 0;
                            const bool r1 = (a.rm[a1 * W + vwj] >> bit) & 1u;
                            ro = TM::add(TM::from_time(a.finish[a1 * V + vs_]), r1 ? 0 : wt(a.gap[a1]));
                        }
                        const int64_t rel = old1 ? ro : sR[i1 * VS + os];
                        const bool on = has1 && (all_on || cls_on(eo, c1));
                        X = on ? TM::mx(X, rel) : X;
                    }
                    if (tcar) X = head ? TM::mx(X, tcv) : X;
                    if (__any(extra != 0u)) {
                        // rare: wide fan-in.  The wave's lanes share each such
                        // position's gathers beyond two (64 per pass, loads of
                        // a pass in flight together), then a wave max hands
                        // the result to the position's lane
                        uint64_t todo = __ballot(extra != 0u);
                        while (todo) {
                            const int ld = __ffsll((unsigned long long)todo) - 1;
                            todo &= todo - 1;
                            const int64_t e0 = a.gat_ptr[r0 + ld] + 2, e1 = a.gat_ptr[r0 + ld + 1];
                            int64_t mx = 0;
                            for (int64_t eb = e0; eb < e1; eb += 64) {
                                const int64_t e = eb + lane;
                                if (e < e1) {
                                    const uint8_t c = a.gat_cls[e];
                                    const int32_t sp = a.gat_spos[e];
                                    int64_t rel;
                                    if (sp < prev_r0) {
                                        const int64_t sx = a.gat_src[e];
                                        const bool rs = (a.rm[sx * W + vwj] >> bit) & 1u;
                                        rel = TM::add(TM::from_time(a.finish[sx * V + vs_]),
                                                      rs ? 0 : wt(a.gat_gap[e]));
                                    } else {
                                        rel = sR[(sp - prev_r0) * VS + os];
                                    }
                                    if (cls_on(eo, c)) mx = TM::mx(mx, rel);
                                }
                            }
                            // (bit patterns of nonnegative doubles order as integers)
                            mx = wave_max64(mx);
                            if (lane == ld) X = TM::mx(X, mx);
                        }
                    }
                    int64_t dp;
                    if (UNI) {
                        dp = TM::i(__builtin_floor((double)(uint32_t)dur * TM::d((int64_t)tev)));
                    } else if (TLDS) {
                        const uint64_t te = tev;
                        if (shift_only) {
                            dp = (int64_t)(((uint64_t)dur * (uint32_t)te) >> ((uint32_t)(te >> 32) & 0xff));
                        } else {
                            dp = scaled8(dur, te, a.table, (int64_t)cls * V + vs_);
                        }
                    } else {
                        dp = scaled(dur, a.table[(int64_t)cls * V + vs_]);
                    }
                    const bool live = ok && !rmv;
                    dp = live ? dp : 0;
                    const int64_t gp = live ? gap : 0;
                    // one position per lane: c -> max(c + A, B), a run head
                    // written with the head value; the round's first
                    // position takes the carry (no effect on a head)
                    int64_t sa = ok ? (head ? TM::head : TM::add(dp, gp)) : 0;
                    int64_t sb = ok ? TM::add(TM::add(X, dp), gp) : 0;
                    if (q == 0 && ok) sb = TM::mx(TM::add(crv, sa), sb);
                    wave_scan<UNI>(sa, sb);
                    const int64_t Rv = sb;
                    F = TM::sub(Rv, gp);
                    S = TM::sub(F, dp);
                    if (ok) sR[q * VS + os] = Rv;
                    if (ok && tcar && (flags & 2u)) sTC[tcx + os] = Rv;
                    if (ok && !rmv) {
                        if (jj == 0) msS0 = TM::mx(msS0, F);
                        else msS1 = TM::mx(msS1, F);
                    }
                    st = ok;
                }
                Fs[jj] = F;
                Ss[jj] = S;
                sts[jj] = st;
            }
            put_next();
#pragma unroll
            for (int jj = 0; jj < PS; jj++) {   // the wave's variant slots only
                const int os = wv + NW * jj;
                const bool vw_ok = os < VS && v0 + os < a.V;
                const int64_t vs_ = vw_ok ? v0 + os : 0;
                // formed on every lane (lanes past the round's end store to
                // the dummy), so the choice is a select
                const int64_t off = rowoff(node, V) + vs_;
                gi64 *oa = (gi64 *)(a.finish + off);
                asm volatile("" : "+v"(oa));
                gi64 *o = sts[jj] ? oa : dummy;
                asm volatile("" : "+v"(o));  // one unconditional store per slot
                *o = TM::to_time(Fs[jj]);
                if (START) {
                    gi64 *osa = (gi64 *)(a.start + off);
                    asm volatile("" : "+v"(osa));
                    gi64 *os2 = sts[jj] ? osa : dummy;
                    asm volatile("" : "+v"(os2));
                    *os2 = TM::to_time(Ss[jj]);
                }
            }
            DN = DNs;
        } else {
        // ---- big round: slots of consecutive positions across all waves ----
        load_next();
        const int ke = per_slot(rn);              // positions per slot this round
        const bool wact = __any(slot * ke < rn);  // some position of this wave is live
        // walk: local max-plus recurrence over this slot's K positions
        int64_t Fl[K][VPL], Dp[K][VPL], Dd[K][VPL];
        int32_t U[K];
        int64_t Gp[K][VPL];                       // gap of each kept task (0 if removed)
        uint32_t FLk[K];                          // flags (0 past the round's end)
#pragma unroll
        for (int i = 0; i < K; i++) {
            U[i] = 0;
            FLk[i] = 0;
#pragma unroll
            for (int j = 0; j < VPL; j++) Gp[i][j] = 0;
        }
        int64_t A[VPL], B[VPL];
#pragma unroll
        for (int j = 0; j < VPL; j++) { A[j] = 0; B[j] = 0; }
        // high word added to a position's finish before the makespan max:
        // that of the head value for positions not kept (removed, or past
        // the round's end; its low word is 0)
        constexpr uint32_t kNk = (uint32_t)((uint64_t)TM::head >> 32);
        uint32_t nkh[K][VPL];
#pragma unroll
        for (int i = 0; i < K; i++)
#pragma unroll
            for (int j = 0; j < VPL; j++) nkh[i][j] = kNk;
        Dyn<K, VPL> DNb;
        constexpr bool NEXT_BIG = !decltype(next_small_tag)::value;
        const int ke1 = per_slot(rn1);                      // next round's layout
        const int qs1 = (int)(((uint32_t)slot & 0xffffu) * ((uint32_t)ke1 & 0xffu));
        {
#pragma unroll
            for (int i = 0; i < K; i++) {
                // a big next round's loads go out position by position, between
                // this round's positions
                if (NEXT_BIG && i > 0) issue_big_at(rn1, ke1, qs1, bN, r0, DNb, i - 1);
                if (!wact || i >= ke) continue;
                const int q = slot * ke + i;
                const bool ok = q < rn;
                const int4 w0 = rec_w(b0, q, 0), w1 = rec_w(b0, q, 1), w2 = rec_w(b0, q, 2);
                const int64_t dur = ((int64_t)(uint32_t)w0.y << 32) | (uint32_t)w0.x;
                const int64_t gap = UNI ? TM::w32((uint32_t)w0.z)
                                    : (((int64_t)(uint32_t)w0.w << 32) | (uint32_t)w0.z);
                const int32_t node = w1.x, s0 = w1.y, s1 = w1.z, p0 = w1.w, p1 = w2.x;
                // positions past the round's end hold stale LDS: nothing read
                // from them may form an address
                const uint32_t cl = (uint32_t)w2.y;
                const int cls = ok ? (int)(cl & 0xffff) : 0;
                const uint8_t c0 = (cl >> 16) & 0xff, c1 = cl >> 24;
                const uint32_t flags = ok ? (uint32_t)w2.z : 0u;
                uint32_t rbq = sRm[b0][q];        // read on every lane: a select, not a masked read
                asm volatile("" : "+v"(rbq));
                const uint32_t rb = ok ? rbq : 0u;   // removal bits of the task
                const bool head = flags & 1u;
                U[i] = node;
                FLk[i] = flags;
                const bool old0 = p0 < prev_r0, old1 = p1 < prev_r0;
                int i0 = p0 - prev_r0, i1 = p1 - prev_r0;
                i0 = i0 < 0 ? 0 : (i0 >= RP ? RP - 1 : i0);
                i1 = i1 < 0 ? 0 : (i1 >= RP ? RP - 1 : i1);
                const bool has0 = ok && s0 >= 0;
                const bool has1 = ok && s1 >= 0;
                // wave-uniform skips: chain phases have few gathers and heads
                const bool any0 = __any(has0);
                const bool any1 = __any(has1);
                const bool anyh = __any(head);
                const uint32_t extra = flags >> 8;
                const int tcx = ((flags >> 2) & 63u) * VS + o0;
                // latest release over the parents present in each variant; every
                // wave-uniform decision below is taken once for all VPL variants
                int64_t X[VPL];
#pragma unroll
                for (int j = 0; j < VPL; j++) X[j] = TM::zero;
                if (any0) {
                    Vals<VPL> yn = *reinterpret_cast<const Vals<VPL> *>(&sR[i0 * VS + o0]);
                    // read on every lane: the choice below stays a select
                    // instead of a branch that sinks half of the read
#pragma unroll
                    for (int j = 0; j < VPL; j++) asm volatile("" : "+v"(yn.x[j]));
                    const int64_t g0g = UNI ? TM::w32((uint32_t)w2.w) : D.g0gap[i];
#pragma unroll
                    for (int j = 0; j < VPL; j++) {
                        const int64_t ro = TM::add(TM::from_time(D.f0[i].x[j]),
                                                   ((D.r0w[i] >> (vsh + j)) & 1u) ? 0 : g0g);
                        const int64_t rel = old0 ? ro : yn.x[j];
                        const bool on = has0 && (all_on || cls_on(eon[j], c0));
                        X[j] = on ? rel : TM::zero;
                    }
                }
                if (any1) {
                    Vals<VPL> ro{};
                    if (__any(has1 && old1)) {           // rare: loaded on demand
                        const int64_t a1 = has1 && old1 ? s1 : 0;
                        const uint32_t r1w = a.rm[a1 * W + vw];
                        const int64_t g1 = a.gap[a1];
                        const Vals<VPL> f1 = *reinterpret_cast<const Vals<VPL> *>(a.finish + a1 * V + vvf);
#pragma unroll
                        for (int j = 0; j < VPL; j++)
                            ro.x[j] = TM::add(TM::from_time(f1.x[j]),
                                              ((r1w >> (vsh + j)) & 1u) ? 0 : wt(g1));
                    }
                    const Vals<VPL> yn = *reinterpret_cast<const Vals<VPL> *>(&sR[i1 * VS + o0]);
#pragma unroll
                    for (int j = 0; j < VPL; j++) {
                        const int64_t rel = old1 ? ro.x[j] : yn.x[j];
                        const bool on = has1 && (all_on || cls_on(eon[j], c1));
                        X[j] = on ? TM::mx(X[j], rel) : X[j];
                    }
                }
                if (tcar && anyh) {                            // previous task of the thread
                    const Vals<VPL> tc = *reinterpret_cast<const Vals<VPL> *>(&sTC[tcx]);
#pragma unroll
                    for (int j = 0; j < VPL; j++) X[j] = head ? TM::mx(X[j], tc.x[j]) : X[j];
                }
                if (__any(extra != 0u)) {
                    // rare: wide fan-in.  For each slot with such a position,
                    // the wave's lanes share its gathers beyond two: lane l
                    // takes gather l / LPS of a pass for its own variants (the
                    // variants of lane l % LPS of every slot), then a max over
                    // the lanes holding the same variants reaches the slot
                    uint64_t todo = __ballot(extra != 0u && lis == 0);
                    while (todo) {
                        const int ld = __ffsll((unsigned long long)todo) - 1;
                        todo &= todo - 1;
                        const int qs = __shfl(q, ld, 64);
                        const int64_t e0 = a.gat_ptr[r0 + qs] + 2, e1 = a.gat_ptr[r0 + qs + 1];
                        int64_t mx[VPL];
#pragma unroll
                        for (int j = 0; j < VPL; j++) mx[j] = 0;
                        for (int64_t eb = e0; eb < e1; eb += 64 / LPS) {
                            const int64_t e = eb + lane / LPS;
                            if (e < e1) {
                                const uint8_t c = a.gat_cls[e];
                                const int32_t sp = a.gat_spos[e];
                                Vals<VPL> rel;
                                if (sp < prev_r0) {
                                    const int64_t sx = a.gat_src[e];
                                    const uint32_t rw = a.rm[sx * W + vw];
                                    const int64_t gg = a.gat_gap[e];
                                    const Vals<VPL> fx = *reinterpret_cast<const Vals<VPL> *>(a.finish + sx * V + vvf);
#pragma unroll
                                    for (int j = 0; j < VPL; j++)
                                        rel.x[j] = TM::add(TM::from_time(fx.x[j]),
                                                           ((rw >> (vsh + j)) & 1u) ? 0 : wt(gg));
                                } else {
                                    rel = *reinterpret_cast<const Vals<VPL> *>(&sR[(sp - prev_r0) * VS + o0]);
                                }
#pragma unroll
                                for (int j = 0; j < VPL; j++)
                                    if (cls_on(eon[j], c)) mx[j] = TM::mx(mx[j], rel.x[j]);
                            }
                        }
                        // (bit patterns of nonnegative doubles order as integers)
                        for (int o = LPS; o < 64; o <<= 1) {
#pragma unroll
                            for (int j = 0; j < VPL; j++) mx[j] = max64(mx[j], shfl_xor64(mx[j], o));
                        }
                        if (lane / LPS == ld / LPS) {
#pragma unroll
                            for (int j = 0; j < VPL; j++) X[j] = TM::mx(X[j], mx[j]);
                        }
                    }
                }
                if (anyh) {                                    // a run starts: reset the fold
#pragma unroll
                    for (int j = 0; j < VPL; j++) {
                        A[j] = head ? TM::head : A[j];          // the carry no longer reaches it
                        B[j] = head ? 0 : B[j];
                    }
                }
#pragma unroll
                for (int j = 0; j < VPL; j++) {
                    const bool rmv = (rb >> (o0 + j)) & 1u;
                    const bool live = ok && !rmv;
                    int64_t dp;
                    if (UNI) {
                        const uint64_t te = sT[cls * VS + o0 + j];
                        const uint32_t du = live ? (uint32_t)dur : 0u;   // removed: zero duration
                        dp = TM::i(__builtin_floor((double)du * TM::d((int64_t)te)));
                    } else if (TLDS) {
                        const uint64_t te = sT[cls * VS + o0 + j];
                        if (shift_only) {
                            dp = (int64_t)(((uint64_t)dur * (uint32_t)te) >> ((uint32_t)(te >> 32) & 0xff));
                        } else {
                            dp = scaled8(dur, te, a.table, (int64_t)cls * V + vvf + j);
                        }
                    } else {
                        dp = scaled(dur, a.table[(int64_t)cls * V + vvf + j]);
                    }
                    if (!UNI) dp = live ? dp : 0;
                    const int64_t gp = live ? gap : 0;
                    const int64_t F = TM::add(TM::mx(B[j], X[j]), dp);
                    Dp[i][j] = TM::add(A[j], dp);
                    A[j] = TM::add(Dp[i][j], gp);
                    B[j] = TM::add(F, gp);
                    Fl[i][j] = F;
                    if (START) Dd[i][j] = dp;
                    Gp[i][j] = gp;
                    nkh[i][j] = live ? 0u : kNk;
                }
            }
        }
        if constexpr (NEXT_BIG) issue_big_at(rn1, ke1, qs1, bN, r0, DNb, K - 1);
        else issue(next_small_tag, rn1, bN, r0, DNb);
        put_next();
        // slot summaries (variant-major); slot 0 absorbs the carry and
        // starts its variant (the head value); slots of idle waves are the
        // identity
#pragma unroll
        for (int j = 0; j < VPL; j++) {
            const int e = (o0 + j) * NSP + slot;
            sA[e] = slot == 0 ? TM::head : A[j];
            sB[e] = slot == 0 ? TM::mx(TM::add(carry[j], A[j]), B[j]) : B[j];
        }
        __syncthreads();                                     // B1
        // inclusive scan of slot summaries per variant: DPP within the wave,
        // then earlier 64-slot chunks of the same variant; chunks whose
        // slots all lie past the round's end are skipped
        const int ls = (rn - 1) / ke;                        // last live slot
        int64_t xa[VPL], xb[VPL];
        bool cact[VPL];
        if (NS == 64 * VPL) {
            // wave w scans variant w, lane l its VPL consecutive slots: the
            // lane folds them first (keeping each prefix), one wave scan
            // covers the 64 lane totals, and every slot then takes the
            // release of the lanes before it (lane 0 sees 0: its slot 0
            // already holds the carry)
            const int e0 = wv * NSP + VPL * lane;
            int64_t ta[VPL], tb[VPL];
#pragma unroll
            for (int m = 0; m < VPL; m++) {
                ta[m] = sA[e0 + m];
                tb[m] = sB[e0 + m];
                if (m > 0) compose<UNI>(ta[m - 1], tb[m - 1], ta[m], tb[m]);
            }
            int64_t pa = ta[VPL - 1], pb = tb[VPL - 1];
            wave_scan<UNI>(pa, pb);
            const int qlo = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)pb, 0x138, 0xf, 0xf, true);   // wave_shr:1
            const int qhi = __builtin_amdgcn_update_dpp(0, (int)((uint64_t)pb >> 32), 0x138, 0xf, 0xf, true);
            const int64_t qb = join64(qlo, qhi);
#pragma unroll
            for (int m = 0; m < VPL; m++) sB[e0 + m] = TM::mx(TM::add(qb, ta[m]), tb[m]);
        } else if (NS <= 64 * VPL) {
            // a wave scans whole variants (its VPL chunks hold them): the
            // chunks of one variant follow each other in the same wave
            int64_t pa = 0, pb = 0;
#pragma unroll
            for (int j = 0; j < VPL; j++) {
                const int e = wv * 64 * VPL + j * 64 + lane;
                cact[j] = __any((e % NS) <= ls);
                xa[j] = 0; xb[j] = 0;
                if (cact[j]) {
                    xa[j] = sA[e]; xb[j] = sB[e];
                    wave_scan<UNI>(xa[j], xb[j]);
                    // after the last chunk (a variant's first slot is a head)
                    if (j > 0) compose<UNI>(pa, pb, xa[j], xb[j]);
                    sB[e] = xb[j];
                }
                pa = readlane64(xa[j], 63);
                pb = readlane64(xb[j], 63);
            }
        } else {
#pragma unroll
            for (int j = 0; j < VPL; j++) {
                const int e = tid + j * NT;
                cact[j] = __any((e % NS) <= ls);
                xa[j] = 0; xb[j] = 0;
                if (cact[j]) {
                    xa[j] = sA[e]; xb[j] = sB[e];
                    wave_scan<UNI>(xa[j], xb[j]);
                }
            }
#pragma unroll
            for (int j = 0; j < VPL; j++) {
                const int e = tid + j * NT;
                if (lane == 63) { sTA[e >> 6] = xa[j]; sTB[e >> 6] = xb[j]; }
            }
            __syncthreads();
#pragma unroll
            for (int j = 0; j < VPL; j++) {
                const int e = tid + j * NT;
                const int chunk = (e % NS) >> 6;
                const int first = (e / NS) * (NS >> 6);
                if (cact[j] && chunk > 0) {
                    int64_t qa = sTA[first], qb = sTB[first];
                    for (int c = 1; c < chunk; c++) {
                        int64_t ca = sTA[first + c], cb = sTB[first + c];
                        compose<UNI>(qa, qb, ca, cb);
                        qa = ca; qb = cb;
                    }
                    compose<UNI>(qa, qb, xa[j], xb[j]);
                }
            }
#pragma unroll
            for (int j = 0; j < VPL; j++)
                if (cact[j]) sB[tid + j * NT] = xb[j];
        }
        __syncthreads();                                     // B2
        // finalize: carry-in, results, stores, releases for the next round
        // (the carry-in is read once, before any LDS write of the pass)
        int64_t cin[VPL];
#pragma unroll
        for (int j = 0; j < VPL; j++)
            cin[j] = slot == 0 ? carry[j] : sB[(o0 + j) * NSP + (slot > 0 ? slot - 1 : 0)];
        // does any lane of the wave end a thread's run in this round (its
        // release then goes to the thread carries)?  Mostly not.
        bool anylast = false;
        if (tcar) {
            uint32_t lf = 0;
#pragma unroll
            for (int i = 0; i < K; i++) lf |= FLk[i];
            anylast = __any(lf & 2u);
        }
#pragma unroll
        for (int i = 0; i < K; i++) {
            const int q = slot * ke + i;
            const bool ok = i < ke && q < rn;
            Vals<VPL> fv, sv, rv;
#pragma unroll
            for (int j = 0; j < VPL; j++) { fv.x[j] = 0; sv.x[j] = 0; rv.x[j] = 0; }
            if (wact) {
                const uint32_t flags = FLk[i];
                const bool last = tcar && (flags & 2u);
                const int tcx = ((flags >> 2) & 63u) * VS + o0;
#pragma unroll
                for (int j = 0; j < VPL; j++) {
                    // positions after a run head hold Dp = head value + weights
                    // (below every time, or -inf): the carry has no effect
                    const int64_t F = TM::mx(TM::add(cin[j], Dp[i][j]), Fl[i][j]);
                    rv.x[j] = TM::add(F, Gp[i][j]);
                    fv.x[j] = TM::to_time(F);
                    if (START) sv.x[j] = TM::to_time(TM::sub(F, Dd[i][j]));
                    // makespan over kept tasks (lanes past V never publish theirs)
                    // (positions past ke were not walked: no finish to take)
                    if (i < ke) {
                        const int64_t nk = (int64_t)((uint64_t)nkh[i][j] << 32);
                        if (UNI) ms[j] = TM::mx(ms[j], TM::add(F, nk));
                        else ms[j] = max64(ms[j], (int64_t)((uint64_t)F + (uint64_t)nk));
                    }
                }
                // positions past the round's end write their own unused slot
                // (no young gather reads it); slots past ke would overlap the
                // next slot's positions
                if (i < ke) *reinterpret_cast<Vals<VPL> *>(&sR[q * VS + o0]) = rv;
                if (__builtin_expect(anylast, 0)) {            // wave-uniform: mostly skipped
                    if (last) *reinterpret_cast<Vals<VPL> *>(&sTC[tcx]) = rv;
                }
            }
            // the result address is formed on every lane (an address that
            // no lane stores to is never used), so the choice of the dummy
            // target is a select rather than a masked block
            const bool st = ok && lok;
            const int64_t off = rowoff(U[i], V) + vf;
            gi64 *oa = (gi64 *)(a.finish + off);
            asm volatile("" : "+v"(oa));
            gi64 *o = st ? oa : dummy;
            asm volatile("" : "+v"(o));      // keep one unconditional global store
            store_vals(o, fv);
            if (START) {
                gi64 *osa = (gi64 *)(a.start + off);
                asm volatile("" : "+v"(osa));
                gi64 *os = st ? osa : dummy;
                asm volatile("" : "+v"(os));
                store_vals(os, sv);
            }
        }
#pragma unroll
        for (int j = 0; j < VPL; j++) carry[j] = sB[(o0 + j) * NSP + ls];
        if (slot == 0) {
#pragma unroll
            for (int j = 0; j < VPL; j++) sCarry[o0 + j] = carry[j];
        }
        DN = DNb;
        }   // big round
        prev_r0 = r0;
        D = DN;
        const int bt = b0; b0 = b1; b1 = b2; b2 = bt;
        m0r0 = m1r0; m0rn = m1rn; m1r0 = m2r0; m1rn = m2rn;
        m2r0 = m3r0; m2rn = m3rn; m3r0 = m4r0; m3rn = m4rn;
        __syncthreads();                                     // B3
    };
    // one loop per kind of round and kind of the round after it (the
    // prefetch layout); every kind appears in the order, so each pass of
    // the outer loop takes at least one round
    const std::true_type sm{};
    const std::false_type bg{};
    while (k < nr) {
        for (; k < nr && m0rn <= kSmall && m1rn <= kSmall; k++) round(sm, sm);
        for (; k < nr && m0rn <= kSmall && m1rn > kSmall; k++) round(sm, bg);
        for (; k < nr && m0rn > kSmall && m1rn <= kSmall; k++) round(bg, sm);
        for (; k < nr && m0rn > kSmall && m1rn > kSmall; k++) round(bg, bg);
    }
#pragma unroll
    for (int j = 0; j < VPL; j++) atomicMax(&sMs[o0 + j], (unsigned long long)ms[j]);
    if (wv < VS) atomicMax(&sMs[wv], (unsigned long long)msS0);
    if (PS > 1 && wv + NW < VS) atomicMax(&sMs[wv + NW], (unsigned long long)msS1);
    __syncthreads();
    // (bit patterns of nonnegative doubles order as integers)
    if (tid < VS && v0 + tid < a.V) a.makespan[v0 + tid] = TM::to_time((int64_t)sMs[tid]);
}

// Removal bits per schedule position for each workgroup's VS variants:
// rmp[g][q] = bits g*VS .. g*VS+VS-1 of task pos_node[q]'s removal row.
// A block transposes 128 positions x 64 words through LDS: the row reads are
// contiguous (16 bytes per lane when rows are 16-byte aligned), and every
// lane writes 16 bytes of one workgroup's row (rows are padded to a multiple
// of 16 bytes).
template <int VS, typename RmT, bool V4>
__global__ __launch_bounds__(256) void k_rm_pos(int64_t n, int64_t stride, int32_t W, int32_t nwg,
                                                const int32_t *__restrict__ pos_node,
                                                const uint32_t *__restrict__ rm,
                                                RmT *__restrict__ rmp) {
    constexpr int TP = 128;                       // positions per block
    constexpr int PER = 16 / (int)sizeof(RmT);    // positions per 16-byte store
    constexpr int SEG = TP / PER;                 // stores per workgroup row
    __shared__ uint32_t tile[TP][65];
    const int64_t q0 = (int64_t)blockIdx.x * TP;
    const int w0 = blockIdx.y * 64;
    if constexpr (V4) {
        // 16 lanes per row, 16 rows per pass, all 8 passes in flight (W % 4 == 0)
        constexpr int LD = TP * 16 / 256;
        uint4 v[LD];
#pragma unroll
        for (int r = 0; r < LD; r++) {
            const int i = threadIdx.x + r * 256;
            const int64_t q = q0 + (i >> 4);
            const int w = w0 + (i & 15) * 4;
            const bool ok = q < n && w < W;
            v[r] = ok ? *reinterpret_cast<const uint4 *>(rm + (int64_t)pos_node[q] * W + w)
                      : make_uint4(0u, 0u, 0u, 0u);
        }
#pragma unroll
        for (int r = 0; r < LD; r++) {
            const int i = threadIdx.x + r * 256;
            uint32_t *t = &tile[i >> 4][(i & 15) * 4];
            t[0] = v[r].x; t[1] = v[r].y; t[2] = v[r].z; t[3] = v[r].w;
        }
    } else {
        constexpr int LD = TP * 64 / 256;         // words loaded per lane, all in flight
        uint32_t v[LD];
#pragma unroll
        for (int r = 0; r < LD; r++) {
            const int i = threadIdx.x + r * 256;
            const int64_t q = q0 + (i >> 6);
            const int w = w0 + (i & 63);
            v[r] = (q < n && w < W) ? rm[(int64_t)pos_node[q < n ? q : 0] * W + (w < W ? w : 0)] : 0u;
        }
#pragma unroll
        for (int r = 0; r < LD; r++) {
            const int i = threadIdx.x + r * 256;
            tile[i >> 6][i & 63] = v[r];
        }
    }
    __syncthreads();
    const int g0 = (int)((int64_t)w0 * 32 / VS);
    int64_t g1 = (int64_t)(w0 + 64) * 32 / VS;
    if (g1 > nwg) g1 = nwg;
    constexpr uint32_t mask = VS >= 32 ? ~0u : ((1u << VS) - 1u);
    for (int64_t i = threadIdx.x; i < (g1 - g0) * SEG; i += 256) {
        const int g = g0 + (int)(i / SEG);
        const int pl = (int)(i % SEG) * PER;
        if (q0 + pl >= n) continue;               // the row's padding ends at stride >= n
        const int bitpos = g * VS;
        const int wl = bitpos / 32 - w0, sh = bitpos % 32;
        union {
            RmT b[PER];
            uint4 v;
        } u;
#pragma unroll
        for (int m = 0; m < PER; m++) u.b[m] = (RmT)((tile[pl + m][wl] >> sh) & mask);
        *reinterpret_cast<uint4 *>(rmp + (int64_t)g * stride + q0 + pl) = u.v;
    }
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

template <int LPS, int VPL, int K, bool TLDS, bool START, bool UNI, int NT>
void launch_one(int grid, hipStream_t s, const int32_t *r0, const int32_t *rn,
                const int64_t *nrp, const Rec *rec, const PipeArgs &args) {
    const size_t dyn = TLDS ? (size_t)args.n_cls * LPS * VPL * sizeof(uint64_t) : 0;
    k_sim_pipe<LPS, VPL, K, TLDS, START, UNI, NT><<<grid, NT, dyn, s>>>(r0, rn, nrp, rec, args);
}

// LDS of one workgroup: the kernel's static arrays plus the scale table
template <int LPS, int VPL, int K, int NT>
bool table_fits(int32_t n_cls) {
    constexpr int VS = LPS * VPL;
    if ((int64_t)n_cls * VS > kTabLds) return false;
    hipFuncAttributes at{};
    if (hipFuncGetAttributes(&at, reinterpret_cast<const void *>(
                                      &k_sim_pipe<LPS, VPL, K, true, false, false, NT>)) != hipSuccess)
        return false;
    return at.sharedSizeBytes + (size_t)n_cls * VS * sizeof(uint64_t) <= kLdsBytes;
}

// Device memory one simulation call uses besides its inputs and outputs:
// the round table (cnt, r0, rn), the scan's chunk sums, the removal bits per
// schedule position of each workgroup's variants (rmp) and the target of
// idle lanes' stores.  Laid out in one region, each piece 256-byte aligned.
struct SimLayout {
    size_t cnt, csum, r0, rn, dummy, rmp, bytes;
};

template <int LPS, int VPL, int K, int NT = kNT>
SimLayout sim_layout(const dd_sched *sch, const dd_variants *var) {
    constexpr int VS = LPS * VPL;
    constexpr int RP = (NT / LPS) * K;
    typedef typename std::conditional<(VS <= 8), uint8_t, uint16_t>::type RmT;
    constexpr int64_t kPer = 16 / (int64_t)sizeof(RmT);
    const int64_t ns = sch->n_steps;
    const int64_t max_rounds = ns + (sch->n + RP - 1) / RP + 1;
    const int64_t grid = (var->V + VS - 1) / VS;
    const int64_t rstride = (sch->n + kPer - 1) / kPer * kPer;
    SimLayout L{};
    size_t off = 0;
    auto take = [&](size_t bytes) {
        const size_t at = off;
        off = (off + bytes + 255) & ~(size_t)255;
        return at;
    };
    L.cnt = take(sizeof(int64_t) * (size_t)(ns + 2));
    L.csum = take(sizeof(int64_t) * (size_t)scan_temp_count(ns));
    L.r0 = take(sizeof(int32_t) * (size_t)max_rounds);
    L.rn = take(sizeof(int32_t) * (size_t)max_rounds);
    L.dummy = take(sizeof(int64_t) * 2 * NT);
    L.rmp = take(sizeof(RmT) * (size_t)grid * (size_t)(rstride > 0 ? rstride : kPer));
    L.bytes = off;
    return L;
}

// region == nullptr: the call allocates its memory from the library's cache;
// else it uses region (at least sim_layout().bytes), allocating nothing
template <int LPS, int VPL, int K, int NT = kNT>
hipError_t launch_pipe(const dd_graph *g, const dd_sched *sch, const dd_variants *var,
                       int64_t *finish, int64_t *start, int64_t *makespan, hipStream_t s,
                       unsigned char *region) {
    constexpr int VS = LPS * VPL;
    constexpr int RP = (NT / LPS) * K;
    const int64_t ns = sch->n_steps;
    typedef typename std::conditional<(VS <= 8), uint8_t, uint16_t>::type RmT;
    const int grid = (var->V + VS - 1) / VS;
    constexpr int64_t kPer = 16 / (int64_t)sizeof(RmT);
    const int64_t rstride = (sch->n + kPer - 1) / kPer * kPer;   // rmp row stride
    const SimLayout L = sim_layout<LPS, VPL, K, NT>(sch, var);
    unsigned char *base = region;
    hipError_t e = hipSuccess;
    if (!region) {
        e = dalloc(reinterpret_cast<void **>(&base), L.bytes, s);
        if (e != hipSuccess) return e;
    }
    int64_t *cnt = reinterpret_cast<int64_t *>(base + L.cnt);
    int64_t *csum = reinterpret_cast<int64_t *>(base + L.csum);
    int64_t *dummy = reinterpret_cast<int64_t *>(base + L.dummy);
    int32_t *r0 = reinterpret_cast<int32_t *>(base + L.r0);
    int32_t *rn = reinterpret_cast<int32_t *>(base + L.rn);
    RmT *rmp = reinterpret_cast<RmT *>(base + L.rmp);
    if (sch->n > 0) {
        const dim3 tg((unsigned)((sch->n + 127) / 128), (unsigned)((var->W + 63) / 64));
        if (var->W % 4 == 0)
            k_rm_pos<VS, RmT, true><<<tg, 256, 0, s>>>(sch->n, rstride, var->W, grid, sch->pos_node,
                                                       var->rm_bits, rmp);
        else
            k_rm_pos<VS, RmT, false><<<tg, 256, 0, s>>>(sch->n, rstride, var->W, grid, sch->pos_node,
                                                        var->rm_bits, rmp);
    }
    if (ns > 0) k_round_count<<<grid_for(ns, 256), 256, 0, s>>>(ns, sch->step_ptr, RP, cnt);
    e = scan_exclusive_ws(cnt, cnt, ns, csum, s);
    if (e == hipSuccess && ns > 0)
        k_round_fill<<<grid_for(ns, 256), 256, 0, s>>>(ns, sch->step_ptr, cnt, RP, r0, rn);
    const uint64_t cls_mask = sch->mask & g->cross_mask;
    PipeArgs args{sch->gat_ptr, sch->gat_src, sch->gat_spos, sch->gat_cls, sch->gat_gap, g->gap,
                  var->table, var->n_cls, var->rm_bits, rmp, rstride, var->edge_on,
                  cls_mask, sch->thread_carry ? 1 : 0, var->V, var->W, finish, start, makespan,
                  dummy};
    const int64_t *nrp = cnt + ns;
    const bool tl = table_fits<LPS, VPL, K, NT>(var->n_cls);
    // uniform: every gather class on in every variant, shift-only scales,
    // durations and gaps below 2^32 (a source's gap then rides in its
    // record), times within the bounds of the double arithmetic
    const bool uni = tl && (var->all_mask & cls_mask) == cls_mask && !var->any_magic &&
                     g->dmax < (int64_t(1) << 32) && g->gmax < (int64_t(1) << 32) &&
                     var->f64_ok;
    const Rec *rc = sch->rec;
    if (e == hipSuccess) {
        if (uni && start) launch_one<LPS, VPL, K, true, true, true, NT>(grid, s, r0, rn, nrp, rc, args);
        else if (uni) launch_one<LPS, VPL, K, true, false, true, NT>(grid, s, r0, rn, nrp, rc, args);
        else if (tl && start) launch_one<LPS, VPL, K, true, true, false, NT>(grid, s, r0, rn, nrp, rc, args);
        else if (tl) launch_one<LPS, VPL, K, true, false, false, NT>(grid, s, r0, rn, nrp, rc, args);
        else if (start) launch_one<LPS, VPL, K, false, true, false, NT>(grid, s, r0, rn, nrp, rc, args);
        else launch_one<LPS, VPL, K, false, false, false, NT>(grid, s, r0, rn, nrp, rc, args);
        e = hipGetLastError();
    }
    if (!region) dfree(base, s);
    return e;
}

// the kernel instance for a launch shape: <lanes per slot, variants per
// lane, positions per slot>; a round holds at most 512 positions (LDS record
// ring); two variants per lane when V is even (16 B loads and stores stay
// inside a row).  f(instance) is called with the instance as template
// arguments.
template <class F>
auto with_shape(const dd_variants *var, int vs_hint, F &&f) {
    const int vs = vs_hint > 0 ? vs_hint : strip_width(var->V);
    const bool pair = (var->V % 2) == 0;
    switch (vs) {
        case 1: return f(std::integral_constant<int, 1>{}, std::integral_constant<int, 1>{},
                         std::integral_constant<int, 1>{});
        case 2: return pair ? f(std::integral_constant<int, 1>{}, std::integral_constant<int, 2>{},
                                std::integral_constant<int, 1>{})
                            : f(std::integral_constant<int, 2>{}, std::integral_constant<int, 1>{},
                                std::integral_constant<int, 2>{});
        case 4: return pair ? f(std::integral_constant<int, 2>{}, std::integral_constant<int, 2>{},
                                std::integral_constant<int, 2>{})
                            : f(std::integral_constant<int, 4>{}, std::integral_constant<int, 1>{},
                                std::integral_constant<int, 4>{});
        case 8: return pair ? f(std::integral_constant<int, 4>{}, std::integral_constant<int, 2>{},
                                std::integral_constant<int, 4>{})
                            : f(std::integral_constant<int, 8>{}, std::integral_constant<int, 1>{},
                                std::integral_constant<int, 8>{});
        default: return pair ? f(std::integral_constant<int, 8>{}, std::integral_constant<int, 2>{},
                                 std::integral_constant<int, 4>{})
                             : f(std::integral_constant<int, 16>{}, std::integral_constant<int, 1>{},
                                 std::integral_constant<int, 8>{});
    }
}

// Scratch of the allocation-free entry point: one array per GPU, held until
// the process ends.  Host code takes its device address once per device
// (hipGetSymbolAddress) and uses only that address.
constexpr size_t kScratchBytes = size_t(64) << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
unsigned char *g_scratch_ptr[kMaxDevices];

}  // namespace

hipError_t launch_simulate(const dd_graph *g, const dd_sched *sch, const dd_variants *var,
                           int64_t *finish, int64_t *start, int64_t *makespan, int vs_hint,
                           hipStream_t s) {
    return with_shape(var, vs_hint, [&](auto lps, auto vpl, auto k) {
        return launch_pipe<decltype(lps)::value, decltype(vpl)::value, decltype(k)::value>(
            g, sch, var, finish, start, makespan, s, nullptr);
    });
}

hipError_t simulate_noalloc(const dd_graph *g, const dd_sched *sch, const dd_variants *var,
                            int64_t *finish, int64_t *start, int64_t *makespan, hipStream_t s,
                            size_t *need, size_t *limit) {
    *limit = kScratchBytes;
    *need = with_shape(var, 0, [&](auto lps, auto vpl, auto k) {
        return sim_layout<decltype(lps)::value, decltype(vpl)::value, decltype(k)::value>(sch, var)
            .bytes;
    });
    if (*need > kScratchBytes) return hipErrorInvalidValue;
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    unsigned char *ptr = nullptr;
    {
        std::lock_guard<std::mutex> lk(g_scratch_mu);
        if (!g_scratch_ptr[dev]) {
            void *p = nullptr;
            e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
            if (e != hipSuccess) return e;
            g_scratch_ptr[dev] = static_cast<unsigned char *>(p);
        }
        ptr = g_scratch_ptr[dev];
    }
    return with_shape(var, 0, [&](auto lps, auto vpl, auto k) {
        return launch_pipe<decltype(lps)::value, decltype(vpl)::value, decltype(k)::value>(
            g, sch, var, finish, start, makespan, s, ptr);
    });
}

}  // namespace dd
