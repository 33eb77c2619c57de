// Graph load: validation, thread-chain ranking, cross-thread edge lists,
// plus the prefix-sum utility used across the library.
//
// The task graph is the one of Sec. 4.2: tasks with an execution thread,
// duration and gap (Sec. 4.2.1) and the dependency types of Sec. 4.2.2.
// Consecutive tasks on one thread are ordered (a dependency type itself);
// the chain of each thread is ranked here by pointer jumping so that every
// later kernel can address "position p on thread t".  A dependency between
// two tasks of the same thread is implied by the thread order (release
// times never decrease along a thread) and is dropped after checking that
// it points forward.

#include "dd_common.h"
#include "dd_internal.h"

namespace dd {

// ---------------------------------------------------------------------------
// exclusive scan (three passes: chunk sums, scan of sums, apply)
namespace {
constexpr int kScanBS = 256;
constexpr int kScanIPT = 16;
constexpr int64_t kScanChunk = kScanBS * kScanIPT;

__global__ __launch_bounds__(kScanBS) void k_scan_chunk_sums(const int64_t *in, int64_t n,
                                                             int64_t *csum) {
    const int64_t lo = (int64_t)blockIdx.x * kScanChunk;
    const int64_t hi = lo + kScanChunk < n ? lo + kScanChunk : n;
    int64_t s = 0;
    for (int64_t i = lo + threadIdx.x; i < hi; i += kScanBS) s += in[i];
    int64_t tot;
    (void)block_excl_scan<kScanBS>(s, &tot);
    if (threadIdx.x == 0) csum[blockIdx.x] = tot;
}

__global__ __launch_bounds__(1024) void k_scan_chunk_offsets(int64_t *csum, int64_t nc,
                                                             int64_t *out_total) {
    int64_t carry = 0;
    for (int64_t base = 0; base < nc; base += 1024) {
        int64_t i = base + threadIdx.x;
        int64_t v = i < nc ? csum[i] : 0;
        int64_t tot;
        int64_t ex = block_excl_scan<1024>(v, &tot);
        if (i < nc) csum[i] = carry + ex;
        carry += tot;
    }
    if (threadIdx.x == 0) *out_total = carry;
}

__global__ __launch_bounds__(kScanBS) void k_scan_apply(const int64_t *in, int64_t n,
                                                        const int64_t *coff, int64_t *out) {
    const int64_t lo = (int64_t)blockIdx.x * kScanChunk + (int64_t)threadIdx.x * kScanIPT;
    int64_t v[kScanIPT];
    int64_t s = 0;
#pragma unroll
    for (int k = 0; k < kScanIPT; k++) {
        v[k] = (lo + k < n) ? in[lo + k] : 0;
        s += v[k];
    }
    int64_t tot;
    int64_t ex = block_excl_scan<kScanBS>(s, &tot) + coff[blockIdx.x];
#pragma unroll
    for (int k = 0; k < kScanIPT; k++) {
        if (lo + k < n) out[lo + k] = ex;
        ex += v[k];
    }
}
}  // namespace

int64_t scan_temp_count(int64_t n) {
    const int64_t nc = (n + kScanChunk - 1) / kScanChunk;
    return nc < 1 ? 1 : nc;
}

hipError_t scan_exclusive_ws(const int64_t *in, int64_t *out, int64_t n, int64_t *csum,
                             hipStream_t s) {
    const int64_t nc = scan_temp_count(n);
    if (n > 0) k_scan_chunk_sums<<<(unsigned)nc, kScanBS, 0, s>>>(in, n, csum);
    // (with n == 0 the single chunk sum is never read: the offsets pass
    // scans one chunk of zero tasks)
    k_scan_chunk_offsets<<<1, 1024, 0, s>>>(csum, n > 0 ? nc : 0, out + n);
    if (n > 0) k_scan_apply<<<(unsigned)nc, kScanBS, 0, s>>>(in, n, csum, out);
    return hipGetLastError();
}

hipError_t scan_exclusive(const int64_t *in, int64_t *out, int64_t n, hipStream_t s) {
    int64_t *csum = nullptr;
    hipError_t e = dalloc_n(&csum, (size_t)scan_temp_count(n), s);
    if (e != hipSuccess) return e;
    e = scan_exclusive_ws(in, out, n, csum, s);
    dfree(csum, s);
    return e;
}

// ---------------------------------------------------------------------------
// validation of per-task fields
namespace {
constexpr int kBS = 256;

constexpr int kValBlocks = 256;    // grid-stride blocks: one set of atomics per block

__global__ __launch_bounds__(kBS) void k_validate_nodes(
    int32_t n, int32_t T, const int32_t *__restrict__ prev, const int32_t *__restrict__ tid,
    const int64_t *__restrict__ dur, const int64_t *__restrict__ gap,
    const uint16_t *__restrict__ cls, const int64_t *__restrict__ in_ptr,
    int32_t *__restrict__ succ, int32_t *__restrict__ heads, uint32_t *__restrict__ err,
    LoadStats *__restrict__ st, bool one_head) {
    uint32_t e = 0;
    // sums split at bit 32 so that no partial sum can overflow
    int64_t dhi = 0, dlo = 0, ghi = 0, glo = 0, dm = 0, gm = 0, cm = 0;
    for (int64_t u = (int64_t)blockIdx.x * kBS + threadIdx.x; u < n;
         u += (int64_t)gridDim.x * kBS) {
        const int32_t t = tid[u];
        const bool t_ok = t >= 0 && t < T;
        if (!t_ok) e |= ERR_THREAD_RANGE;
        const int32_t p = prev[u];
        if (p < -1 || p >= n || p == u) {
            e |= ERR_PREV_RANGE;
        } else if (p >= 0) {
            if (tid[p] != t) e |= ERR_PREV_THREAD;
            else succ[p] = (int32_t)u + 1;   // one claimer wins; the others are found later
        } else if (t_ok && one_head) {
            if (atomicAdd(&heads[t], 1) != 0) e |= ERR_HEADS;
        }
        int64_t d = dur[u], g = gap[u];
        if (d < 0 || g < 0) e |= ERR_NEG_TIME;
        if (d >= kTimeLimit || g >= kTimeLimit) e |= ERR_BIG_TIME;
        if (d < 0 || d >= kTimeLimit) d = 0;
        if (g < 0 || g >= kTimeLimit) g = 0;
        if (in_ptr[u + 1] < in_ptr[u]) e |= ERR_PTR_ORDER;
        const int64_t c = cls ? cls[u] : 0;
        dhi += d >> 32; dlo += d & 0xffffffffll;
        ghi += g >> 32; glo += g & 0xffffffffll;
        dm = d > dm ? d : dm;
        gm = g > gm ? g : gm;
        cm = c > cm ? c : cm;
    }
    // wave reduction, then the block's waves through LDS, one atomic set per block
    dhi = wave_sum64(dhi); dlo = wave_sum64(dlo);
    ghi = wave_sum64(ghi); glo = wave_sum64(glo);
    dm = wave_max64(dm); gm = wave_max64(gm); cm = wave_max64(cm);
    for (int o = 32; o > 0; o >>= 1) e |= (uint32_t)__shfl_xor((int)e, o, 64);
    constexpr int NW = kBS / 64;
    __shared__ int64_t red[8][NW];
    const int w = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) {
        red[0][w] = dhi; red[1][w] = dlo; red[2][w] = ghi; red[3][w] = glo;
        red[4][w] = dm; red[5][w] = cm; red[6][w] = e; red[7][w] = gm;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int i = 1; i < NW; i++) {
            dhi += red[0][i]; dlo += red[1][i]; ghi += red[2][i]; glo += red[3][i];
            dm = red[4][i] > dm ? red[4][i] : dm;
            cm = red[5][i] > cm ? red[5][i] : cm;
            e |= (uint32_t)red[6][i];
            gm = red[7][i] > gm ? red[7][i] : gm;
        }
        if (dhi) atomicAdd(&st->dsum_hi, (unsigned long long)dhi);
        if (dlo) atomicAdd(&st->dsum_lo, (unsigned long long)dlo);
        if (ghi) atomicAdd(&st->gsum_hi, (unsigned long long)ghi);
        if (glo) atomicAdd(&st->gsum_lo, (unsigned long long)glo);
        atomic_max_hot(&st->dmax, (unsigned long long)dm);
        atomic_max_hot(&st->gmax, (unsigned long long)gm);
        atomic_max_hot(&st->cls_max, (unsigned long long)cm);
        atomic_or_hot(err, e);
    }
}

// (runs right after the per-task pass, before its errors are read, so every
// index is clamped to its array; also reports a task named as previous task
// by two tasks, which left only one of them in succ)
__global__ __launch_bounds__(kBS) void k_validate_edges(int32_t n, int64_t E,
                                                        const int64_t *__restrict__ in_ptr,
                                                        const int32_t *__restrict__ in_src,
                                                        const uint8_t *__restrict__ ecls,
                                                        const int32_t *__restrict__ prev,
                                                        const int32_t *__restrict__ succ,
                                                        uint32_t *__restrict__ err) {
    const int64_t u = (int64_t)blockIdx.x * kBS + threadIdx.x;
    uint32_t e = 0;
    if (u < n) {
        const int32_t p = prev[u];
        if (p >= 0 && p < n && succ[p] != (int32_t)u + 1) e |= ERR_SUCC;
        const int64_t k0 = in_ptr[u] > 0 ? in_ptr[u] : 0;
        const int64_t k1 = in_ptr[u + 1] < E ? in_ptr[u + 1] : E;
        for (int64_t k = k0; k < k1; k++) {
            const int32_t s = in_src[k];
            if (s < 0 || s >= n) e |= ERR_SRC_RANGE;
            else if (s == u) e |= ERR_SELF_LOOP;
            if (ecls && ecls[k] >= 64) e |= ERR_EDGE_CLS;
        }
    }
    for (int o = 32; o > 0; o >>= 1) e |= (uint32_t)__shfl_xor((int)e, o, 64);
    if ((threadIdx.x & 63) == 0 && e) atomicOr(err, e);
}

// pointer jumping (Wyllie): rank = number of predecessors on the thread
__global__ __launch_bounds__(kBS) void k_rank_init(int32_t n, const int32_t *__restrict__ prev,
                                                   int32_t *__restrict__ nxt,
                                                   int32_t *__restrict__ rank) {
    const int64_t u = (int64_t)blockIdx.x * kBS + threadIdx.x;
    if (u < n) {
        nxt[u] = prev[u];
        rank[u] = prev[u] >= 0 ? 1 : 0;
    }
}

__global__ __launch_bounds__(kBS) void k_rank_step(int32_t n, const int32_t *__restrict__ nxt_in,
                                                   const int32_t *__restrict__ rank_in,
                                                   int32_t *__restrict__ nxt_out,
                                                   int32_t *__restrict__ rank_out) {
    const int64_t u = (int64_t)blockIdx.x * kBS + threadIdx.x;
    if (u < n) {
        const int32_t p = nxt_in[u];
        if (p >= 0) {
            // unsigned: a looping chain (reported afterwards) must not overflow
            rank_out[u] = (int32_t)((uint32_t)rank_in[u] + (uint32_t)rank_in[p]);
            nxt_out[u] = nxt_in[p];
        } else {
            rank_out[u] = rank_in[u];
            nxt_out[u] = -1;
        }
    }
}

__global__ __launch_bounds__(kBS) void k_rank_check(int32_t n, const int32_t *__restrict__ nxt,
                                                    uint32_t *__restrict__ err) {
    const int64_t u = (int64_t)blockIdx.x * kBS + threadIdx.x;
    bool bad = u < n && nxt[u] != -1;
    if (__any(bad) && (threadIdx.x & 63) == 0) atomicOr(err, ERR_CHAIN_CYCLE);
}

// Chain ranking in two levels.  Tasks of a thread are mostly close in id
// (traces interleave a few threads), so a tile of kRankTile consecutive ids
// resolves most of each chain with pointer jumping in LDS: every task gets
// d (predecessors up to and including the first one outside the tile) and
// e (that outside task, -1 if the chain starts in the tile), so that
// rank(u) = d + rank(e).  The outside tasks named as e (the tile exits) are
// then ranked by one workgroup, again by pointer jumping in LDS, and every
// task adds its exit's rank.  A thread order that loops inside a tile or
// across exits is reported like the plain pointer jumping does.
constexpr int kRankTile = 1024;
constexpr int kRankXMax = 8192;     // tile exits ranked in LDS at most

__global__ __launch_bounds__(kRankTile) void k_rank_tile(int32_t n, const int32_t *__restrict__ prev,
                                                         int32_t *__restrict__ dloc,
                                                         int32_t *__restrict__ ext,
                                                         int64_t *__restrict__ xflag,
                                                         uint32_t *__restrict__ err) {
    __shared__ int32_t sn[2][kRankTile], sd[2][kRankTile], se[2][kRankTile];
    const int64_t b0 = (int64_t)blockIdx.x * kRankTile;
    const int i = threadIdx.x;
    const int64_t u = b0 + i;
    const bool ok = u < n;
    int32_t p = ok ? prev[u] : -1;
    if (p < -1 || p >= n || p == u) p = -1;   // reported by the per-task pass
    const bool in = p >= b0 && p < b0 + kRankTile && p < n;
    int nn = in ? (int)(p - b0) : -1;
    int d = p >= 0 ? 1 : 0;
    int e = in ? -1 : p;
    int buf = 0;
    sn[0][i] = nn; sd[0][i] = d; se[0][i] = e;
    __syncthreads();
    for (int it = 0; it < 11; it++) {        // 2^10 = kRankTile: every in-tile chain ends
        if (nn >= 0) {
            const int j = nn;
            d += sd[buf][j];
            e = se[buf][j];
            nn = sn[buf][j];
        }
        buf ^= 1;
        sn[buf][i] = nn; sd[buf][i] = d; se[buf][i] = e;
        __syncthreads();
    }
    if (__any(ok && nn >= 0) && (i & 63) == 0) atomicOr(err, ERR_CHAIN_CYCLE);
    if (ok) {
        dloc[u] = d;
        ext[u] = e;
        if (e >= 0) xflag[e] = 1;
    }
}

__global__ __launch_bounds__(kBS) void k_rank_xlist(int32_t n, const int64_t *__restrict__ xidx,
                                                    int32_t *__restrict__ xlist) {
    const int64_t u = (int64_t)blockIdx.x * kBS + threadIdx.x;
    if (u < n && xidx[u + 1] != xidx[u]) xlist[xidx[u]] = (int32_t)u;
}

// ranks of the tile exits (one workgroup); err[1] is set when there are more
// than kRankXMax of them (the caller then ranks by plain pointer jumping)
__global__ __launch_bounds__(1024) void k_rank_exits(int32_t n, const int64_t *__restrict__ xidx,
                                                     const int32_t *__restrict__ xlist,
                                                     const int32_t *__restrict__ dloc,
                                                     const int32_t *__restrict__ ext,
                                                     int32_t *__restrict__ rank,
                                                     uint32_t *__restrict__ err) {
    __shared__ int32_t sn[2][kRankXMax], sd[2][kRankXMax];
    const int64_t nx = xidx[n];
    if (nx > kRankXMax) {
        if (threadIdx.x == 0) err[1] = 1u;
        return;
    }
    constexpr int PER = kRankXMax / 1024;
    int nn[PER], d[PER];
#pragma unroll
    for (int k = 0; k < PER; k++) {
        const int x = threadIdx.x + k * 1024;
        nn[k] = -1; d[k] = 0;
        if (x < nx) {
            const int32_t u = xlist[x];
            const int32_t e = ext[u];
            d[k] = dloc[u];
            nn[k] = e >= 0 ? (int)xidx[e] : -1;
        }
        sn[0][x] = nn[k]; sd[0][x] = d[k];
    }
    __syncthreads();
    int buf = 0;
    for (int it = 0; it < 14; it++) {        // 2^13 = kRankXMax: every exit chain ends
#pragma unroll
        for (int k = 0; k < PER; k++) {
            if (nn[k] >= 0) {
                const int j = nn[k];
                d[k] += sd[buf][j];
                nn[k] = sn[buf][j];
            }
        }
        buf ^= 1;
#pragma unroll
        for (int k = 0; k < PER; k++) {
            const int x = threadIdx.x + k * 1024;
            sn[buf][x] = nn[k]; sd[buf][x] = d[k];
        }
        __syncthreads();
    }
    bool bad = false;
#pragma unroll
    for (int k = 0; k < PER; k++) {
        const int x = threadIdx.x + k * 1024;
        bad |= x < nx && nn[k] >= 0;
        if (x < nx) rank[xlist[x]] = d[k];
    }
    if (__any(bad) && (threadIdx.x & 63) == 0) atomicOr(err, ERR_CHAIN_CYCLE);
}

__global__ __launch_bounds__(kBS) void k_rank_final(int32_t n, const int32_t *__restrict__ dloc,
                                                    const int32_t *__restrict__ ext,
                                                    const int64_t *__restrict__ xidx,
                                                    int32_t *__restrict__ rank) {
    const int64_t u = (int64_t)blockIdx.x * kBS + threadIdx.x;
    if (u >= n || xidx[u + 1] != xidx[u]) return;   // exits hold their rank already
    const int32_t e = ext[u];
    rank[u] = dloc[u] + (e >= 0 ? rank[e] : 0);
}

__global__ __launch_bounds__(kBS) void k_thread_len(int32_t n, const int32_t *__restrict__ succ,
                                                    const int32_t *__restrict__ tid,
                                                    const int32_t *__restrict__ rank,
                                                    int64_t *__restrict__ len) {
    const int64_t u = (int64_t)blockIdx.x * kBS + threadIdx.x;
    if (u < n && succ[u] == 0) len[tid[u]] = (int64_t)rank[u] + 1;   // last task of its thread (no successor)
}

__global__ __launch_bounds__(kBS) void k_order(int32_t n, const int32_t *__restrict__ tid,
                                               const int32_t *__restrict__ rank,
                                               const int64_t *__restrict__ base,
                                               int32_t *__restrict__ order) {
    const int64_t u = (int64_t)blockIdx.x * kBS + threadIdx.x;
    if (u < n) order[base[tid[u]] + rank[u]] = (int32_t)u;
}

// same-thread dependencies: must point forward; dropped.  Cross-thread: counted.
__global__ __launch_bounds__(kBS) void k_cross_count(
    int32_t n, const int64_t *__restrict__ in_ptr, const int32_t *__restrict__ in_src,
    const uint8_t *__restrict__ ecls, const int32_t *__restrict__ tid,
    const int32_t *__restrict__ rank, int64_t *__restrict__ cnt, uint32_t *__restrict__ err,
    LoadStats *__restrict__ st) {
    const int64_t u = (int64_t)blockIdx.x * kBS + threadIdx.x;
    uint32_t e = 0;
    uint64_t mask = 0;
    if (u < n) {
        int64_t c = 0;
        const int32_t tu = tid[u];
        for (int64_t k = in_ptr[u]; k < in_ptr[u + 1]; k++) {
            const int32_t s = in_src[k];
            if (tid[s] == tu) {
                if (rank[s] >= rank[u]) e |= ERR_BACK_EDGE;
            } else {
                c++;
                mask |= 1ull << (ecls ? ecls[k] : 0);
            }
        }
        cnt[u] = c;
    }
    for (int o = 32; o > 0; o >>= 1) {
        e |= (uint32_t)__shfl_xor((int)e, o, 64);
        mask |= (uint64_t)shfl_xor64((int64_t)mask, o);
    }
    if ((threadIdx.x & 63) == 0) {
        atomic_or_hot(err, e);
        atomic_or_hot(&st->cross_mask, (unsigned long long)mask);
    }
}

__global__ __launch_bounds__(kBS) void k_cross_fill(
    int32_t n, const int64_t *__restrict__ in_ptr, const int32_t *__restrict__ in_src,
    const uint8_t *__restrict__ ecls, const int32_t *__restrict__ tid,
    const int64_t *__restrict__ xptr, int32_t *__restrict__ xsrc, uint8_t *__restrict__ xcls) {
    const int64_t u = (int64_t)blockIdx.x * kBS + threadIdx.x;
    if (u >= n) return;
    int64_t o = xptr[u];
    const int32_t tu = tid[u];
    for (int64_t k = in_ptr[u]; k < in_ptr[u + 1]; k++) {
        const int32_t s = in_src[k];
        if (tid[s] != tu) {
            xsrc[o] = s;
            xcls[o] = ecls ? ecls[k] : 0;
            o++;
        }
    }
}
}  // namespace

hipError_t launch_validate_nodes(const dd_graph *g, const int64_t *in_ptr, int32_t *succ,
                                 int32_t *heads, uint32_t *err, LoadStats *st, hipStream_t s) {
    int blocks = grid_for(g->n, kBS);
    if (blocks > kValBlocks) blocks = kValBlocks;
    k_validate_nodes<<<blocks, kBS, 0, s>>>(g->n, g->n_threads, g->thread_prev,
                                                         g->thread_id, g->dur, g->gap, g->cls,
                                                         in_ptr, succ, heads, err, st,
                                                         !g->shared);
    return hipGetLastError();
}

hipError_t launch_validate_edges(const dd_graph *g, const int64_t *in_ptr, const int32_t *in_src,
                                 const uint8_t *edge_cls, const int32_t *succ, uint32_t *err,
                                 hipStream_t s) {
    k_validate_edges<<<grid_for(g->n, kBS), kBS, 0, s>>>(g->n, g->n_edges, in_ptr, in_src, edge_cls,
                                                         g->thread_prev, succ, err);
    return hipGetLastError();
}

hipError_t launch_rank_tiles(const dd_graph *g, int32_t *dloc, int32_t *ext, int32_t *xlist,
                             int64_t *xidx, uint32_t *err, hipStream_t s) {
    const int32_t n = g->n;
    hipError_t e = hipMemsetAsync(xidx, 0, sizeof(int64_t) * ((size_t)n + 1), s);
    if (e != hipSuccess) return e;
    k_rank_tile<<<(unsigned)((n + kRankTile - 1) / kRankTile), kRankTile, 0, s>>>(n, g->thread_prev,
                                                                               dloc, ext, xidx, err);
    e = scan_exclusive(xidx, xidx, n, s);
    if (e != hipSuccess) return e;
    k_rank_xlist<<<grid_for(n, kBS), kBS, 0, s>>>(n, xidx, xlist);
    k_rank_exits<<<1, 1024, 0, s>>>(n, xidx, xlist, dloc, ext, g->rank, err);
    k_rank_final<<<grid_for(n, kBS), kBS, 0, s>>>(n, dloc, ext, xidx, g->rank);
    return hipGetLastError();
}

hipError_t launch_rank_chains(const dd_graph *g, const int32_t *succ, int32_t *nxt,
                              int32_t *nxt2, int32_t *rank2, uint32_t *err, hipStream_t s) {
    (void)succ;
    const int32_t n = g->n;
    int gr = grid_for(n, kBS);
    k_rank_init<<<gr, kBS, 0, s>>>(n, g->thread_prev, nxt, g->rank);
    int steps = 1;
    while ((int64_t(1) << steps) <= (int64_t)n + 1) steps++;
    int32_t *a_n = nxt, *a_r = g->rank, *b_n = nxt2, *b_r = rank2;
    for (int i = 0; i < steps; i++) {
        k_rank_step<<<gr, kBS, 0, s>>>(n, a_n, a_r, b_n, b_r);
        int32_t *t;
        t = a_n; a_n = b_n; b_n = t;
        t = a_r; a_r = b_r; b_r = t;
    }
    if (a_r != g->rank) (void)hipMemcpyAsync(g->rank, a_r, sizeof(int32_t) * (size_t)n,
                                       hipMemcpyDeviceToDevice, s);
    k_rank_check<<<gr, kBS, 0, s>>>(n, a_n, err);
    return hipGetLastError();
}

hipError_t launch_build_order(const dd_graph *g, const int32_t *succ, int64_t *len,
                              hipStream_t s) {
    const int32_t n = g->n;
    (void)hipMemsetAsync(len, 0, sizeof(int64_t) * ((size_t)g->n_threads + 1), s);
    k_thread_len<<<grid_for(n, kBS), kBS, 0, s>>>(n, succ, g->thread_id, g->rank, len);
    hipError_t e = scan_exclusive(len, g->thread_base, g->n_threads, s);
    if (e != hipSuccess) return e;
    k_order<<<grid_for(n, kBS), kBS, 0, s>>>(n, g->thread_id, g->rank, g->thread_base, g->order);
    return hipGetLastError();
}

hipError_t launch_cross_edges(dd_graph *g, const int64_t *in_ptr, const int32_t *in_src,
                              const uint8_t *edge_cls, int64_t *cnt, uint32_t *err, LoadStats *st,
                              hipStream_t s) {
    k_cross_count<<<grid_for(g->n, kBS), kBS, 0, s>>>(g->n, in_ptr, in_src, edge_cls,
                                                      g->thread_id, g->rank, cnt, err, st);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return scan_exclusive(cnt, g->xin_ptr, g->n, s);
}

hipError_t launch_cross_fill(dd_graph *g, const int64_t *in_ptr, const int32_t *in_src,
                             const uint8_t *edge_cls, hipStream_t s) {
    k_cross_fill<<<grid_for(g->n, kBS), kBS, 0, s>>>(g->n, in_ptr, in_src, edge_cls,
                                                     g->thread_id, g->xin_ptr, g->xin_src,
                                                     g->xin_cls);
    return hipGetLastError();
}

}  // namespace dd
