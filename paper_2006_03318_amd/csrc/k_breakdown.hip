// Runtime breakdown of every variant (Sec. 6.2, Fig. 6: where the iteration
// time goes once the CPU and the GPU overlap), from a finished simulation:
//   total    = the iteration time (makespan);
//   CPU-only = total minus all GPU kernel runtime, i.e. minus the sum of the
//              scaled durations d' of the kernels kept in the variant;
//   GPU-only = the time the CPU is blocked on the GPU: for every call that
//              waits for GPU work (synchronization, device-to-host copy), its
//              start minus the moment its thread reached it (the release of
//              the previous task on the thread, 0 for the first);
//   CPU+GPU parallel = total - CPU-only - GPU-only.
// A call's start is its finish minus its scaled duration, and a release is
// finish + g', so the finish array alone carries the schedule.
//
// The tasks with a role are first ordered by task class (a counting sort),
// so along a workgroup's chunk the class, and with it each lane's scale
// entry, changes rarely: a lane reloads its entry only when the (wave-
// uniform) class changes.  Each workgroup owns 1,024 variants and a chunk of
// the ordered tasks, so a task's fields are
// wave-uniform and the per-variant reads (removal words, finish values of
// waiting calls) are contiguous across the wave; a thread serves four
// consecutive variants.  Partial sums go to a per-variant accumulator with
// one atomic per variant and thread.

#include "dd_common.h"
#include "dd_internal.h"

namespace dd {
namespace {

constexpr int kBT = 256;          // threads per workgroup
constexpr int kVL = 4;            // variants per thread (divides 32)
constexpr int64_t kChunk = 512;   // ordered tasks per workgroup
constexpr int kBatch = 8;         // tasks whose loads are issued together


__device__ __forceinline__ bool has_role(uint8_t r) { return r == 1u || r == 2u; }

// Counting sort of the tasks with a role by class.  With few classes each
// block first counts (and ranks) its own tasks in LDS, so one global atomic
// per (block, class) replaces one per task: thousands of tasks share a
// handful of counters.
constexpr int kLdsCls = 2048;     // classes counted in LDS at most

__global__ __launch_bounds__(kBT) void k_bd_count(int64_t n, int32_t n_cls,
                                                  const uint8_t *__restrict__ role,
                                                  const uint16_t *__restrict__ cls,
                                                  unsigned long long *__restrict__ hist) {
    __shared__ uint32_t h[kLdsCls];
    const int64_t u = (int64_t)blockIdx.x * kBT + threadIdx.x;
    const bool lds = n_cls <= kLdsCls;
    const bool has = u < n && has_role(role[u]);
    const uint32_t c = has ? cls[u] : 0u;
    if (lds) {
        for (int i = threadIdx.x; i < n_cls; i += kBT) h[i] = 0;
        __syncthreads();
        if (has) atomicAdd(&h[c], 1u);
        __syncthreads();
        for (int i = threadIdx.x; i < n_cls; i += kBT)
            if (h[i]) atomicAdd(&hist[i], (unsigned long long)h[i]);
    } else if (has) {
        atomicAdd(&hist[c], 1ull);
    }
}

__global__ __launch_bounds__(kBT) void k_bd_scatter(int64_t n, int32_t n_cls,
                                                    const uint8_t *__restrict__ role,
                                                    const uint16_t *__restrict__ cls,
                                                    unsigned long long *__restrict__ cursor,
                                                    int32_t *__restrict__ order) {
    __shared__ uint32_t h[kLdsCls];
    __shared__ unsigned long long base[kLdsCls];
    const int64_t u = (int64_t)blockIdx.x * kBT + threadIdx.x;
    const bool has = u < n && has_role(role[u]);
    const uint32_t c = has ? cls[u] : 0u;
    if (n_cls <= kLdsCls) {
        for (int i = threadIdx.x; i < n_cls; i += kBT) h[i] = 0;
        __syncthreads();
        const uint32_t rank = has ? atomicAdd(&h[c], 1u) : 0u;   // rank inside the block
        __syncthreads();
        for (int i = threadIdx.x; i < n_cls; i += kBT)
            if (h[i]) base[i] = atomicAdd(&cursor[i], (unsigned long long)h[i]);
        __syncthreads();
        if (has) order[base[c] + rank] = (int32_t)u;
    } else if (has) {
        order[atomicAdd(&cursor[c], 1ull)] = (int32_t)u;
    }
}

struct BdArgs {
    int32_t V, W, nvb, nch;
    const ScaleEntry *table;
    const uint32_t *rm;
    const int64_t *finish;
    unsigned long long *acc;      // [2][V]: kernel time, blocked time
};

// scaled duration: MAGIC when some q of the launch is not a power of two
// (else a shift suffices), D32 when every duration is below 2^32 (one 32x32
// multiply); the multiply-high of the general form is four quarter-rate
// multiplies, which bound the kernel when taken for every (task, variant)
template <bool MAGIC, bool D32>
__device__ __forceinline__ int64_t bd_scale(int64_t d, const ScaleEntry &se) {
    const uint64_t a = D32 ? (uint64_t)(uint32_t)d * (uint64_t)se.p : (uint64_t)d * (uint64_t)se.p;
    if (MAGIC && se.magic) return (int64_t)(__umul64hi(a, se.magic) >> se.shift);
    return (int64_t)(a >> se.shift);
}

// per-task arrays are kernel arguments marked restrict, so the compiler
// reads them with scalar loads (every lane of the workgroup needs the same
// task's fields)
template <bool MAGIC, bool D32>
__global__ __launch_bounds__(kBT) void k_bd_accum(const int64_t *__restrict__ m_ptr,
                                                  const int32_t *__restrict__ order,
                                                  const uint8_t *__restrict__ role,
                                                  const int64_t *__restrict__ dur,
                                                  const int64_t *__restrict__ gap,
                                                  const uint16_t *__restrict__ cls,
                                                  const int32_t *__restrict__ tprev, BdArgs a) {
    // XCD-aware: the workgroups of one XCD (b % 8) take consecutive
    // (variant block, chunk) pairs
    const int64_t total = (int64_t)a.nvb * a.nch;
    int64_t b = blockIdx.x;
    if ((total & 7) == 0) b = (int64_t)(blockIdx.x & 7) * (total >> 3) + (blockIdx.x >> 3);
    const int vb = (int)(b / a.nch), ch = (int)(b % a.nch);
    // kVL consecutive variants per lane: one removal word serves them all,
    // and the per-task work (order, class, duration, role) is shared
    const int64_t V = a.V, W = a.W;
    const int64_t vf = ((int64_t)vb * kBT + threadIdx.x) * kVL;
    bool ok[kVL];
    int64_t vc[kVL];
#pragma unroll
    for (int t = 0; t < kVL; t++) {
        ok[t] = vf + t < V;
        vc[t] = ok[t] ? vf + t : 0;
    }
    const int64_t vw = vc[0] >> 5;
    const uint32_t vsh = (uint32_t)(vc[0] & 31);     // kVL divides 32: one word
    const int64_t m = *m_ptr;
    const int64_t i0 = (int64_t)ch * kChunk;
    const int64_t i1 = i0 + kChunk < m ? i0 + kChunk : m;
    int64_t ksum[kVL], wsum[kVL];
    ScaleEntry se[kVL];
#pragma unroll
    for (int t = 0; t < kVL; t++) {
        ksum[t] = 0;
        wsum[t] = 0;
        se[t] = ScaleEntry{0ull, 1u, 0u};
    }
    int32_t ccls = -1;
    for (int64_t ib = i0; ib < i1; ib += kBatch) {
        // a batch of tasks: every load of a stage issued before any is used
        // (slots past the chunk's end read task 0 and are skipped)
        int64_t uu[kBatch];
        {   // one vector load brings the batch's task ids; lane j's goes to all
            const int j = (int)(threadIdx.x & (kBatch - 1));
            const int32_t mine = order[ib + j < i1 ? ib + j : i1 - 1];
#pragma unroll
            for (int t = 0; t < kBatch; t++) uu[t] = __builtin_amdgcn_readlane(mine, t);
        }
        int32_t cc[kBatch];
        int64_t dd[kBatch];
        uint32_t rr[kBatch], rw[kBatch];
#pragma unroll
        for (int j = 0; j < kBatch; j++) {
            cc[j] = cls[uu[j]];
            dd[j] = dur[uu[j]];
            rr[j] = role[uu[j]];
            rw[j] = a.rm[uu[j] * W + vw] >> vsh;
        }
#pragma unroll
        for (int j = 0; j < kBatch; j++) {
            if (ib + j >= i1) break;               // past the chunk's end (wave-uniform)
            if (cc[j] != ccls) {                   // wave-uniform: the class changed
#pragma unroll
                for (int t = 0; t < kVL; t++) se[t] = a.table[(int64_t)cc[j] * V + vc[t]];
                ccls = cc[j];
            }
            if (rr[j] != 1u) continue;             // waiting calls: k_bd_wait
#pragma unroll
            for (int t = 0; t < kVL; t++)
                ksum[t] += ((rw[j] >> t) & 1u) ? 0 : bd_scale<MAGIC, D32>(dd[j], se[t]);
        }
    }
#pragma unroll
    for (int t = 0; t < kVL; t++)
        if (ok[t] && ksum[t]) atomicAdd(&a.acc[vc[t]], (unsigned long long)ksum[t]);
}

// The waiting calls (a handful per iteration) as a list: one atomic per
// wave that holds any.
__global__ __launch_bounds__(kBT) void k_bd_wait_list(int64_t n, const uint8_t *__restrict__ role,
                                                      unsigned long long *__restrict__ wcount,
                                                      int32_t *__restrict__ wlist) {
    const int64_t u = (int64_t)blockIdx.x * kBT + threadIdx.x;
    const bool w = u < n && role[u] == 2u;
    const uint64_t bal = __ballot(w);
    if (!bal) return;
    const int lane = threadIdx.x & 63;
    const int first = __ffsll((unsigned long long)bal) - 1;
    unsigned long long base = 0;
    if (lane == first) base = atomicAdd(wcount, (unsigned long long)__popcll(bal));
    base = (unsigned long long)__shfl((long long)base, first, 64);
    if (w) wlist[base + __popcll(bal & ((1ull << lane) - 1ull))] = (int32_t)u;
}

// GPU-only time of every waiting call u and variant v: its start minus the
// moment its thread reached it.  Blocks along x cover the variants (one per
// thread, so every load and atomic is contiguous across the wave); blocks
// along y take the calls in turn.  Contributions are nonnegative integers,
// so the order of the atomics does not change the sums.
template <bool MAGIC, bool D32>
__global__ __launch_bounds__(kBT) void k_bd_wait(const unsigned long long *__restrict__ wcount,
                                                 const int32_t *__restrict__ wlist,
                                                 const int64_t *__restrict__ dur,
                                                 const int64_t *__restrict__ gap,
                                                 const uint16_t *__restrict__ cls,
                                                 const int32_t *__restrict__ tprev, BdArgs a) {
    const int64_t V = a.V, W = a.W;
    const int64_t v = (int64_t)blockIdx.x * kBT + threadIdx.x;
    if (v >= V) return;
    const int64_t cnt = (int64_t)*wcount;
    const int64_t vw = v >> 5;
    const uint32_t vb = (uint32_t)(v & 31);
    int64_t sum = 0;
    for (int64_t i = blockIdx.y; i < cnt; i += gridDim.y) {
        const int64_t u = wlist[i];
        const bool rmu = (a.rm[u * W + vw] >> vb) & 1u;
        const int64_t dp = rmu ? 0 : bd_scale<MAGIC, D32>(dur[u], a.table[(int64_t)cls[u] * V + v]);
        const int64_t start = a.finish[u * V + v] - dp;
        const int32_t p = tprev[u];
        int64_t reached = 0;
        if (p >= 0) {
            const bool rmp = (a.rm[(int64_t)p * W + vw] >> vb) & 1u;
            reached = a.finish[(int64_t)p * V + v] + (rmp ? 0 : gap[p]);
        }
        sum += start - reached;
    }
    if (sum) atomicAdd(&a.acc[V + v], (unsigned long long)sum);
}

__global__ __launch_bounds__(kBT) void k_bd_final(int32_t V, const int64_t *__restrict__ makespan,
                                                  const unsigned long long *__restrict__ acc,
                                                  int64_t *__restrict__ out) {
    const int64_t v = (int64_t)blockIdx.x * kBT + threadIdx.x;
    if (v >= V) return;
    const int64_t ms = makespan[v];
    const int64_t cpu_only = ms - (int64_t)acc[v];
    const int64_t gpu_only = (int64_t)acc[V + v];
    out[v * 4 + 0] = ms;
    out[v * 4 + 1] = cpu_only;
    out[v * 4 + 2] = gpu_only;
    out[v * 4 + 3] = ms - cpu_only - gpu_only;
}

}  // namespace

hipError_t launch_breakdown(const dd_graph *g, const dd_variants *var, const uint8_t *role_dev,
                            const int64_t *finish, const int64_t *makespan, int64_t *scratch,
                            int32_t *order, int64_t *out, hipStream_t s) {
    // scratch: [2][V] accumulators, [n_cls + 1] class counts / cursors, the
    // count of waiting calls; order: [n] tasks with a role by class, then
    // [n] waiting calls
    unsigned long long *acc = reinterpret_cast<unsigned long long *>(scratch);
    unsigned long long *hist = acc + 2 * (size_t)var->V;
    const int64_t C = var->n_cls;
    unsigned long long *wcount = hist + C + 1;
    int32_t *wlist = order + g->n;
    hipError_t e = hipMemsetAsync(scratch, 0, sizeof(int64_t) * (2 * (size_t)var->V + C + 2), s);
    if (e != hipSuccess) return e;
    const int64_t n = g->n;
    if (n > 0) {
        k_bd_count<<<grid_for(n, kBT), kBT, 0, s>>>(n, var->n_cls, role_dev, g->cls, hist);
        e = scan_exclusive(reinterpret_cast<int64_t *>(hist), reinterpret_cast<int64_t *>(hist),
                           C, s);
        if (e != hipSuccess) return e;
        k_bd_scatter<<<grid_for(n, kBT), kBT, 0, s>>>(n, var->n_cls, role_dev, g->cls, hist, order);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    // chunks cover n tasks (a bound known without a read-back); each
    // workgroup stops at the count of tasks with a role, hist[C], which the
    // scatter leaves in place (no task has class C)
    const int nvb = (var->V + kBT * kVL - 1) / (kBT * kVL);
    const int64_t nch64 = (n + kChunk - 1) / kChunk;
    if (n > 0) {
        BdArgs a{var->V, var->W, nvb, (int32_t)nch64, var->table, var->rm_bits, finish, acc};
        const unsigned grid = (unsigned)(nvb * nch64);
        const int64_t *mp = reinterpret_cast<const int64_t *>(hist + C);
        const bool d32 = g->dmax < (int64_t(1) << 32);
        // waiting calls: at most 64 blocks of calls per variant block
        const dim3 wg((unsigned)((var->V + kBT - 1) / kBT), 64u);
        k_bd_wait_list<<<grid_for(n, kBT), kBT, 0, s>>>(n, role_dev, wcount, wlist);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        if (var->any_magic && d32) {
            k_bd_accum<true, true><<<grid, kBT, 0, s>>>(mp, order, role_dev, g->dur, g->gap, g->cls, g->thread_prev, a);
            k_bd_wait<true, true><<<wg, kBT, 0, s>>>(wcount, wlist, g->dur, g->gap, g->cls, g->thread_prev, a);
        } else if (var->any_magic) {
            k_bd_accum<true, false><<<grid, kBT, 0, s>>>(mp, order, role_dev, g->dur, g->gap, g->cls, g->thread_prev, a);
            k_bd_wait<true, false><<<wg, kBT, 0, s>>>(wcount, wlist, g->dur, g->gap, g->cls, g->thread_prev, a);
        } else if (d32) {
            k_bd_accum<false, true><<<grid, kBT, 0, s>>>(mp, order, role_dev, g->dur, g->gap, g->cls, g->thread_prev, a);
            k_bd_wait<false, true><<<wg, kBT, 0, s>>>(wcount, wlist, g->dur, g->gap, g->cls, g->thread_prev, a);
        } else {
            k_bd_accum<false, false><<<grid, kBT, 0, s>>>(mp, order, role_dev, g->dur, g->gap, g->cls, g->thread_prev, a);
            k_bd_wait<false, false><<<wg, kBT, 0, s>>>(wcount, wlist, g->dur, g->gap, g->cls, g->thread_prev, a);
        }
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    k_bd_final<<<grid_for(var->V, kBT), kBT, 0, s>>>(var->V, makespan, acc, out);
    return hipGetLastError();
}

}  // namespace dd
