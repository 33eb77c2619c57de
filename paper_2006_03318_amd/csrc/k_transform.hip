// Per-(class, variant) shrink/scale table (Sec. 4.4, "shrink/scale"
// primitive; the AMP recipe of Sec. 5.1 divides durations by 3 or 2).
//
// A scaled duration is floor(d * p / q) in integer nanoseconds.  To keep the
// simulation kernel free of 64-bit division, each (p, q) becomes a
// multiply-shift:  q = 2^k  ->  (d*p) >> k;  otherwise, with l = ceil(log2 q)
// and m = ceil(2^(62+l) / q),  floor(a / q) = floor(a * m / 2^(62+l)) for
// every a < 2^62 (Granlund & Montgomery, "Division by invariant integers
// using multiplication", PLDI 1994, Thm. 4.2 with N = 62); the load-time
// range check guarantees d * p < 2^62.

#include "dd_common.h"
#include "dd_internal.h"

namespace dd {
namespace {

constexpr int kBS = 256;

__device__ uint32_t ceil_log2(uint32_t q) {
    uint32_t l = 0;
    while ((1u << l) < q) l++;
    return l;
}

constexpr int kTabBlocks = 512;   // grid-stride blocks: one set of atomics per block

__global__ __launch_bounds__(kBS) void k_scale_table(const dd_ratio *__restrict__ in, int64_t count,
                                                     ScaleEntry *__restrict__ out,
                                                     uint32_t *__restrict__ err,
                                                     unsigned long long *__restrict__ pmax,
                                                     unsigned long long *__restrict__ rmax_bits) {
    uint32_t e = 0, mg = 0;
    int64_t pm = 0;
    int64_t rb = 0;
    for (int64_t i = (int64_t)blockIdx.x * kBS + threadIdx.x; i < count;
         i += (int64_t)gridDim.x * kBS) {
        int32_t p = 1, q = 1;
        if (in) { p = in[i].p; q = in[i].q; }
        ScaleEntry se{0ull, 0u, 0u};
        if (p < 0 || q < 1) {
            e |= ERR_SCALE;
        } else {
            se.p = (uint32_t)p;
            const uint32_t uq = (uint32_t)q;
            const uint32_t l = ceil_log2(uq);
            if ((uq & (uq - 1)) == 0) {
                se.shift = l;                       // power of two
            } else {
                // m = floor(2^(62+l) / q) + 1 by long division in base 2^32:
                // 2^(62+l) = hi * 2^64 with hi = 2^(l-2) < q (l >= 2 here)
                uint64_t r = 1ull << (l - 2);
                uint64_t t = r << 32;
                const uint64_t d1 = t / uq;
                r = t % uq;
                t = r << 32;
                const uint64_t d0 = t / uq;
                se.magic = ((d1 << 32) | d0) + 1;  // q is not a power of two: remainder != 0
                se.shift = l - 2;
                mg = 1;
            }
            pm = p > pm ? p : pm;
            const double ratio = (double)p / (double)q;
            const int64_t b = (int64_t)__double_as_longlong(ratio);   // order-preserving for ratio >= 0
            rb = b > rb ? b : rb;
        }
        out[i] = se;
    }
    // wave, then the block's waves through LDS: one set of atomics per block
    pm = wave_max64(pm);
    rb = wave_max64(rb);
    for (int o = 32; o > 0; o >>= 1) {
        e |= (uint32_t)__shfl_xor((int)e, o, 64);
        mg |= (uint32_t)__shfl_xor((int)mg, o, 64);
    }
    constexpr int NW = kBS / 64;
    __shared__ int64_t red[4][NW];
    const int w = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) {
        red[0][w] = pm; red[1][w] = rb; red[2][w] = e; red[3][w] = mg;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int k = 1; k < NW; k++) {
            pm = red[0][k] > pm ? red[0][k] : pm;
            rb = red[1][k] > rb ? red[1][k] : rb;
            e |= (uint32_t)red[2][k];
            mg |= (uint32_t)red[3][k];
        }
        atomic_or_hot(err, e);
        atomic_or_hot(err + 1, mg);
        atomic_max_hot(pmax, (unsigned long long)pm);
        atomic_max_hot(rmax_bits, (unsigned long long)rb);
    }
}

}  // namespace

hipError_t launch_build_scale_table(const dd_ratio *scale_dev, int32_t n_cls, int32_t V,
                                    ScaleEntry *table, uint32_t *err, hipStream_t s) {
    // err[0] = error bits, err[1] = some q is not a power of two, err[2..3] = pmax,
    // err[4..5] = max ratio bits (caller-zeroed)
    const int64_t count = (int64_t)n_cls * V;
    unsigned long long *pmax = reinterpret_cast<unsigned long long *>(err + 2);
    unsigned long long *rmax = reinterpret_cast<unsigned long long *>(err + 4);
    const int64_t nb = grid_for(count, kBS);
    if (count > 0)
        k_scale_table<<<(unsigned)(nb < kTabBlocks ? nb : kTabBlocks), kBS, 0, s>>>(scale_dev, count, table,
                                                                                   err, pmax, rmax);
    return hipGetLastError();
}

}  // namespace dd
