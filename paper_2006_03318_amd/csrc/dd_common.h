// Device helpers shared by the dd kernels (wave64 / CDNA4).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dd {

__device__ __forceinline__ int64_t shfl_up64(int64_t x, int d) {
    int lo = __shfl_up((int)(uint32_t)(uint64_t)x, d, 64);
    int hi = __shfl_up((int)(uint32_t)((uint64_t)x >> 32), d, 64);
    return (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}

__device__ __forceinline__ int64_t shfl_xor64(int64_t x, int d) {
    int lo = __shfl_xor((int)(uint32_t)(uint64_t)x, d, 64);
    int hi = __shfl_xor((int)(uint32_t)((uint64_t)x >> 32), d, 64);
    return (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}

__device__ __forceinline__ int64_t wave_sum64(int64_t x) {
    for (int o = 32; o > 0; o >>= 1) x += shfl_xor64(x, o);
    return x;
}

__device__ __forceinline__ int64_t wave_max64(int64_t x) {
    for (int o = 32; o > 0; o >>= 1) {
        int64_t y = shfl_xor64(x, o);
        x = y > x ? y : x;
    }
    return x;
}

// Exclusive scan of one int64 per thread across a block of BS threads
// (BS a multiple of 64, <= 1024).  Returns the exclusive prefix; *total gets
// the block sum.  Every thread of the block must call it.
template <int BS>
__device__ int64_t block_excl_scan(int64_t x, int64_t *total) {
    static_assert(BS % 64 == 0 && BS <= 1024, "block size");
    constexpr int NW = BS / 64;
    __shared__ int64_t wpart[NW];
    __shared__ int64_t wtot;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    int64_t incl = x;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        int64_t y = shfl_up64(incl, o);
        if (lane >= o) incl += y;
    }
    if (lane == 63) wpart[w] = incl;
    __syncthreads();
    if (w == 0) {
        int64_t v = lane < NW ? wpart[lane] : 0;
        int64_t in2 = v;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            int64_t y = shfl_up64(in2, o);
            if (lane >= o) in2 += y;
        }
        if (lane < NW) wpart[lane] = in2 - v;
        if (lane == NW - 1) wtot = in2;
    }
    __syncthreads();
    int64_t r = incl - x + wpart[w];
    *total = wtot;
    __syncthreads();
    return r;
}

// Load that bypasses the per-CU cache (reads the device-coherent value).
template <class T>
__device__ __forceinline__ T load_coherent(const T *p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Atomics on one word that every wave of a launch updates: the atomic is
// skipped when the word (read device-coherently) already covers the value.
// The word only grows, so a skip never loses an update, and a launch of
// thousands of waves does not queue on that word.
__device__ __forceinline__ void atomic_max_hot(unsigned long long *p, unsigned long long v) {
    if (v > load_coherent(p)) atomicMax(p, v);
}
__device__ __forceinline__ void atomic_or_hot(unsigned long long *p, unsigned long long v) {
    if (v & ~load_coherent(p)) atomicOr(p, v);
}
__device__ __forceinline__ void atomic_or_hot(uint32_t *p, uint32_t v) {
    if (v & ~load_coherent(p)) atomicOr(p, v);
}

}  // namespace dd
