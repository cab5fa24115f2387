// Device-side helpers shared by the library's kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/kareus.h"

#define KR_BLOCK 256
#define KR_WAVES (KR_BLOCK / 64)
#define KR_INF_BITS 0x7FF0000000000000ull

namespace kr {

// Positive finite doubles order like their bit patterns; +inf is above all of them.
__device__ __forceinline__ uint64_t dbits(double x) { return (uint64_t)__double_as_longlong(x); }
__device__ __forceinline__ double bitsd(uint64_t b) { return __longlong_as_double((long long)b); }

// Lexicographic (T, E, idx) order on bit patterns.
__device__ __forceinline__ bool key_less(uint64_t ta, uint64_t ea, int32_t ia, uint64_t tb,
                                         uint64_t eb, int32_t ib)
{
    if (ta != tb) return ta < tb;
    if (ea != eb) return ea < eb;
    return ia < ib;
}

struct MinU64 {
    __device__ __forceinline__ uint64_t operator()(uint64_t a, uint64_t b) const { return a < b ? a : b; }
};
struct MaxU64 {
    __device__ __forceinline__ uint64_t operator()(uint64_t a, uint64_t b) const { return a > b ? a : b; }
};
struct SumI32 {
    __device__ __forceinline__ int32_t operator()(int32_t a, int32_t b) const { return a + b; }
};
struct SumI64 {
    __device__ __forceinline__ int64_t operator()(int64_t a, int64_t b) const { return a + b; }
};

template <typename T>
__device__ __forceinline__ T shfl_up(T v, int d)
{
    return __shfl_up(v, d, 64);
}

// Inclusive scan within a wave64.
template <typename T, typename Op>
__device__ __forceinline__ T wave_inclusive(T x, Op op)
{
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        T y = shfl_up(x, d);
        if (lane >= d) x = op(x, y);
    }
    return x;
}

// Exclusive block scan (blockDim.x == KR_BLOCK).  `lds` holds KR_WAVES values.
// Returns the exclusive prefix; *total receives the block aggregate.  Contains two
// barriers; every thread of the block must call it.
template <typename T, typename Op>
__device__ __forceinline__ T block_exclusive(T v, T identity, Op op, T *lds, T *total)
{
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    T inc = wave_inclusive(v, op);
    if (lane == 63) lds[wave] = inc;
    __syncthreads();
    T before = identity, all = identity;
#pragma unroll
    for (int w = 0; w < KR_WAVES; ++w) {
        T s = lds[w];
        if (w < wave) before = op(before, s);
        all = op(all, s);
    }
    T ex = shfl_up(inc, 1);
    if (lane == 0) ex = identity;
    __syncthreads();
    *total = all;
    return op(before, ex);
}

template <typename T, typename Op>
__device__ __forceinline__ T block_reduce(T v, T identity, Op op, T *lds)
{
    T total;
    block_exclusive(v, identity, op, lds, &total);
    return total;
}

}  // namespace kr
