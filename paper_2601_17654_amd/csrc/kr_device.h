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

// Barrier for LDS traffic only: unlike __syncthreads() it does not wait for
// outstanding global loads, so register prefetches stay in flight across it.
__device__ __forceinline__ void lds_barrier()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Value of a uniform-indexed lane.
__device__ __forceinline__ uint64_t lane_u64(uint64_t x, int lane)
{
    const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)x, lane);
    const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)(x >> 32), lane);
    return ((uint64_t)hi << 32) | lo;
}
__device__ __forceinline__ int32_t lane_i32(int32_t x, int lane)
{
    return __builtin_amdgcn_readlane(x, lane);
}

// One DPP step of a wave minimum over unsigned 64-bit values.
template <int CTRL, int ROWS>
__device__ __forceinline__ uint64_t dpp_min_u64(uint64_t x)
{
    const uint32_t lo = (uint32_t)x, hi = (uint32_t)(x >> 32);
    const uint32_t ylo = __builtin_amdgcn_update_dpp(lo, lo, CTRL, ROWS, 0xF, false);
    const uint32_t yhi = __builtin_amdgcn_update_dpp(hi, hi, CTRL, ROWS, 0xF, false);
    const uint64_t y = ((uint64_t)yhi << 32) | ylo;
    return y < x ? y : x;
}

// Minimum over a full wave64 (all lanes active), uniform result: pairs, quads, half
// rows and rows by DPP permutes, then rows 0-1 and 0-3 by row broadcasts; lane 63
// ends up holding the minimum.
__device__ __forceinline__ uint64_t wave_min_u64(uint64_t x)
{
    x = dpp_min_u64<0xB1, 0xF>(x);   // quad_perm [1,0,3,2]
    x = dpp_min_u64<0x4E, 0xF>(x);   // quad_perm [2,3,0,1]
    x = dpp_min_u64<0x141, 0xF>(x);  // row_half_mirror
    x = dpp_min_u64<0x140, 0xF>(x);  // row_mirror
    x = dpp_min_u64<0x142, 0xA>(x);  // row_bcast:15 into rows 1 and 3
    x = dpp_min_u64<0x143, 0xC>(x);  // row_bcast:31 into rows 2 and 3
    return lane_u64(x, 63);
}

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

// Exclusive block scan (blockDim.x == 64 * NW, KR_BLOCK by default).  `lds` holds NW
// values.  Returns the exclusive prefix; *total receives the block aggregate.  Contains
// two barriers; every thread of the block must call it.
template <typename T, typename Op, int NW = KR_WAVES>
__device__ __forceinline__ T block_exclusive(T v, T identity, Op op, T *lds, T *total)
{
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    T inc = wave_inclusive(v, op);
    if (lane == 63) lds[wave] = inc;
    __syncthreads();
    T before = identity, all = identity;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
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
