// Wave-level helpers on doubles (gfx950, wave64): one-instruction minimum and DPP wave
// minima.
#pragma once

#include "kr_device.h"

namespace kr {

// Minimum of two non-NaN doubles in one instruction (the compiler's fmin adds operand
// canonicalisation it cannot prove unnecessary here).
__device__ __forceinline__ double vmin(double a, double b)
{
    double r;
    asm("v_min_f64 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
    return r;
}

// One DPP step of a wave minimum over doubles (rows not written keep their own value).
template <int CTRL, int ROWS>
__device__ __forceinline__ double dpp_min_f64(double x)
{
    const uint64_t b = dbits(x);
    const uint32_t lo = (uint32_t)b, hi = (uint32_t)(b >> 32);
    uint32_t ylo, yhi;
    if constexpr (ROWS == 0xF) {  // every lane reads a lane of its own row
        ylo = __builtin_amdgcn_mov_dpp(lo, CTRL, 0xF, 0xF, false);
        yhi = __builtin_amdgcn_mov_dpp(hi, CTRL, 0xF, 0xF, false);
    } else {  // rows outside ROWS keep their own value
        ylo = __builtin_amdgcn_update_dpp(lo, lo, CTRL, ROWS, 0xF, false);
        yhi = __builtin_amdgcn_update_dpp(hi, hi, CTRL, ROWS, 0xF, false);
    }
    return vmin(bitsd(((uint64_t)yhi << 32) | ylo), x);
}

// Minima over the wave of two non-NaN doubles (same DPP pattern as wave_min_u64: pairs,
// quads, half rows, rows, then row broadcasts into rows 1-3), interleaved; results
// uniform.  Every lane must be active.
__device__ __forceinline__ void wave_min2_f64(double &x, double &y)
{
    x = dpp_min_f64<0xB1, 0xF>(x);
    y = dpp_min_f64<0xB1, 0xF>(y);
    x = dpp_min_f64<0x4E, 0xF>(x);
    y = dpp_min_f64<0x4E, 0xF>(y);
    x = dpp_min_f64<0x141, 0xF>(x);
    y = dpp_min_f64<0x141, 0xF>(y);
    x = dpp_min_f64<0x140, 0xF>(x);
    y = dpp_min_f64<0x140, 0xF>(y);
    x = dpp_min_f64<0x142, 0xA>(x);
    y = dpp_min_f64<0x142, 0xA>(y);
    x = dpp_min_f64<0x143, 0xC>(x);
    y = dpp_min_f64<0x143, 0xC>(y);
    x = bitsd(lane_u64(dbits(x), 63));
    y = bitsd(lane_u64(dbits(y), 63));
}

// Position of this lane among the set lanes of m below it.
__device__ __forceinline__ int lane_rank(uint64_t m)
{
    return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                          __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0));
}

}  // namespace kr
