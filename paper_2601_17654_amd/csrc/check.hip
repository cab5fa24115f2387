// Input validation for the entry points that take cost tables or point sets.
//
// The partition cost model (Sections 2.1, 4.2, 4.5) and GetFrontier (Section 4.3) are
// defined for finite, non-negative times and powers.  A value is accepted iff x + 0.0
// is finite with a clear sign bit (so -0.0 counts as 0): in bits, the high word of
// x + 0.0 is below 0x7FF00000.  One pass, grid-stride, 16 bytes per lane and load; the
// verdict goes to a device status word, KR_OK unless some value fails.
#include <algorithm>

#include "kr_device.h"
#include "kr_launch.h"

namespace kr {

__global__ void check_init_kernel(int32_t *status)
{
    if (threadIdx.x == 0) *status = KR_OK;
}

__device__ __forceinline__ uint32_t high_word(double x) { return (uint32_t)(dbits(x + 0.0) >> 32); }

__global__ void __launch_bounds__(256) check_values_kernel(const double *x, int64_t n,
                                                           int32_t *status)
{
    // an 8-byte-aligned array starts with one lone value, then pairs of 16 bytes
    const int head = ((uintptr_t)x & 15) ? 1 : 0;
    const int64_t n2 = (n - head) / 2;
    typedef double f64x2 __attribute__((ext_vector_type(2)));
    const f64x2 *x2 = (const f64x2 *)(x + head);
    const int64_t stride = (int64_t)gridDim.x * 256;
    uint32_t worst = 0;  // largest high word seen
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n2; i += stride) {
        const f64x2 v = __builtin_nontemporal_load(x2 + i);
        worst = max(worst, max(high_word(v.x), high_word(v.y)));
    }
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        if (head) worst = max(worst, high_word(x[0]));
        if ((n - head) & 1) worst = max(worst, high_word(x[n - 1]));
    }
    if (__ballot(worst >= 0x7FF00000u) && (threadIdx.x & 63) == 0)
        __hip_atomic_store(status, (int32_t)KR_ENONFINITE, __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
}

// Launches the check of arrays xs[i] (n[i] doubles each, 8-byte aligned), writing the
// verdict to *status.
hipError_t launch_check(const double *const *xs, const int64_t *n, int count, int32_t *status,
                        hipStream_t st)
{
    hipLaunchKernelGGL(check_init_kernel, dim3(1), dim3(64), 0, st, status);
    for (int i = 0; i < count; ++i) {
        if (n[i] <= 0) continue;
        const int64_t blocks = std::min<int64_t>(2048, (n[i] / 2 + 255) / 256 + 1);
        hipLaunchKernelGGL(check_values_kernel, dim3((unsigned)blocks), dim3(256), 0, st, xs[i],
                           n[i], status);
    }
    return hipGetLastError();
}

}  // namespace kr
