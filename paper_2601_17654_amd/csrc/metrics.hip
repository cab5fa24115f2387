// Frontier comparison metrics of the evaluation (Section 6.1, "Metrics"): point set B
// against baseline point set A.  Every quantity is a minimum under a predicate, so each
// is exact and independent of the reduction order.  Three launches: per-block minima of
// the first pass (least time and energy of A, least time of B); per-block minima of the
// second pass, which needs the first pass's deadline d and budget b; one block that
// combines them and forms the reductions.
#include <math.h>

#include "kr_device.h"
#include "kr_launch.h"

namespace kr {

namespace {

struct CmpMin {
    __device__ __forceinline__ double operator()(double a, double b) const { return b < a ? b : a; }
};

constexpr int kP1 = 3;  // minT_A, minE_A, minT_B
constexpr int kP2 = 5;  // E_A(d), T_A(b), E_B at minT_B, E_B(d), T_B(b)

__device__ __forceinline__ double bmin(double v, double *lds)
{
    return block_reduce(v, (double)INFINITY, CmpMin(), lds);
}

__global__ void __launch_bounds__(KR_BLOCK) cmp_pass1_kernel(CmpArgs a)
{
    __shared__ double lds[KR_WAVES];
    const int64_t stride = (int64_t)gridDim.x * KR_BLOCK;
    double ta = INFINITY, ea = INFINITY, tb = INFINITY;
    for (int64_t i = (int64_t)blockIdx.x * KR_BLOCK + threadIdx.x; i < a.nA; i += stride) {
        ta = a.TA[i] < ta ? a.TA[i] : ta;
        ea = a.EA[i] < ea ? a.EA[i] : ea;
    }
    for (int64_t i = (int64_t)blockIdx.x * KR_BLOCK + threadIdx.x; i < a.nB; i += stride)
        tb = a.TB[i] < tb ? a.TB[i] : tb;
    ta = bmin(ta, lds);
    ea = bmin(ea, lds);
    tb = bmin(tb, lds);
    if (threadIdx.x == 0) {
        a.part[blockIdx.x * kP1 + 0] = ta;
        a.part[blockIdx.x * kP1 + 1] = ea;
        a.part[blockIdx.x * kP1 + 2] = tb;
    }
}

// The first pass's results, reduced redundantly by every block that needs them.
__device__ __forceinline__ void pass1_totals(const CmpArgs &a, double *lds, double *d, double *b,
                                             double *tb)
{
    double v[kP1] = {INFINITY, INFINITY, INFINITY};
    for (int j = threadIdx.x; j < a.blocks; j += KR_BLOCK)
        for (int k = 0; k < kP1; ++k) {
            const double x = a.part[j * kP1 + k];
            v[k] = x < v[k] ? x : v[k];
        }
    *d = bmin(v[0], lds);
    *b = bmin(v[1], lds);
    *tb = bmin(v[2], lds);
}

__global__ void __launch_bounds__(KR_BLOCK) cmp_pass2_kernel(CmpArgs a)
{
    __shared__ double lds[KR_WAVES];
    double d, b, tbl;
    pass1_totals(a, lds, &d, &b, &tbl);
    const int64_t stride = (int64_t)gridDim.x * KR_BLOCK;
    double v[kP2] = {INFINITY, INFINITY, INFINITY, INFINITY, INFINITY};
    for (int64_t i = (int64_t)blockIdx.x * KR_BLOCK + threadIdx.x; i < a.nA; i += stride) {
        const double t = a.TA[i], e = a.EA[i];
        if (t <= d && e < v[0]) v[0] = e;
        if (e <= b && t < v[1]) v[1] = t;
    }
    for (int64_t i = (int64_t)blockIdx.x * KR_BLOCK + threadIdx.x; i < a.nB; i += stride) {
        const double t = a.TB[i], e = a.EB[i];
        if (t == tbl && e < v[2]) v[2] = e;
        if (t <= d && e < v[3]) v[3] = e;
        if (e <= b && t < v[4]) v[4] = t;
    }
    for (int k = 0; k < kP2; ++k) {
        const double r = bmin(v[k], lds);
        if (threadIdx.x == 0) a.part2[blockIdx.x * kP2 + k] = r;
    }
}

__global__ void __launch_bounds__(KR_BLOCK) cmp_final_kernel(CmpArgs a)
{
    __shared__ double lds[KR_WAVES];
    double d, b, tbl;
    pass1_totals(a, lds, &d, &b, &tbl);
    double v[kP2] = {INFINITY, INFINITY, INFINITY, INFINITY, INFINITY};
    for (int j = threadIdx.x; j < a.blocks; j += KR_BLOCK)
        for (int k = 0; k < kP2; ++k) {
            const double x = a.part2[j * kP2 + k];
            v[k] = x < v[k] ? x : v[k];
        }
    for (int k = 0; k < kP2; ++k) v[k] = bmin(v[k], lds);
    if (threadIdx.x != 0) return;
    // A's leftmost point is (d, E_A(d)): its least time and the least energy there
    const double ea = v[0], ta = v[1], ebl = v[2];
    const double eb = v[3] == INFINITY ? NAN : v[3];
    const double tb = v[4] == INFINITY ? NAN : v[4];
    a.out[0] = (d - tbl) / d * 100.0;
    a.out[1] = (ea - ebl) / ea * 100.0;
    a.out[2] = (ea - eb) / ea * 100.0;
    a.out[3] = (ta - tb) / ta * 100.0;
    a.out[4] = d;
    a.out[5] = ea;
    a.out[6] = eb;
    a.out[7] = b;
    a.out[8] = ta;
    a.out[9] = tb;
}

}  // namespace

hipError_t launch_compare(const CmpArgs &a, hipStream_t st)
{
    hipLaunchKernelGGL(cmp_pass1_kernel, dim3(a.blocks), dim3(KR_BLOCK), 0, st, a);
    hipLaunchKernelGGL(cmp_pass2_kernel, dim3(a.blocks), dim3(KR_BLOCK), 0, st, a);
    hipLaunchKernelGGL(cmp_final_kernel, dim3(1), dim3(KR_BLOCK), 0, st, a);
    return hipGetLastError();
}

}  // namespace kr
