// Allocation-free GetFrontier (Section 4.3): kr_pareto_filter with its workspace in a
// fixed device array instead of a caller-supplied buffer, for callers that cannot
// allocate device memory (code under HIP graph capture, tight serving loops).
//
// The array lives in this file as a static __device__ variable, so each device the
// library runs on holds one copy until the process ends.  In host code its name is only
// a host-side stand-in; the device address of a device's copy comes from
// hipGetSymbolAddress, asked once per device (with that device current) on the entry
// point's first call there, and only that address is handed to kernels.
#include <mutex>

#include "../../include/kareus.h"
#include "kr_launch.h"

namespace {

// >= kr_pareto_filter_workspace(KR_NOALLOC_MAX_POINTS, KR_NOALLOC_MAX_SEGS); checked when
// a device's address is first taken.
constexpr size_t kScratchBytes = (size_t)KR_NOALLOC_SCRATCH_MIB << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};

// Device address of the current device's scratch array, or nullptr on a HIP error.
void *scratch_address()
{
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        if (kr_pareto_filter_workspace(KR_NOALLOC_MAX_POINTS, KR_NOALLOC_MAX_SEGS) > kScratchBytes)
            return nullptr;
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return nullptr;
        g_scratch_ptr[dev] = p;
    }
    return g_scratch_ptr[dev];
}

}  // namespace

extern "C" kr_status kr_pareto_filter_noalloc(int64_t n_total, const double *T, const double *E,
                                              const int64_t *seg_off, int32_t n_seg, int64_t cap,
                                              int64_t *out_off, int32_t *out_idx, double *out_T,
                                              double *out_E, int32_t *status_out, void *stream)
{
    if (n_total < 0 || n_seg < 0) return KR_EINVAL;
    if (n_total > KR_NOALLOC_MAX_POINTS || n_seg > KR_NOALLOC_MAX_SEGS) return KR_ECAPACITY;
    void *ws = scratch_address();
    if (!ws) return KR_EHIP;
    return kr_pareto_filter(n_total, T, E, seg_off, n_seg, cap, out_off, out_idx, out_T, out_E,
                            status_out, ws, kScratchBytes, stream);
}
