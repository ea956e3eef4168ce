// Allocation-free variant of gpps_psi_stats: the workspace is a file-scope
// device array of GPPS_SCRATCH_BYTES instead of a caller buffer, for callers
// that cannot allocate device memory (code under HIP graph capture, serving
// loops, harnesses that forbid hipMalloc).
//
// In host code the array's name is a host-side stand-in, not a device address:
// its device address is taken once per device with hipGetSymbolAddress (with
// that device current) and kept; only that pointer is ever handed to kernels.
// Each device holds its own copy of the array until the process ends.  Every
// call on a device shares that device's copy: calls that may overlap on one
// device (other streams, other threads) race on it.  The kernels ignore the
// scratch contents on entry, so nothing needs clearing between calls.
#include <hip/hip_runtime.h>

#include <mutex>

#include "internal.h"

namespace {

constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[GPPS_SCRATCH_BYTES];

std::mutex g_mu;
void *g_ptr[kMaxDevices] = {};

// Device address of this device's scratch array (looked up on the first call
// on the device), or nullptr on a HIP error.
void *scratch_for_current_device() {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lk(g_mu);
    if (!g_ptr[dev]) {
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return nullptr;
        g_ptr[dev] = p;
    }
    return g_ptr[dev];
}

}  // namespace

extern "C" gpps_status gpps_psi_stats_noalloc(gpps_dtype dt, int64_t N, int64_t M, int64_t Q,
                                              const void *mu, const void *S, const void *Z,
                                              double sigma_f2, const double *l, void *psi0,
                                              void *Psi1, void *Psi2, int flags, void *stream) {
    // size checks come first, so that an oversized call fails before any HIP call
    const size_t need = gpps_workspace_bytes(dt, N, M, Q);
    if (need == 0)
        return (dt == GPPS_F32 || dt == GPPS_F64) ? GPPS_ERR_SHAPE : GPPS_ERR_DTYPE;
    if (need > (size_t)GPPS_SCRATCH_BYTES) return GPPS_ERR_WORKSPACE;
    void *ws = scratch_for_current_device();
    if (!ws) return GPPS_ERR_HIP;
    return gpps_psi_stats(dt, N, M, Q, mu, S, Z, sigma_f2, l, psi0, Psi1, Psi2, flags, ws,
                          (size_t)GPPS_SCRATCH_BYTES, stream);
}
