// Unit-rate probes for the measurement harness: the sustained issue rates of the
// three units the psi-statistic kernels spend their time in (vector fp32 FMA,
// v_exp_f32, and the 32x32x16 f16 matrix instruction), measured on the device
// at its running clock.  Each probe is a fixed number of independent dependency
// chains per lane in a grid of several waves per SIMD, so that issue, not
// latency, bounds it; results go to a caller-provided sink so that nothing is
// optimised away.
#include <hip/hip_runtime.h>

#include "internal.h"

namespace gpps {
namespace {

typedef float v16f __attribute__((ext_vector_type(16)));
typedef _Float16 v8h __attribute__((ext_vector_type(8)));

constexpr int kChains = 8;
constexpr int kBlocks = 2048;   // 8 workgroups of 4 waves per compute unit
constexpr int kThreads = 256;

__global__ __launch_bounds__(kThreads) void probe_fma_kernel(int iters, float *__restrict__ sink) {
    float a[kChains];
#pragma unroll
    for (int k = 0; k < kChains; ++k) a[k] = 1e-3f * threadIdx.x + k;
    for (int i = 0; i < iters; ++i) {
#pragma unroll
        for (int k = 0; k < kChains; ++k) a[k] = fmaf(a[k], 0.9999f, 1e-4f);
    }
    float s = 0.f;
#pragma unroll
    for (int k = 0; k < kChains; ++k) s += a[k];
    sink[blockIdx.x * kThreads + threadIdx.x] = s;
}

__global__ __launch_bounds__(kThreads) void probe_exp_kernel(int iters, float *__restrict__ sink) {
    float a[kChains];
#pragma unroll
    for (int k = 0; k < kChains; ++k) a[k] = 1e-4f * threadIdx.x + 0.1f * k;
    for (int i = 0; i < iters; ++i) {
#pragma unroll
        for (int k = 0; k < kChains; ++k) a[k] = __builtin_amdgcn_exp2f(-a[k]);  // stays in (0, 1]
    }
    float s = 0.f;
#pragma unroll
    for (int k = 0; k < kChains; ++k) s += a[k];
    sink[blockIdx.x * kThreads + threadIdx.x] = s;
}

__global__ __launch_bounds__(kThreads) void probe_mfma_kernel(int iters, float *__restrict__ sink) {
    v8h A, B;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        A[e] = (_Float16)(1e-3f * (threadIdx.x & 63) + e);
        B[e] = (_Float16)(1e-3f);
    }
    v16f acc[4];
#pragma unroll
    for (int k = 0; k < 4; ++k)
#pragma unroll
        for (int t = 0; t < 16; ++t) acc[k][t] = 0.f;
    for (int i = 0; i < iters; ++i) {
#pragma unroll
        for (int k = 0; k < 4; ++k) acc[k] = __builtin_amdgcn_mfma_f32_32x32x16_f16(A, B, acc[k], 0, 0, 0);
    }
    float s = 0.f;
#pragma unroll
    for (int k = 0; k < 4; ++k)
#pragma unroll
        for (int t = 0; t < 16; ++t) s += acc[k][t];
    sink[blockIdx.x * kThreads + threadIdx.x] = s;
}

template <typename K>
hipError_t timed(K kernel, int iters, float *sink, hipStream_t st, float &ms) {
    hipEvent_t a, b;
    hipError_t e = hipEventCreate(&a);
    if (e != hipSuccess) return e;
    if ((e = hipEventCreate(&b)) != hipSuccess) {
        (void)hipEventDestroy(a);
        return e;
    }
    kernel<<<kBlocks, kThreads, 0, st>>>(iters / 8, sink);   // warm-up
    (void)hipEventRecord(a, st);
    kernel<<<kBlocks, kThreads, 0, st>>>(iters, sink);
    (void)hipEventRecord(b, st);
    e = hipGetLastError();
    if (e == hipSuccess) e = hipEventSynchronize(b);
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, a, b);
    (void)hipEventDestroy(a);
    (void)hipEventDestroy(b);
    return e;
}

}  // namespace
}  // namespace gpps

extern "C" {

size_t gpps_probe_sink_bytes(void) { return sizeof(float) * gpps::kBlocks * gpps::kThreads; }

gpps_status gpps_probe_unit_rates(void *sink, size_t sink_bytes, double *rates, void *stream) {
    using namespace gpps;
    if (!sink || !rates) return GPPS_ERR_NULL;
    if (sink_bytes < gpps_probe_sink_bytes()) return GPPS_ERR_WORKSPACE;
    hipStream_t st = static_cast<hipStream_t>(stream);
    float *s = static_cast<float *>(sink);
    const double lanes = double(kBlocks) * kThreads;
    const int it_fma = 4096, it_exp = 2048, it_mfma = 1024;
    float ms = 0.f;
    if (timed(probe_fma_kernel, it_fma, s, st, ms) != hipSuccess) return GPPS_ERR_HIP;
    rates[0] = 2.0 * lanes * kChains * it_fma / (ms * 1e-3);        // fp32 flops/s (FMA = 2)
    if (timed(probe_exp_kernel, it_exp, s, st, ms) != hipSuccess) return GPPS_ERR_HIP;
    rates[1] = lanes * kChains * it_exp / (ms * 1e-3);               // exponentials/s
    if (timed(probe_mfma_kernel, it_mfma, s, st, ms) != hipSuccess) return GPPS_ERR_HIP;
    rates[2] = (lanes / 64.0) * 4.0 * it_mfma * (2.0 * 32 * 32 * 16) / (ms * 1e-3);  // f16 flops/s
    return GPPS_OK;
}

}  // extern "C"
