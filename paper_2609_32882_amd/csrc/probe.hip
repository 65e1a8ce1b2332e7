// Dense MFMA rate probe, the measured counterpart of the bf16 dense peak the
// attention kernels are rated against: every CU runs 16 waves (4 per SIMD),
// each issuing independent chains of 32x32x16 bf16 MFMAs with operands in
// registers, so the matrix cores never wait on memory or on a dependency.
#include "common.hpp"
#include "internal.hpp"

namespace vsa2 {

constexpr int PROBE_NT = 1024;   // 16 waves per workgroup, one workgroup per CU
constexpr int PROBE_CHAINS = 4;  // independent accumulators per wave

__global__ __launch_bounds__(PROBE_NT) void mfma_peak_kernel(float* __restrict__ sink, int iters) {
    bf16x8_t a, b;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        a[i] = static_cast<__bf16>(1.0f + 1e-3f * static_cast<float>((threadIdx.x + i) & 7));
        b[i] = static_cast<__bf16>(1e-3f * static_cast<float>(i));
    }
    f32x16_t c[PROBE_CHAINS];
#pragma unroll
    for (int j = 0; j < PROBE_CHAINS; ++j)
#pragma unroll
        for (int i = 0; i < 16; ++i) c[j][i] = 0.f;
    for (int it = 0; it < iters; ++it)
#pragma unroll
        for (int j = 0; j < PROBE_CHAINS; ++j) c[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c[j], 0, 0, 0);
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < PROBE_CHAINS; ++j)
#pragma unroll
        for (int i = 0; i < 16; ++i) s += c[j][i];
    // a store no value reaches in practice keeps every chain alive
    if (s == -1.0f) sink[0] = s;
}

hipError_t launch_mfma_peak(int iters, float* sink, int64_t* flops, hipStream_t s) {
    int dev = 0, cus = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    *flops = static_cast<int64_t>(cus) * (PROBE_NT / 64) * PROBE_CHAINS * static_cast<int64_t>(iters) *
             (2LL * 32 * 32 * 16);
    if (iters == 0) return hipSuccess;
    hipLaunchKernelGGL(mfma_peak_kernel, dim3(static_cast<unsigned>(cus)), dim3(PROBE_NT), 0, s, sink, iters);
    return hipGetLastError();
}

}  // namespace vsa2
