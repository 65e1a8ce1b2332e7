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

// ---------------------------------------------------------------------------
// Atomic-accumulation floor of a fused backward: the dQ traffic a single
// key-stationary kernel would need if it added each pair's dQ tile (64
// queries x D, fp32) into an fp32 accumulator with atomics, without any of
// the arithmetic.  One workgroup per key block walks its transposed list
// and adds 1.0 to every element of each listed query block's tile.
// ---------------------------------------------------------------------------
constexpr int ATOMIC_NT = 256;

__global__ __launch_bounds__(ATOMIC_NT) void dq_atomic_probe_kernel(const int32_t* __restrict__ kv_ptr,
                                                                    const int32_t* __restrict__ kv_idx,
                                                                    int64_t col_cap, float* __restrict__ acc,
                                                                    int Hq, int Hkv, int N, int D) {
    const int64_t krow = blockIdx.x;
    const int64_t bkv = krow / N;
    const int b = static_cast<int>(bkv / Hkv), hkv = static_cast<int>(bkv % Hkv);
    const int grp = Hq / Hkv;
    int64_t e0 = kv_ptr[krow], e1 = kv_ptr[krow + 1];
    e0 = e0 < 0 ? 0 : (e0 > col_cap ? col_cap : e0);
    e1 = e1 < e0 ? e0 : (e1 > col_cap ? col_cap : e1);
    const int64_t qrow0 = (static_cast<int64_t>(b) * Hq + hkv * grp) * N;
    const int tile = 64 * D;
    for (int64_t e = e0; e < e1; ++e) {
        const int ent = kv_idx[e];
        if (ent < 0 || ent / N >= grp) continue;
        float* dst = acc + (qrow0 + ent) * tile;
        for (int i = threadIdx.x; i < tile; i += ATOMIC_NT) unsafeAtomicAdd(dst + i, 1.0f);
    }
}

hipError_t launch_dq_atomic_probe(const int32_t* kv_ptr, const int32_t* kv_idx, int64_t col_cap, float* acc,
                                  int batch, int Hq, int Hkv, int N, int D, hipStream_t s) {
    const int64_t krows = static_cast<int64_t>(batch) * Hkv * N;
    if (krows == 0) return hipSuccess;
    hipLaunchKernelGGL(dq_atomic_probe_kernel, dim3(static_cast<unsigned>(krows)), dim3(ATOMIC_NT), 0, s, kv_ptr,
                       kv_idx, col_cap, acc, Hq, Hkv, N, D);
    return hipGetLastError();
}

}  // namespace vsa2
