// Work order of the attention kernels: longest rows first within each XCD.
//
// The attention kernels run one workgroup per block-list row (a CSR row for
// the forward and dQ, a CSC row for dK/dV), and the hardware dispatcher
// hands workgroups to each XCD in grid order, refilling a slot as soon as a
// workgroup finishes: it is an in-order work queue per XCD.  Putting the
// longest rows at the front of each XCD's range makes that queue a
// longest-processing-time-first schedule, so the last workgroups to start
// are short and the tail of the launch stays short when row lengths vary
// (mass selection; key in-degrees).  The ranges themselves are the ones
// xcd_item gives each XCD, so the rows of an XCD (and the heads whose tiles
// its L2 holds) do not change.
//
// Rows are grouped into 32 length classes, class = len * 32 / (max_len + 1),
// heaviest class first and row order inside a class (a stable, deterministic
// counting sort).  Rows of equal length (top-k) keep their order.
#include "common.hpp"
#include "internal.hpp"

namespace vsa2 {

constexpr int PLAN_NT = 256;
constexpr int PLAN_CLASSES = 32;

__device__ __forceinline__ int64_t row_len(const int32_t* ptr, int64_t row, int64_t cap) {
    int64_t a = ptr[row], b = ptr[row + 1];
    a = a < 0 ? 0 : (a > cap ? cap : a);
    b = b < a ? a : (b > cap ? cap : b);
    return b - a;
}

// One workgroup per XCD range x (8 workgroups).  Thread t owns the
// contiguous rows [beg + t*per, beg + min((t+1)*per, len)) of the range.
__global__ __launch_bounds__(PLAN_NT) void lpt_order_kernel(const int32_t* __restrict__ ptr, int64_t nrows,
                                                            int64_t cap, int32_t* __restrict__ order) {
    __shared__ uint32_t hist[PLAN_CLASSES][PLAN_NT];
    __shared__ uint32_t part[PLAN_NT];
    __shared__ int64_t red[PLAN_NT / 64];
    const int t = threadIdx.x;
    const int64_t x = blockIdx.x;
    const int64_t q = nrows >> 3, r = nrows & 7;
    const int64_t beg = x * q + (x < r ? x : r);
    const int64_t len = q + (x < r ? 1 : 0);
    const int64_t per = (len + PLAN_NT - 1) / PLAN_NT;
    const int64_t i0 = t * per < len ? t * per : len;
    const int64_t i1 = (t + 1) * per < len ? (t + 1) * per : len;

    // longest row of the range
    int64_t mx = 0;
    for (int64_t i = i0; i < i1; ++i) {
        const int64_t c = row_len(ptr, beg + i, cap);
        mx = c > mx ? c : mx;
    }
    for (int off = 32; off >= 1; off >>= 1) {
        const int64_t o = __shfl_xor(mx, off, 64);
        mx = o > mx ? o : mx;
    }
    if ((t & 63) == 0) red[t >> 6] = mx;
    __syncthreads();
    mx = red[0];
#pragma unroll
    for (int w = 1; w < PLAN_NT / 64; ++w) mx = red[w] > mx ? red[w] : mx;
    auto cls_of = [&](int64_t c) -> int {   // 0 = heaviest class
        return PLAN_CLASSES - 1 - static_cast<int>(c * PLAN_CLASSES / (mx + 1));
    };

    // per-thread class histogram
#pragma unroll
    for (int c = 0; c < PLAN_CLASSES; ++c) hist[c][t] = 0;
    for (int64_t i = i0; i < i1; ++i) hist[cls_of(row_len(ptr, beg + i, cap))][t] += 1;
    __syncthreads();

    // exclusive scan over (class, thread) in that order: thread t scans the
    // 32 consecutive slots k = 32t .. 32t+31 of the flattened [class][thread]
    // array, then the 256 partial sums are scanned
    uint32_t* flat = &hist[0][0];
    uint32_t sum = 0;
#pragma unroll
    for (int j = 0; j < PLAN_CLASSES; ++j) sum += flat[t * PLAN_CLASSES + j];
    part[t] = sum;
    __syncthreads();
    for (int off = 1; off < PLAN_NT; off <<= 1) {
        const uint32_t v = t >= off ? part[t - off] : 0u;
        __syncthreads();
        part[t] += v;
        __syncthreads();
    }
    uint32_t run = part[t] - sum;   // exclusive
#pragma unroll
    for (int j = 0; j < PLAN_CLASSES; ++j) {
        const uint32_t v = flat[t * PLAN_CLASSES + j];
        flat[t * PLAN_CLASSES + j] = run;
        run += v;
    }
    __syncthreads();

    // stable scatter: the thread's rows in order, each after the earlier
    // rows of its class
    for (int64_t i = i0; i < i1; ++i) {
        const int c = cls_of(row_len(ptr, beg + i, cap));
        const uint32_t pos = hist[c][t]++;
        order[beg + pos] = static_cast<int32_t>(beg + i);
    }
}

hipError_t launch_lpt_order(const int32_t* ptr, int64_t nrows, int64_t cap, int32_t* order, hipStream_t s) {
    if (nrows <= 0) return hipSuccess;
    hipLaunchKernelGGL(lpt_order_kernel, dim3(8), dim3(PLAN_NT), 0, s, ptr, nrows, cap, order);
    return hipGetLastError();
}

}  // namespace vsa2
