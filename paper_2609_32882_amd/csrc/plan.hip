// Work order of the attention kernels: longest rows first within each XCD.
//
// The attention kernels run one workgroup per block-list row (a CSR row for
// the forward and dQ, a CSC row for dK/dV), and the hardware dispatcher
// hands workgroups to each XCD in grid order, refilling a slot as soon as a
// workgroup finishes: it is an in-order work queue per XCD.  Putting the
// longest rows first makes that queue a longest-processing-time-first
// schedule, so the last workgroups to start are short and the tail of the
// launch stays short when row lengths vary (mass selection; key
// in-degrees).  The rows are reordered only inside each segment where an
// XCD's range (the rows xcd_item gives it) meets one head's N rows: the
// rows of an XCD do not change, and workgroups resident together keep
// working on one head, whose tiles its L2 holds (sorting a whole XCD range
// mixes its heads and, measured at 720p, raised the dK/dV kernel's L2 miss
// share from 74% to 89%).
//
// Rows are grouped into 32 length classes, class = len * 32 / (max_len + 1)
// over the segment, heaviest class first and row order inside a class (a
// stable, deterministic counting sort).  Rows of equal length (top-k) keep
// their order.
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

// Longest-first order of the rows [beg, beg + len), written at the same
// positions of order[].  Thread t owns the contiguous rows
// [beg + t*per, beg + min((t+1)*per, len)).
__device__ void lpt_segment(const int32_t* __restrict__ ptr, int64_t cap, int32_t* __restrict__ order, int64_t beg,
                            int64_t len, uint32_t (*hist)[PLAN_NT], uint32_t* part, int64_t* red) {
    const int t = threadIdx.x;
    const int64_t per = (len + PLAN_NT - 1) / PLAN_NT;
    const int64_t i0 = t * per < len ? t * per : len;
    const int64_t i1 = (t + 1) * per < len ? (t + 1) * per : len;

    // longest row of the segment
    int64_t mx = 0;
    for (int64_t i = i0; i < i1; ++i) {
        const int64_t c = row_len(ptr, beg + i, cap);
        mx = c > mx ? c : mx;
    }
    for (int off = 32; off >= 1; off >>= 1) {
        const int64_t o = __shfl_xor(mx, off, 64);
        mx = o > mx ? o : mx;
    }
    __syncthreads();                   // the previous segment is done with red / hist
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

// One workgroup per head (rows [h*n_per_head, (h+1)*n_per_head)), which
// sorts each piece of the head that falls into one XCD range.
__global__ __launch_bounds__(PLAN_NT) void lpt_order_kernel(const int32_t* __restrict__ ptr, int64_t nrows,
                                                            int64_t n_per_head, int64_t cap,
                                                            int32_t* __restrict__ order) {
    __shared__ uint32_t hist[PLAN_CLASSES][PLAN_NT];
    __shared__ uint32_t part[PLAN_NT];
    __shared__ int64_t red[PLAN_NT / 64];
    const int64_t h0 = static_cast<int64_t>(blockIdx.x) * n_per_head;
    const int64_t h1 = h0 + n_per_head < nrows ? h0 + n_per_head : nrows;
    const int64_t q = nrows >> 3, r = nrows & 7;
    int64_t s0 = h0;
    while (s0 < h1) {
        // XCD range holding row s0 and its end
        int64_t x = 0, xend = 0;
        for (x = 0; x < 8; ++x) {
            xend = (x + 1) * q + (x + 1 < r ? x + 1 : r);
            if (s0 < xend) break;
        }
        const int64_t s1 = xend < h1 ? xend : h1;
        lpt_segment(ptr, cap, order, s0, s1 - s0, hist, part, red);
        s0 = s1;
    }
}

hipError_t launch_lpt_order(const int32_t* ptr, int64_t nrows, int64_t n_per_head, int64_t cap, int32_t* order,
                            hipStream_t s) {
    if (nrows <= 0) return hipSuccess;
    const int64_t heads = (nrows + n_per_head - 1) / n_per_head;
    hipLaunchKernelGGL(lpt_order_kernel, dim3(static_cast<unsigned>(heads)), dim3(PLAN_NT), 0, s, ptr, nrows,
                       n_per_head, cap, order);
    return hipGetLastError();
}

}  // namespace vsa2

namespace vsa2 {

// ---------------------------------------------------------------------------
// Magnitude flags of the 64-token blocks.
//
// bf16 products round P (in P.V and P^T dO) and dS (in dS K and dS^T Q) to 8
// significant bits.  Those rounding errors are independent per element, but
// the products multiply them by the other operand: when the keys (queries,
// values) of a block share a large common component, the errors of a row
// add up coherently along that component and are no longer small next to
// the result, which is a difference of such components.  Large values also
// make the softmax peaked, so P close to 1 repeats across the queries of a
// block.  The attention kernels therefore take two-term (hi + lo) operands
// on every block pair where a value of the query block or of the key block
// (its K or V rows) exceeds SCALE_FLAG_BF16_BITS in magnitude, and one-term
// operands elsewhere.  Flag = 1 when some real token of the block holds such
// a value (padding tokens are ignored: no output may depend on them).
// Layout (see block_flag_layout): one byte per query block (b*Hq + h)*N + n,
// one per key block (b*Hkv + h)*N + n (K and V combined), then per KV group
// b*Hkv + h one word "some query block of the group's query heads is
// flagged" and one word "some key block of the head is flagged", so a kernel
// whose head has no flagged block reads no per-pair flag.
//
// Row flags (the backward's dS): dS = P (dP - Delta), and Delta = dO . O is
// large in every row that attends to a large-magnitude block, so the dS of
// that row's other pairs are large as well even where both blocks of the
// pair are small; rounded to one bf16 term they add an error coherent along
// the queries' (keys') common component to dK (dQ).  The backward therefore
// takes two-term dS on every pair of a query block whose row touches a
// flagged block (its own flag included), and keeps the pair rule for P.
// One byte per query block: bit 0 its own flag, bit 1 the row flag; one
// word per KV group: some query block of the group has the row flag.
// ---------------------------------------------------------------------------
constexpr uint32_t SCALE_FLAG_BF16_BITS = 0x40E0u;   // 7.0 in bf16

__global__ __launch_bounds__(256) void block_flag_kernel(const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
                                                         const uint16_t* __restrict__ v, uint8_t* __restrict__ flag_q,
                                                         uint8_t* __restrict__ flag_kv, int32_t* __restrict__ any_q,
                                                         int32_t* __restrict__ any_kv,
                                                         int64_t rows_q, int64_t rows_kv, int N, int D, int Hq,
                                                         int Hkv, cube_grid grid) {
    const int lane = threadIdx.x & 63;
    const int64_t row = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
    if (row >= rows_q + rows_kv) return;                 // whole waves leave together
    const bool is_q = row < rows_q;
    const int64_t r = is_q ? row : row - rows_q;
    const uint64_t real = cube_real_mask(grid, static_cast<int>(r % N), lane);
    // the block is 64 tokens x D contiguous bf16 values; lane l reads the
    // 16-byte chunks l, l + 64, ... (chunk c holds token c / (D / 8))
    const int64_t elems = static_cast<int64_t>(64) * D;
    const int chunks = 64 * D / 8;
    uint32_t mx = 0;
    auto scan = [&](const uint16_t* base) {
        const uint4* p = reinterpret_cast<const uint4*>(base + r * elems);
        for (int c = lane; c < chunks; c += 64) {
            const int tok = c / (D / 8);
            if (!((real >> tok) & 1)) continue;
            const uint4 w = p[c];
            const uint32_t u[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const uint32_t a = u[i] & 0x7fffu, b = (u[i] >> 16) & 0x7fffu;
                mx = a > mx ? a : mx;
                mx = b > mx ? b : mx;
            }
        }
    };
    if (is_q) {
        scan(q);
    } else {
        scan(k);
        scan(v);
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
        const uint32_t o = static_cast<uint32_t>(__shfl_xor(static_cast<int>(mx), off, 64));
        mx = o > mx ? o : mx;
    }
    const bool big = mx > SCALE_FLAG_BF16_BITS;
    if (lane == 0) {
        (is_q ? flag_q : flag_kv)[r] = big ? 1 : 0;
        if (big) {   // every writer stores the same value: the result does not depend on their order
            const int64_t bh = r / N;
            if (is_q) any_q[(bh / Hq) * Hkv + (bh % Hq) / (Hq / Hkv)] = 1;
            else any_kv[bh] = 1;
        }
    }
}

__global__ __launch_bounds__(256) void zero_i32_kernel(int32_t* __restrict__ p, int64_t n) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i < n) p[i] = 0;
}

// Row flags, first step (one wave per query block): bit 0 = the block's own
// flag, bit 1 = its own flag or |Delta| above DELTA_FLAG at one of its
// queries with attention mass (scaled LSE below +inf; padding queries and
// empty rows have none); the group word is set for bit 1.  The statistics
// hold, per 64-token block, 64 scaled LSE values then 64 negated Deltas.
__global__ __launch_bounds__(256) void row_flag_init_kernel(const uint8_t* __restrict__ flag_q,
                                                            const float* __restrict__ stat,
                                                            uint8_t* __restrict__ qrow, int32_t* __restrict__ any_row,
                                                            int64_t rows_q, int N, int Hq, int Hkv) {
    const int lane = threadIdx.x & 63;
    const int64_t r = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
    if (r >= rows_q) return;                          // wave-uniform
    const float ls = stat[r * 128 + lane], nd = stat[r * 128 + 64 + lane];
    const bool dbig = __any(ls != INFINITY && fabsf(nd) > DELTA_FLAG);
    const bool f = flag_q[r] != 0;
    if (lane == 0) {
        qrow[r] = static_cast<uint8_t>((f ? 1 : 0) | (f || dbig ? 2 : 0));
        if (f || dbig) {     // every writer stores the same value
            const int64_t bh = r / N;
            any_row[(bh / Hq) * Hkv + (bh % Hq) / (Hq / Hkv)] = 1;
        }
    }
}

// Row flags, second step: one wave per key block; a flagged key block sets
// bit 1 of every query block in its transposed list (entries
// hq_local * N + n_q, as the dK/dV kernel reads them; entries outside
// [0, grp*N) are skipped).  Concurrent writers of one byte all store
// (bit 0 from the first step) | 2, so the result does not depend on order.
__global__ __launch_bounds__(256) void row_flag_scatter_kernel(const uint8_t* __restrict__ flag_kv,
                                                               const int32_t* __restrict__ kv_ptr,
                                                               const int32_t* __restrict__ kv_idx, int64_t col_cap,
                                                               uint8_t* __restrict__ qrow,
                                                               int32_t* __restrict__ any_row, int64_t rows_kv, int N,
                                                               int Hq, int Hkv) {
    const int lane = threadIdx.x & 63;
    const int64_t r = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
    if (r >= rows_kv || !flag_kv[r]) return;          // wave-uniform
    int64_t e0 = kv_ptr[r], e1 = kv_ptr[r + 1];
    e0 = e0 < 0 ? 0 : (e0 > col_cap ? col_cap : e0);
    e1 = e1 < e0 ? e0 : (e1 > col_cap ? col_cap : e1);
    const int grp = Hq / Hkv;
    const int64_t bkv = r / N;
    const int64_t b = bkv / Hkv, hkv = bkv % Hkv;
    const int64_t qrow0 = (b * Hq + hkv * grp) * N;
    bool any = false;
    for (int64_t e = e0 + lane; e < e1; e += 64) {
        const int ent = kv_idx[e];
        if (ent < 0 || ent / N >= grp) continue;
        uint8_t* c = qrow + qrow0 + ent;
        *c = static_cast<uint8_t>(*c | 2);
        any = true;
    }
    if (__any(any) && lane == 0) any_row[bkv] = 1;
}

static size_t flag_align(size_t x) { return (x + 255) / 256 * 256; }

// Each array starts on a 256-byte boundary, so the kernels' 32-bit reads of
// the word holding a flag byte stay aligned and inside the array's span.
block_flag_layout block_flags_at(void* base, int64_t rows_q, int64_t rows_kv, int64_t groups) {
    block_flag_layout f;
    char* b = static_cast<char*>(base);
    f.q = reinterpret_cast<uint8_t*>(b);
    f.kv = reinterpret_cast<uint8_t*>(b + flag_align(rows_q));
    f.any_q = reinterpret_cast<int32_t*>(b + flag_align(rows_q) + flag_align(rows_kv));
    f.any_kv = f.any_q + groups;
    f.qrow = reinterpret_cast<uint8_t*>(b + flag_align(rows_q) + flag_align(rows_kv) + flag_align(8 * groups));
    f.any_row = reinterpret_cast<int32_t*>(b + 2 * flag_align(rows_q) + flag_align(rows_kv) + flag_align(8 * groups));
    return f;
}

size_t block_flags_bytes(int64_t rows_q, int64_t rows_kv, int64_t groups) {
    return 2 * flag_align(rows_q) + flag_align(rows_kv) + flag_align(8 * groups) + flag_align(4 * groups);
}

hipError_t launch_block_flags(const void* q, const void* k, const void* v, const block_flag_layout& f, int64_t rows_q,
                              int64_t rows_kv, int N, int D, int Hq, int Hkv, const cube_grid& cg, hipStream_t s) {
    const int64_t rows = rows_q + rows_kv;
    if (rows <= 0) return hipSuccess;
    const int64_t groups = rows_kv / N;
    hipLaunchKernelGGL(zero_i32_kernel, dim3(static_cast<unsigned>((2 * groups + 255) / 256)), dim3(256), 0, s,
                       f.any_q, 2 * groups);
    hipLaunchKernelGGL(block_flag_kernel, dim3(static_cast<unsigned>((rows + 3) / 4)), dim3(256), 0, s,
                       static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k),
                       static_cast<const uint16_t*>(v), f.q, f.kv, f.any_q, f.any_kv, rows_q, rows_kv, N, D, Hq, Hkv,
                       cg);
    return hipGetLastError();
}

// Row flags from the block flags (which the same workspace already holds),
// the statistics (Deltas) and the transposed lists.
hipError_t launch_row_flags(const block_flag_layout& f, const float* stat, const int32_t* kv_ptr,
                            const int32_t* kv_idx, int64_t col_cap, int64_t rows_q, int64_t rows_kv, int N, int Hq,
                            int Hkv, hipStream_t s) {
    if (rows_q <= 0 || rows_kv <= 0) return hipSuccess;
    const int64_t groups = rows_kv / N;
    hipLaunchKernelGGL(zero_i32_kernel, dim3(static_cast<unsigned>((groups + 255) / 256)), dim3(256), 0, s,
                       f.any_row, groups);
    hipLaunchKernelGGL(row_flag_init_kernel, dim3(static_cast<unsigned>((rows_q + 3) / 4)), dim3(256), 0, s,
                       f.q, stat, f.qrow, f.any_row, rows_q, N, Hq, Hkv);
    hipLaunchKernelGGL(row_flag_scatter_kernel, dim3(static_cast<unsigned>((rows_kv + 3) / 4)), dim3(256), 0, s,
                       f.kv, kv_ptr, kv_idx, col_cap, f.qrow, f.any_row, rows_kv, N, Hq, Hkv);
    return hipGetLastError();
}

}  // namespace vsa2
