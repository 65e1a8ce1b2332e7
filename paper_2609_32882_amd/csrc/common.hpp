// Device-side building blocks shared by the gfx950 kernels of this library:
// element types, bf16 rounding, the 32x32 MFMA tile contraction and the
// LDS tile layouts used by the attention and router kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "internal.hpp"

namespace vsa2 {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16_t;

// ---------------------------------------------------------------------------
// Element types.  bf16 values travel as raw uint16 bit patterns.
// ---------------------------------------------------------------------------
struct bf16_t { uint16_t bits; };

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
    return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_vt;
typedef __attribute__((ext_vector_type(2))) float f32x2_vt;

// Round-to-nearest-even float -> bf16 with the hardware conversion
// (v_cvt_pk_bf16_f32), two values per instruction.
__device__ __forceinline__ uint32_t pack2_bf16(float lo, float hi) {
    const f32x2_vt v = {lo, hi};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_vt));
}
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    return static_cast<uint16_t>(pack2_bf16(f, 0.f) & 0xffffu);
}

// 2^x with the hardware exponential (v_exp_f32).
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Round-to-nearest-even double -> bf16 in one rounding: truncate to float
// with a sticky bit in the last place (round-to-odd), then round the float.
// Round-to-odd at 24 bits followed by RNE at 8 bits equals direct RNE.
__device__ __forceinline__ uint16_t f64_to_bf16(double d) {
    float f = __double2float_rz(d);
    uint32_t u = __float_as_uint(f);
    if (static_cast<double>(f) != d && (u & 0x7f800000u) != 0x7f800000u) u |= 1u;
    return f32_to_bf16(__uint_as_float(u));
}

// Element conversions for the two supported input types.
__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16_t x) { return bf16_to_f32(x.bits); }
__device__ __forceinline__ void from_f32(float& y, float x) { y = x; }
__device__ __forceinline__ void from_f32(bf16_t& y, float x) { y.bits = f32_to_bf16(x); }

// ---------------------------------------------------------------------------
// 32x32 MFMA tile contraction over a "macro k-step" of 16.
//
// For C[32x32] += A[32x16] * B[16x32]: lane l supplies row (l % 32) of A and
// column (l % 32) of B, each as 8 consecutive k values starting at
// 8 * (l / 32) (its "k-slots").  Any assignment of k-slots works as long as A
// and B use the same one, because the contraction sums over all 16.
//   bf16: one v_mfma_f32_32x32x16_bf16 (8 bf16 per lane = 16 bytes);
//   fp32: eight v_mfma_f32_32x32x2_f32, the j-th taking slot j of each lane
//         (so it contracts k-slots {j, 8 + j}).
// Accumulator layout (both): lane l holds column l % 32 and rows
// 8*(v/4) + 4*(l/32) + (v%4) for v = 0..15.
// ---------------------------------------------------------------------------
struct frag_bf16 { bf16x8_t v; };
struct frag_f32 { float v[8]; };

template <typename T> struct frag_of;
template <> struct frag_of<bf16_t> { using type = frag_bf16; };
template <> struct frag_of<float> { using type = frag_f32; };

__device__ __forceinline__ void mma(f32x16_t& c, const frag_bf16& a, const frag_bf16& b) {
    c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a.v, b.v, c, 0, 0, 0);
}
__device__ __forceinline__ void mma(f32x16_t& c, const frag_f32& a, const frag_f32& b) {
#pragma unroll
    for (int j = 0; j < 8; ++j) c = __builtin_amdgcn_mfma_f32_32x32x2f32(a.v[j], b.v[j], c, 0, 0, 0);
}

// Fragment loads from 16-byte aligned memory (LDS or global).
__device__ __forceinline__ void load_frag(frag_bf16& f, const void* p) {
    f.v = *reinterpret_cast<const bf16x8_t*>(p);
}
__device__ __forceinline__ void load_frag(frag_f32& f, const void* p) {
    const float4* q = reinterpret_cast<const float4*>(p);
    float4 a = q[0], b = q[1];
    f.v[0] = a.x; f.v[1] = a.y; f.v[2] = a.z; f.v[3] = a.w;
    f.v[4] = b.x; f.v[5] = b.y; f.v[6] = b.z; f.v[7] = b.w;
}

// Build a fragment from 8 fp32 values (P or dS operand): bf16 rounds (RNE).
__device__ __forceinline__ void pack_frag(frag_bf16& f, const float* x) {
    typedef __attribute__((__vector_size__(4 * sizeof(uint32_t)))) uint32_t u32x4_t;
    u32x4_t w;
#pragma unroll
    for (int i = 0; i < 4; ++i) w[i] = pack2_bf16(x[2 * i], x[2 * i + 1]);
    f.v = __builtin_bit_cast(bf16x8_t, w);
}
__device__ __forceinline__ void pack_frag(frag_f32& f, const float* x) {
#pragma unroll
    for (int i = 0; i < 8; ++i) f.v[i] = x[i];
}

// Two-term split of 8 fp32 values for compensated products: hi = bf16(x),
// lo = bf16(x - hi), so hi + lo carries about 16 significant bits and
// A*hi + A*lo reproduces A*x to ~2^-17 relative instead of 2^-9.
__device__ __forceinline__ void pack_frag_hilo(frag_bf16& hi, frag_bf16& lo, const float* x) {
    typedef __attribute__((__vector_size__(4 * sizeof(uint32_t)))) uint32_t u32x4_t;
    u32x4_t wh, wl;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        wh[i] = pack2_bf16(x[2 * i], x[2 * i + 1]);
        const float h0 = __uint_as_float(wh[i] << 16), h1 = __uint_as_float(wh[i] & 0xffff0000u);
        wl[i] = pack2_bf16(x[2 * i] - h0, x[2 * i + 1] - h1);
    }
    hi.v = __builtin_bit_cast(bf16x8_t, wh);
    lo.v = __builtin_bit_cast(bf16x8_t, wl);
}
__device__ __forceinline__ void pack_frag_hilo(frag_f32& hi, frag_f32& lo, const float* x) {
#pragma unroll
    for (int i = 0; i < 8; ++i) { hi.v[i] = x[i]; lo.v[i] = 0.f; }
}

// acc plus the sum of a fragment's 8 values as stored (bf16: four v_dot2
// against (1, 1), which add the rounded values in fp32).  Each word goes
// through a scalar first: this compiler turns __builtin_bit_cast of a
// vector element inside an unrolled loop into a cast of element 0.
__device__ __forceinline__ float frag_sum(const frag_bf16& f, float acc) {
    typedef __attribute__((__vector_size__(4 * sizeof(uint32_t)))) uint32_t u32x4_t;
    typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
    const u32x4_t w = __builtin_bit_cast(u32x4_t, f.v);
    const bf16x2_t one = __builtin_bit_cast(bf16x2_t, 0x3f803f80u);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const uint32_t word = w[i];
        acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, word), one, acc, false);
    }
    return acc;
}
__device__ __forceinline__ float frag_sum(const frag_f32& f, float acc) {
#pragma unroll
    for (int i = 0; i < 8; ++i) acc += f.v[i];
    return acc;
}

// Make the compiler complete the loads of a fragment here (an opaque use of
// its registers), so no wait for them is left inside a later loop.
__device__ __forceinline__ void settle(const frag_bf16& f) {
    typedef __attribute__((__vector_size__(4 * sizeof(uint32_t)))) uint32_t u32x4_t;
    const u32x4_t u = __builtin_bit_cast(u32x4_t, f.v);
    asm volatile("" ::"v"(u[0]), "v"(u[1]), "v"(u[2]), "v"(u[3]));
}
__device__ __forceinline__ void settle(const frag_f32& f) {
#pragma unroll
    for (int i = 0; i < 8; ++i) asm volatile("" ::"v"(f.v[i]));
}
__device__ __forceinline__ void settle(float x) { asm volatile("" ::"v"(x)); }
// Moves a fragment into accumulation registers (AGPRs) and keeps it there:
// MFMAs read their A / B operands from AGPRs directly, so a loop-invariant
// operand parked there costs no VGPRs and no copies.
__device__ __forceinline__ void pin_agpr(frag_bf16& f) { asm volatile("" : "+a"(f.v)); }
__device__ __forceinline__ void pin_agpr(frag_f32& f) {
#pragma unroll
    for (int i = 0; i < 8; ++i) asm volatile("" : "+a"(f.v[i]));
}

// A lane's neighbour value by a DPP lane pattern within rows of 16 lanes
// (CTRL: 0x00-0xFF quad_perm, 0x140 row_mirror, 0x141 row_half_mirror).
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float x) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xF, 0xF, false));
}

// Exchange with the lane 32 positions away (the other half of the wave).
__device__ __forceinline__ float swap_half(float x) { return __shfl_xor(x, 32, 64); }

// Key-row slot permutation used by the "transposed" formulations: swapping
// bits 2 and 3 of a row index inside each 32-row tile makes the accumulator
// rows held by one lane (8*(v/4) + 4*(l/32) + v%4) map to two runs of 8
// consecutive keys: 8*(l/32) + v for v < 8 and 16 + 8*(l/32) + (v - 8).
__device__ __forceinline__ int swap_bits_2_3(int r) {
    return (r & ~0xc) | ((r & 4) << 1) | ((r & 8) >> 1);
}

// Physical LDS row of tile row y in the padded tiles below (row stride
// RB + 16 bytes), and its inverse.  Inside each 16-row block, y = 8c + 4b + a
// (a < 4) moves to a row chosen so that the four rows a transposing read
// takes together from one half-wave (y = 4j .. 4j+3, i.e. fixed c and b)
// leave the 64 banks' 8-bank pieces they read disjoint, while any 16
// consecutive rows still fill all 16 bank groups of 16 bytes:
// - stride RB + 16 = 4 banks mod 64 (RB = 256, 512): row 8c + 2a + b, the
//   four rows 8 banks apart;
// - stride 36 banks (RB = 128): row 8(a/2) + 4c + 2(a%2) + b, the four rows
//   at bank offsets {0, 8, 32, 40} + const (their second 32-byte pieces sit
//   16 banks further).
template <int RB>
__host__ __device__ constexpr int tile_slot_of(int c, int b, int a) {
    return RB == 128 ? 8 * (a >> 1) + 4 * c + 2 * (a & 1) + b : 8 * c + 2 * a + b;
}
template <int RB>
__host__ __device__ constexpr int tile_slot(int y) {
    return (y & ~15) | tile_slot_of<RB>((y >> 3) & 1, (y >> 2) & 1, y & 3);
}
template <int RB>
__host__ __device__ constexpr int tile_row_at(int p) {
    const int q = p & 15;
    return (p & ~15) | (RB == 128 ? 8 * ((q >> 2) & 1) + 4 * (q & 1) + ((q >> 1) & 1) + 2 * ((q >> 3) & 1)
                                  : (q & 8) + 4 * (q & 1) + ((q >> 1) & 3));
}
template <int RB>
constexpr bool tile_slot_is_permutation() {
    for (int y = 0; y < 64; ++y)
        if (tile_row_at<RB>(tile_slot<RB>(y)) != y || (tile_slot<RB>(y) >> 4) != (y >> 4)) return false;
    return true;
}
static_assert(tile_slot_is_permutation<128>() && tile_slot_is_permutation<256>() &&
                  tile_slot_is_permutation<512>(), "tile_slot must permute rows inside 16-row blocks");

__device__ __forceinline__ int lane_id() { return threadIdx.x & 63; }

// Workgroup -> work-item mapping that keeps neighbouring items on one XCD.
// Workgroups are dispatched round-robin over the 8 XCDs (workgroup id mod 8),
// each with its own L2.  Mapping XCD x to the contiguous range of items
// [x*q + min(x, r), ...) (q = n / 8, r = n % 8) makes the workgroups of one
// XCD work on the same head and nearby blocks, so the key/value tiles they
// gather stay in that XCD's L2 instead of being fetched by all eight.
__device__ __forceinline__ int64_t xcd_item(int64_t bid, int64_t n) {
    const int64_t q = n >> 3, r = n & 7;
    const int64_t x = bid & 7, i = bid >> 3;
    return x * q + (x < r ? x : r) + i;
}

// Row processed by work item `item` of a launch of n items: order[item]
// (the longest-first order of the item's XCD range), or the item itself
// without an order (or for an out-of-range entry).
__device__ __forceinline__ int64_t work_row(const int32_t* order, int64_t item, int64_t n) {
    if (!order) return item;
    const int64_t r = order[item];
    return (r >= 0 && r < n) ? r : item;
}

// Index of the calling wave inside its workgroup, as a wave-uniform (scalar) value.
__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); }

// ---------------------------------------------------------------------------
// Asynchronous global -> LDS tile copies (global_load_lds_dwordx4).
//
// A tile is ROWS rows of RB bytes (row-major in global memory, row stride
// RB).  One wave instruction writes 1 KB of LDS (lane l -> base + 16 l), so
// each lane fetches whatever unit lands at its physical position.  Loads are
// tracked by vmcnt; callers wait with vm_wait<n>() (at most n of the most
// recent vector-memory operations still outstanding) and make the data
// visible with a raw s_barrier.
// ---------------------------------------------------------------------------
typedef __attribute__((address_space(3))) void lds_void_t;


template <int N>
__device__ __forceinline__ void vm_wait() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    // gfx9 s_waitcnt: vmcnt[3:0] | expcnt[6:4] | lgkmcnt[11:8] | vmcnt_hi[15:14]
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
    asm volatile("" ::: "memory");
}

// Workgroup barrier without the memory fence of __syncthreads (which would
// wait for every outstanding global_load_lds).  The empty asm statements keep
// the compiler from moving LDS accesses across it; the caller has already
// waited (vm_wait) for the tiles it is about to publish.
__device__ __forceinline__ void wg_barrier() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// Scheduling fence: no instruction is moved across it by the compiler's
// scheduler, so LDS reads written before it are issued before the MFMAs
// after it (their waits stay at the first use).  Used to request operand
// fragments one batch ahead of the products that consume them instead of
// right before each one.
__device__ __forceinline__ void lds_order() { __builtin_amdgcn_sched_barrier(0); }

// Wave-uniform 32-bit load through the scalar cache.  Used for block-list
// entries inside the pipelined loops: a vector load there would be counted by
// vmcnt together with the asynchronous tile copies and make the compiler wait
// for all of them before its first use.
__device__ __forceinline__ int32_t scalar_load_i32(const int32_t* p) {
    int32_t v;
    asm volatile("s_load_dword %0, %1, 0x0\n\ts_waitcnt lgkmcnt(0)" : "=s"(v) : "s"(p) : "memory");
    return v;
}

// Two independent wave-uniform 32-bit loads through the scalar cache with one
// wait (a block-list entry and the magnitude flag of an earlier entry).
__device__ __forceinline__ void scalar_load2_i32(const int32_t* a, const int32_t* b, int32_t& x, int32_t& y) {
    asm volatile("s_load_dword %0, %2, 0x0\n\ts_load_dword %1, %3, 0x0\n\ts_waitcnt lgkmcnt(0)"
                 : "=&s"(x), "=&s"(y)
                 : "s"(a), "s"(b)
                 : "memory");
}

// The 32-bit word holding byte i of a byte array (the array's allocation is
// a multiple of 4 bytes from a 4-byte aligned start), and byte i within it.
__device__ __forceinline__ const int32_t* byte_word(const uint8_t* p, int64_t i) {
    return reinterpret_cast<const int32_t*>(p + (i & ~int64_t(3)));
}
__device__ __forceinline__ bool byte_of(int32_t w, int64_t i) { return ((w >> (8 * (i & 3))) & 0xff) != 0; }
__device__ __forceinline__ int byte_val(int32_t w, int64_t i) { return (w >> (8 * (i & 3))) & 0xff; }

// One global_load_lds_dwordx4: lane l copies 16 bytes from base + voff(l) to
// LDS byte address lds + 16 l.  Issued as inline assembly so that the
// compiler's own wait-count bookkeeping, which cannot tell the LDS buffers
// apart, does not put a full vmcnt(0) wait in front of every LDS read; the
// kernels order these copies themselves with vm_wait and wg_barrier.
__device__ __forceinline__ void dma16(uint32_t lds, const void* base, int voff) {
    // readfirstlane works on (signed) 32-bit ints: both halves go back through
    // uint32_t so the low word is zero-extended, never sign-extended.
    const uint32_t l = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(lds)));
    const uint64_t b = reinterpret_cast<uint64_t>(base);
    const uint32_t hi = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(b >> 32)));
    const uint32_t lo = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(b & 0xffffffffu)));
    const uint64_t bs = (static_cast<uint64_t>(hi) << 32) | static_cast<uint64_t>(lo);
    asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2"
                 :
                 : "s"(l), "v"(voff), "s"(bs)
                 : "memory", "m0");
}

// A run of NR (1..4) such copies on one M0 value.  The instruction's
// offset field (13-bit signed) moves the LDS and the global address alike,
// so copy i of the run carries offset 1024 i and writes LDS bytes
// lds + 1024 i + 16 l.  Its global source is base + voff[i] + 1024 i: the
// caller passes base = the tile's address - 3072 and voff[i] = the byte
// offset + 1024 (3 - i), which keeps every voff unsigned.  One M0 write per
// four copies instead of one per copy.
constexpr int DMA_RUN = 4;
constexpr int DMA_BIAS = 1024 * (DMA_RUN - 1);
template <int NR>
__device__ __forceinline__ void dma16_run(uint32_t lds, uint64_t base, const int* voff) {
    static_assert(NR >= 1 && NR <= DMA_RUN, "run length");
    const uint32_t l = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(lds)));
    const uint32_t hi = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(base >> 32)));
    const uint32_t lo = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(base & 0xffffffffu)));
    const uint64_t bs = (static_cast<uint64_t>(hi) << 32) | static_cast<uint64_t>(lo);
    if constexpr (NR == 1)
        asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2"
                     : : "s"(l), "v"(voff[0]), "s"(bs) : "memory", "m0");
    else if constexpr (NR == 2)
        asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %3\n\t"
                     "global_load_lds_dwordx4 %2, %3 offset:1024"
                     : : "s"(l), "v"(voff[0]), "v"(voff[1]), "s"(bs) : "memory", "m0");
    else if constexpr (NR == 3)
        asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %4\n\t"
                     "global_load_lds_dwordx4 %2, %4 offset:1024\n\t"
                     "global_load_lds_dwordx4 %3, %4 offset:2048"
                     : : "s"(l), "v"(voff[0]), "v"(voff[1]), "v"(voff[2]), "s"(bs) : "memory", "m0");
    else
        asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %5\n\t"
                     "global_load_lds_dwordx4 %2, %5 offset:1024\n\t"
                     "global_load_lds_dwordx4 %3, %5 offset:2048\n\t"
                     "global_load_lds_dwordx4 %4, %5 offset:3072"
                     : : "s"(l), "v"(voff[0]), "v"(voff[1]), "v"(voff[2]), "v"(voff[3]), "s"(bs)
                     : "memory", "m0");
}

// Start offset of a block list for a phased sweep.  Row number `local` on
// its XCD starts at its first entry >= (local mod period) * npos / period and
// wraps around, with period = the number of workgroups resident on one XCD
// at a time.  Why this keeps co-resident workgroups on the same tiles: the
// dispatcher starts workgroup j when an earlier one ends, so in steady state
// the resident workgroups are J-period .. J-1 (J = next to dispatch) and
// workgroup J-m has done about m/period of its list, i.e. has advanced
// m*npos/period through the (evenly spread) positions.  Its start offset
// ((J-m) mod period)*npos/period cancels that advance modulo npos: every
// resident workgroup sits at about (J mod period)*npos/period, and the
// tiles they gather are shared through the XCD's L2.  This needs rows of
// (nearly) equal length; a period off by 2x in either direction loses most
// of the effect (measured).  The start depends only on the row number, so
// results stay deterministic.  Entries are read through the scalar cache
// (binary search, ~log2(n) loads).
__device__ __forceinline__ int64_t sweep_start(const int32_t* list, int64_t e0, int64_t cnt, int64_t local,
                                               int period, int npos) {
    if (cnt < 2 || period < 2) return 0;
    const int pos = static_cast<int>(((local % period) * npos) / period);
    int64_t lo = 0, hi = cnt;
    while (lo < hi) {
        const int64_t mid = (lo + hi) >> 1;
        if (scalar_load_i32(list + e0 + mid) < pos) lo = mid + 1;
        else hi = mid;
    }
    return lo == cnt ? 0 : lo;
}

// LDS tiles are stored with a row stride of RB + 16 bytes (64 banks of 4
// bytes: each row starts 4 banks after the previous one), and every fragment
// address is one per-lane base plus a compile-time offset (no per-fragment
// address registers).  When PERM, tile row y sits at LDS row tile_slot<RB>(y).
// Fragment readers take rows in the slot-swapped view of the MFMA layouts
// (lds_frag_s row s = tile row swap_bits_2_3(s)).
//
// bf16 tiles (CPERM) also place the 32-byte column groups of a row (16
// elements each) out of order: group g sits at position cgroup_pos(g) =
// (g & 1) * NG/2 + g/2 (NG = RB/32 groups), so the two 16-column halves of
// a 32-column fragment lie half a row apart.
// Bank conflicts: a 16-byte row read (lds_frag_s) serves 16 lanes per
// clock, which read one column of 16 consecutive tile rows: tile_slot
// permutes inside 16-row blocks and a row starts 4 (or 36) banks after the
// previous one, so they occupy 16 distinct bank groups.  A transposing read
// (lds_frag_tr) serves a half-wave per clock, 32 bytes of each column half
// of 4 tile rows y = 4j .. 4j+3: tile_slot places them so that the 8 pieces
// fill the 64 banks once.  (With the rows in slot-swapped order they
// overlapped 2-fold: 2 extra clocks per read, measured with
// SQ_LDS_BANK_CONFLICT.)
//
// A tile is copied by whole 1 KB wave instructions; lanes whose destination
// is a pad slot (or past the last row) fetch the tile's first 16 bytes
// again.  The per-lane source offsets are the same for every tile of a
// shape: they are computed once and each issue adds a wave-uniform base.
template <int RB>
__host__ __device__ constexpr int cgroup_pos(int g) {
    return (g & 1) * (RB / 64) + (g >> 1);
}
template <int RB>
__host__ __device__ constexpr int cgroup_of_pos(int pos) {
    return pos < RB / 64 ? 2 * pos : 2 * (pos - RB / 64) + 1;
}

template <int ROWS, int RB, int NW, bool PERM, bool CPERM = false>
struct async_tile {
    static constexpr int STRIDE = RB + 16;
    static constexpr int NI = ((ROWS * STRIDE + 1023) / 1024 + NW - 1) / NW * NW;  // 1 KB instructions
    static constexpr int BYTES = NI * 1024;        // LDS bytes to allocate
    static constexpr int PER_WAVE = NI / NW;
    static_assert(RB % 64 == 0, "row bytes");
    // per copy j: the source byte offset within the tile, plus the run
    // bias of dma16_run (1024 (3 - j mod 4))
    int off[PER_WAVE];
    static constexpr int bias(int j) { return DMA_BIAS - 1024 * (j % DMA_RUN); }

    __device__ __forceinline__ async_tile(int wave, int lane) {
#pragma unroll
        for (int j = 0; j < PER_WAVE; ++j) {
            const int p = (wave * PER_WAVE + j) * 1024 + lane * 16;   // physical LDS byte
            const int row = p / STRIDE, col = p % STRIDE;
            const bool data = row < ROWS && col < RB;
            const int lcol = CPERM ? cgroup_of_pos<RB>(col / 32) * 32 + col % 32 : col;
            off[j] = (data ? (PERM ? tile_row_at<RB>(row) : row) * RB + lcol : 0) + bias(j);
        }
    }
    __device__ __forceinline__ void issue(char* lds, const char* g, int wave) const {
        const uint32_t l0 = static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_void_t*)lds)) +
                            wave * PER_WAVE * 1024;
        const uint64_t b = reinterpret_cast<uint64_t>(g) - DMA_BIAS;
#pragma unroll
        for (int j = 0; j < PER_WAVE; j += DMA_RUN) {
            constexpr int R = PER_WAVE % DMA_RUN;
            if (j + DMA_RUN <= PER_WAVE) dma16_run<DMA_RUN>(l0 + j * 1024, b, off + j);
            else dma16_run<R == 0 ? 1 : R>(l0 + j * 1024, b, off + j);
        }
    }
    // A tile of which only the first `rows` rows (>= 1) exist in memory: the
    // other slots are filled from the first row (never read past the end).
    __device__ __forceinline__ void issue_rows(char* lds, const char* g, int wave, int lane, int64_t rows) const {
        const uint32_t l0 = static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_void_t*)lds));
#pragma unroll
        for (int j = 0; j < PER_WAVE; ++j) {
            const int p = (wave * PER_WAVE + j) * 1024 + lane * 16;
            const int row = p / STRIDE;                    // LDS slot
            const int grow = PERM ? tile_row_at<RB>(row) : row;
            const int raw = off[j] - bias(j);
            dma16(l0 + (wave * PER_WAVE + j) * 1024, g, (row < ROWS && grow < rows) ? raw : (raw % RB));
        }
    }
};

// A-operand fragment of a transposed use of a row-major tile.
//
// The tile holds X^T row-major: LDS row = the contraction index (a key or a
// query, stored at LDS row tile_slot(index) when PERM), columns = the output
// rows m (the head dimension d), in the bf16 column-group order above.  The
// MFMA 32x32x16 A operand for output tile rows m0 .. m0+31 (m0 a multiple
// of 32) and contraction indices k0 .. k0+15 needs, in lane l,
// X[m0 + l%32][k0 + 8(l/32) + s] for s = 0..7.  ds_read_b64_tr_b16 gives,
// within each group of 16 lanes, lane j the 4 values E[j/4 + 4c][j%4]
// (c = 0..3) of the 16x4 block E whose row i lane i addresses.  So lane i
// of group G (l = 16G + i) addresses contraction index k0 + 8(G/2) + 4r +
// i/4, columns m0 + 16(G%2) + 4(i%4) .. +3 (column group m0/16 + G%2), and
// read r = 0, 1 returns slots 4r .. 4r+3.  Every address is a per-lane base
// plus compile-time offsets.
template <int RB, bool PERM>
__device__ __forceinline__ void lds_frag_tr(frag_bf16& f, const char* tile, int m0, int k0) {
    typedef short v4i16 __attribute__((ext_vector_type(4)));
    typedef __attribute__((address_space(3))) v4i16 lds_v4i16;
    const int l = lane_id(), i = l & 15, G = l >> 4;
    v4i16 r2[2];
#pragma unroll
    for (int r = 0; r < 2; ++r) {
        // k0 and m0 are multiples of 16 and 32: the slot permutation acts
        // on the lane's part y = 8(G/2) + 4r + i/4 < 16 of the index only,
        // where it adds r to a per-lane row, and column group m0/16 + G%2
        // sits at position (G%2) RB/64 + m0/32, so the address is a per-lane
        // offset plus the constant (k0 + r)(RB + 16) + m0
        const int row = k0 + (PERM ? tile_slot_of<RB>(G >> 1, r, i >> 2) : 8 * (G >> 1) + 4 * r + (i >> 2));
        const int grp = (G & 1) * (RB / 64) + (m0 >> 5);
        const char* p = tile + row * (RB + 16) + grp * 32 + 8 * (i & 3);
        r2[r] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(p));
    }
    typedef __attribute__((__vector_size__(8 * sizeof(short)))) short s16x8_t;
    const s16x8_t w = {r2[0][0], r2[0][1], r2[0][2], r2[0][3], r2[1][0], r2[1][1], r2[1][2], r2[1][3]};
    f.v = __builtin_bit_cast(bf16x8_t, w);
}
// fp32 tiles: plain 4-byte reads of the same elements (no transposing read
// exists for 32-bit data; only the small fp32 problems take this path).
template <int RB, bool PERM>
__device__ __forceinline__ void lds_frag_tr(frag_f32& f, const char* tile, int m0, int k0) {
    const int l = lane_id();
    const int m = m0 + (l & 31);
#pragma unroll
    for (int s = 0; s < 8; ++s) {
        const int k = k0 + 8 * (l >> 5) + s;
        const int row = PERM ? tile_slot<RB>(k) : k;
        f.v[s] = *reinterpret_cast<const float*>(tile + row * (RB + 16) + m * 4);
    }
}

// Fragment of 8 consecutive elements starting at element e0 (a multiple of
// 8) of row s of the slot-swapped view of a padded, slot-permuted LDS tile
// with RB-byte rows (tile row swap_bits_2_3(s), bf16 columns in the
// column-group order above).
template <int RB>
__device__ __forceinline__ void lds_frag_s(frag_bf16& f, const char* tile, int s, int e0) {
    const int row = tile_slot<RB>(swap_bits_2_3(s));
    load_frag(f, tile + row * (RB + 16) + cgroup_pos<RB>(e0 >> 4) * 32 + (e0 & 15) * 2);
}
template <int RB>
__device__ __forceinline__ void lds_frag_s(frag_f32& f, const char* tile, int s, int e0) {
    const int row = tile_slot<RB>(swap_bits_2_3(s));
    const float4 a = *reinterpret_cast<const float4*>(tile + row * (RB + 16) + e0 * 4);
    const float4 b = *reinterpret_cast<const float4*>(tile + row * (RB + 16) + e0 * 4 + 16);
    f.v[0] = a.x; f.v[1] = a.y; f.v[2] = a.z; f.v[3] = a.w;
    f.v[4] = b.x; f.v[5] = b.y; f.v[6] = b.z; f.v[7] = b.w;
}

// ---------------------------------------------------------------------------
// Padded grids.  Real extent (rt, rh, rw) of cube n (index within a head).
// ---------------------------------------------------------------------------
__device__ __forceinline__ int3 cube_extent(const cube_grid& g, int n) {
    const int nw = n % g.Nw, r = n / g.Nw;
    const int nh = r % g.Nh, nt = r / g.Nh;
    return make_int3(min(g.Bt, g.T - nt * g.Bt), min(g.Bh, g.H - nh * g.Bh), min(g.Bw, g.W - nw * g.Bw));
}

__device__ __forceinline__ bool cube_is_full(const cube_grid& g, int3 e) {
    return e.x == g.Bt && e.y == g.Bh && e.z == g.Bw;
}

// Token beta (in-cube raster index) of a cube with extent e is real.
__device__ __forceinline__ bool token_in(const cube_grid& g, int3 e, int beta) {
    const int bw = beta % g.Bw, r = beta / g.Bw;
    const int bh = r % g.Bh, bt = r / g.Bh;
    return bt < e.x && bh < e.y && bw < e.z;
}

// Bit beta set for each real token of 64-token block n (a video cube, or a
// text block when n >= Nv).  Called by a whole wave (lane = its lane index);
// the result is wave-uniform.
__device__ __forceinline__ uint64_t cube_real_mask(const cube_grid& g, int n, int lane) {
    if (!g.padded) return ~0ull;
    if (n >= g.Nv) {
        const int left = g.text_len - (n - g.Nv) * 64;     // real text tokens from this block on
        return left >= 64 ? ~0ull : (left <= 0 ? 0ull : (~0ull >> (64 - left)));
    }
    const int3 e = cube_extent(g, n);
    if (cube_is_full(g, e)) return ~0ull;
    return __ballot(token_in(g, e, lane));
}

}  // namespace vsa2
