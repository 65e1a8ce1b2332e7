// Device-side building blocks shared by the gfx950 kernels of this library:
// element types, bf16 rounding, the 32x32 MFMA tile contraction and the
// LDS tile layouts used by the attention and router kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

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

// Round-to-nearest-even float -> bf16 (NaN kept quiet).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) return static_cast<uint16_t>((u >> 16) | 0x40u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return static_cast<uint16_t>(u >> 16);
}

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
    for (int i = 0; i < 4; ++i)
        w[i] = static_cast<uint32_t>(f32_to_bf16(x[2 * i])) |
               (static_cast<uint32_t>(f32_to_bf16(x[2 * i + 1])) << 16);
    f.v = __builtin_bit_cast(bf16x8_t, w);
}
__device__ __forceinline__ void pack_frag(frag_f32& f, const float* x) {
#pragma unroll
    for (int i = 0; i < 8; ++i) f.v[i] = x[i];
}

// Exchange with the lane 32 positions away (the other half of the wave).
__device__ __forceinline__ float swap_half(float x) { return __shfl_xor(x, 32, 64); }

// ---------------------------------------------------------------------------
// LDS tiles of 64 rows x ROW_BYTES bytes (ROW_BYTES a multiple of 128),
// addressed in 16-byte chunks with an XOR swizzle of the chunk index by the
// row's low 3 bits, so that lanes reading the same logical chunk of
// consecutive rows hit different banks.
// ---------------------------------------------------------------------------
template <int ROW_BYTES>
struct lds_tile {
    static constexpr int CHUNKS = ROW_BYTES / 16;
    static constexpr int BYTES = 64 * ROW_BYTES;
    __device__ static __forceinline__ int offset(int row, int chunk) {
        return row * ROW_BYTES + (chunk ^ (row & 7)) * 16;
    }
};

// Key-row slot permutation used by the "transposed" formulations: swapping
// bits 2 and 3 of a row index inside each 32-row tile makes the accumulator
// rows held by one lane (8*(v/4) + 4*(l/32) + v%4) map to two runs of 8
// consecutive keys: 8*(l/32) + v for v < 8 and 16 + 8*(l/32) + (v - 8).
__device__ __forceinline__ int swap_bits_2_3(int r) {
    return (r & ~0xc) | ((r & 4) << 1) | ((r & 8) >> 1);
}

__device__ __forceinline__ int lane_id() { return threadIdx.x & 63; }

// Fragment of 8 consecutive elements starting at element `e0` of row `row`
// of a swizzled LDS tile (bf16: one 16-byte chunk; fp32: two).
template <int ROW_BYTES>
__device__ __forceinline__ void lds_frag(frag_bf16& f, const char* tile, int row, int e0) {
    load_frag(f, tile + lds_tile<ROW_BYTES>::offset(row, e0 >> 3));
}
template <int ROW_BYTES>
__device__ __forceinline__ void lds_frag(frag_f32& f, const char* tile, int row, int e0) {
    const float4 a = *reinterpret_cast<const float4*>(tile + lds_tile<ROW_BYTES>::offset(row, e0 >> 2));
    const float4 b = *reinterpret_cast<const float4*>(tile + lds_tile<ROW_BYTES>::offset(row, (e0 >> 2) + 1));
    f.v[0] = a.x; f.v[1] = a.y; f.v[2] = a.z; f.v[3] = a.w;
    f.v[4] = b.x; f.v[5] = b.y; f.v[6] = b.z; f.v[7] = b.w;
}

// ---------------------------------------------------------------------------
// Cooperative copy of a 64-row x D tile from global memory into LDS.
// `load` issues the global reads into registers (rows >= nrows read as 0);
// `store` writes them to a swizzled LDS tile.  Straight copies keep the
// [row][D] layout, optionally placing row r at slot swap_bits_2_3(r);
// transposed copies write the [D][64] layout (each thread moves one 8x8
// block through registers).
// ---------------------------------------------------------------------------
template <typename T, int D, int NT>
struct tile_rows {
    static constexpr int E = sizeof(T);
    static constexpr int RB = D * E;           // bytes per row
    static constexpr int CH = RB / 16;          // 16-byte chunks per row
    static constexpr int PER = 64 * CH / NT;    // chunks per thread
    static_assert(PER >= 1 && (64 * CH) % NT == 0, "tile / thread count mismatch");
    uint4 r[PER];

    __device__ __forceinline__ void load(const T* base, int64_t row0, int64_t nrows, int tid) {
        const char* g = reinterpret_cast<const char*>(base);
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const int id = i * NT + tid;
            const int row = id / CH, ch = id % CH;
            if (row0 + row < nrows)
                r[i] = *reinterpret_cast<const uint4*>(g + (row0 + row) * RB + ch * 16);
            else
                r[i] = make_uint4(0, 0, 0, 0);
        }
    }
    __device__ __forceinline__ void store(char* lds, bool permute, int tid) const {
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const int id = i * NT + tid;
            const int row = id / CH, ch = id % CH;
            const int slot = permute ? swap_bits_2_3(row) : row;
            *reinterpret_cast<uint4*>(lds + lds_tile<RB>::offset(slot, ch)) = r[i];
        }
    }
};

template <typename T, int D, int NT>
struct tile_transposed {
    static constexpr int E = sizeof(T);
    static constexpr int RB = 64 * E;           // bytes per LDS row (one d)
    static constexpr int W = 8 * E / 16;        // 16-byte words per 8-element run
    static constexpr int BLOCKS = 8 * (D / 8);  // 8x8 blocks in the tile
    static_assert(BLOCKS <= NT, "one 8x8 block per thread");
    uint4 r[8][W];

    __device__ __forceinline__ void load(const T* base, int64_t row0, int tid) {
        if (tid >= BLOCKS) return;
        const int dc = tid % (D / 8), kb = tid / (D / 8);
        const char* g = reinterpret_cast<const char*>(base);
#pragma unroll
        for (int i = 0; i < 8; ++i)
#pragma unroll
            for (int w = 0; w < W; ++w)
                r[i][w] = *reinterpret_cast<const uint4*>(
                    g + (row0 + kb * 8 + i) * (int64_t)(D * E) + dc * 8 * E + w * 16);
    }
    // The same 8x8 blocks written untransposed: [64 rows][D] (row stride
    // D*E), row r at slot swap_bits_2_3(r) when `permute`.
    __device__ __forceinline__ void store_rows(char* lds, bool permute, int tid) const {
        if (tid >= BLOCKS) return;
        const int dc = tid % (D / 8), kb = tid / (D / 8);
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int row = kb * 8 + i;
            const int slot = permute ? swap_bits_2_3(row) : row;
#pragma unroll
            for (int w = 0; w < W; ++w)
                *reinterpret_cast<uint4*>(lds + lds_tile<D * E>::offset(slot, dc * W + w)) = r[i][w];
        }
    }
    __device__ __forceinline__ void store(char* lds, int tid) const {
        if (tid >= BLOCKS) return;
        const int dc = tid % (D / 8), kb = tid / (D / 8);
        if constexpr (E == 2) {
            // r[i] = 8 bf16 of key kb*8+i: word a = (d 2a, d 2a+1)
            const uint32_t* in[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) in[i] = reinterpret_cast<const uint32_t*>(&r[i][0]);
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const int a = j >> 1;
                uint32_t o[4];
#pragma unroll
                for (int m = 0; m < 4; ++m) {
                    const uint32_t x = in[2 * m][a], y = in[2 * m + 1][a];
                    o[m] = (j & 1) ? ((x >> 16) | (y & 0xffff0000u)) : ((x & 0xffffu) | (y << 16));
                }
                *reinterpret_cast<uint4*>(lds + lds_tile<RB>::offset(dc * 8 + j, kb)) =
                    make_uint4(o[0], o[1], o[2], o[3]);
            }
        } else {
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                float col[8];
#pragma unroll
                for (int i = 0; i < 8; ++i) col[i] = reinterpret_cast<const float*>(&r[i][0])[j];
                *reinterpret_cast<float4*>(lds + lds_tile<RB>::offset(dc * 8 + j, 2 * kb)) =
                    make_float4(col[0], col[1], col[2], col[3]);
                *reinterpret_cast<float4*>(lds + lds_tile<RB>::offset(dc * 8 + j, 2 * kb + 1)) =
                    make_float4(col[4], col[5], col[6], col[7]);
            }
        }
    }
};

}  // namespace vsa2
