// Block-sparse attention forward (VSA2 Sec. 2.1 with a block mask, Sec. 2.2
// Eq. block_sparse) for gfx950.
//
// One workgroup of two waves per query block (64 queries); wave w owns
// queries 32w .. 32w+31.  For every key block listed in the block's CSR row:
//   K, V tiles [64 keys][D] -> LDS, key r at LDS row tile_slot(r)
//   S^T = K Q^T            (MFMA 32x32, Q fragments live in registers)
//   online softmax in fp32 registers (exp2, log2(e)/sqrt(D) folded in)
//   O^T += V^T P^T         (P rounded to the input dtype, MFMA 32x32; the
//                           V^T operand comes from the row-major V tile by
//                           transposing LDS reads)
// Tiles arrive by global_load_lds (no staging registers).  The K and V
// buffers are refilled as soon as their last reader is done: the next K tile
// streams in during this tile's softmax and PV product, the next V tile
// during the next S product.
// In the transposed products a lane owns one query column, so the row max
// and row sum need one exchange with the other half-wave and nothing else.
// On a padded grid the padding keys of a cut cube are masked out of the
// softmax, and padding queries give O = 0 and LSE = -inf.
#include <type_traits>

#include "common.hpp"
#include "internal.hpp"

namespace vsa2 {

constexpr int AF_NT = 128;

// COMP (the forward of a training step): the rounding remainder of O is
// written to o_lo, so that O + o_lo carries about 16 significant bits for
// the backward's Delta = dO . O, and on every block pair of a row that
// touches a large-magnitude block (the query block's own flag or a listed
// key block's) P enters the PV product as two bf16 terms (hi + lo), which
// keeps O itself accurate to about 16 bits there: in such a row the
// rounding of P on a small pair, weighted by how far that pair's dO . V
// lies from the row's mean, reaches Delta as well.  Other rows take
// one-term P.
// PAD: the grid is padded (the masking is compiled only into this variant,
// so the unpadded one keeps its register budget).
template <typename T, int D, bool COMP, bool PAD>
__global__ __launch_bounds__(AF_NT, 2) void attn_fwd_kernel(
    const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ v,
    const int32_t* __restrict__ row_ptr, const int32_t* __restrict__ col_idx, int64_t col_cap,
    T* __restrict__ o, float* __restrict__ lse, T* __restrict__ o_lo, int Hq, int Hkv, int N, float c_log2,
    int period, const int32_t* __restrict__ order, cube_grid grid, block_flag_layout fl) {
    using F = typename frag_of<T>::type;
    constexpr bool SPLIT = COMP && sizeof(T) == 2;   // two-term P possible (bf16 only)
    constexpr int E = sizeof(T);
    constexpr int KS = D / 16;        // macro k-steps over the head dim
    constexpr int MT = D / 32;        // 32-row tiles of O^T
    constexpr int KRB = D * E;        // K and V tile row bytes
    using KT = async_tile<64, KRB, 2, true, E == 2>;
    using VT = KT;
    __shared__ __align__(1024) char k_lds[KT::BYTES];
    __shared__ __align__(1024) char v_lds[VT::BYTES];

    const int tid = threadIdx.x, lane = tid & 63, wave = wave_id(), half = lane >> 5;
    const int64_t row = work_row(order, xcd_item(blockIdx.x, gridDim.x), gridDim.x);
    const int64_t bh = row / N;
    const int n = static_cast<int>(row % N);
    const int b = static_cast<int>(bh / Hq), h = static_cast<int>(bh % Hq);
    const int hkv = h / (Hq / Hkv);
    const int64_t L = static_cast<int64_t>(N) * 64;
    const char* kb = reinterpret_cast<const char*>(k + static_cast<int64_t>(b * Hkv + hkv) * L * D);
    const char* vb = reinterpret_cast<const char*>(v + static_cast<int64_t>(b * Hkv + hkv) * L * D);
    const int64_t qtok = bh * L + static_cast<int64_t>(n) * 64 + wave * 32 + (lane & 31);
    bool q_real = true;
    if constexpr (PAD) q_real = (cube_real_mask(grid, n, lane) >> (wave * 32 + (lane & 31))) & 1;

    int64_t e0 = row_ptr[row], e1 = row_ptr[row + 1];
    e0 = e0 < 0 ? 0 : (e0 > col_cap ? col_cap : e0);
    e1 = e1 < e0 ? e0 : (e1 > col_cap ? col_cap : e1);

    F qf[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) load_frag(qf[ks], q + qtok * D + ks * 16 + half * 8);
    if constexpr (PAD) {
        // a padding query computes with a zero vector (its output is 0
        // anyway), so the wave's shared rescale decisions never depend on
        // what the padding holds
        if (!q_real) {
            const float z[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) pack_frag(qf[ks], z);
        }
    }

    f32x16_t oacc[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int i = 0; i < 16; ++i) oacc[mt][i] = 0.f;
    float m = -INFINITY, l = 0.f, lr = 0.f;   // row sums of p: exact (LSE), as rounded for the products (O)

    // entries outside [0, N) are loaded as block 0 and then ignored
    auto block_of = [&](int64_t e) -> int {
        const int c = scalar_load_i32(col_idx + e);
        return (c >= 0 && c < N) ? c : -1;
    };
    // two-term P on every pair of a row that touches a flagged block: the
    // query block's own flag, else (only when the head holds a flagged key
    // block) a scan of the listed key blocks' flags, 64 entries per step;
    // all of it completes before the first tile copy is issued
    const int64_t kvrow0 = static_cast<int64_t>(b * Hkv + hkv) * N;
    bool big = false;
    if constexpr (SPLIT) {
        big = byte_of(scalar_load_i32(byte_word(fl.q, row)), row);
        if (!big && scalar_load_i32(fl.any_kv + b * Hkv + hkv) != 0) {
            bool hit = false;
            for (int64_t e = e0 + lane; e < e1; e += 64) {
                const int c = col_idx[e];
                if (c >= 0 && c < N && fl.kv[kvrow0 + c]) hit = true;
            }
            big = __any(hit);
        }
    }
    const KT kt(wave, lane);
    const KT& vt_ = kt;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) settle(qf[ks]);   // fragments in registers before the copies start
    // phased sweep: entry j of the row is e0 + (s0 + j) mod cnt
    const int64_t cnt = e1 - e0;
    const int64_t s0 = sweep_start(col_idx, e0, cnt, blockIdx.x >> 3, period, N);
    auto entry = [&](int64_t j) -> int64_t {
        const int64_t t = s0 + j;
        return e0 + (t >= cnt ? t - cnt : t);
    };
    int c_cur = -1;
    if (cnt > 0) {
        c_cur = block_of(entry(0));
        const int cc = c_cur < 0 ? 0 : c_cur;
        kt.issue(k_lds, kb + static_cast<int64_t>(cc) * 64 * KRB, wave);
        vt_.issue(v_lds, vb + static_cast<int64_t>(cc) * 64 * KRB, wave);
    }
    // The walk in two compiled versions: TWO (every pair two-term) and the
    // one-term walk, each scheduled as one piece.
    auto walk = [&](auto two_term) {
        constexpr bool TWO = decltype(two_term)::value;
        for (int64_t j = 0; j < cnt; ++j) {
            const bool has_next = j + 1 < cnt;
            const int c_next = has_next ? block_of(entry(j + 1)) : -1;
            const int64_t nxt_off = static_cast<int64_t>(c_next < 0 ? 0 : c_next) * 64 * KRB;

            vm_wait<VT::PER_WAVE>();          // this K tile has landed (V may still stream)
            wg_barrier();
            // S^T for 64 keys x 32 queries (two 32-key tiles); K fragments are
            // requested one k-step pair ahead of their products
            f32x16_t s[2];
    #pragma unroll
            for (int t2 = 0; t2 < 2; ++t2)
    #pragma unroll
                for (int i = 0; i < 16; ++i) s[t2][i] = 0.f;
            {
                F fa[2][4];
                auto fetch = [&](F* f, int bi) {
    #pragma unroll
                    for (int x = 0; x < 4; ++x)
                        lds_frag_s<KRB>(f[x], k_lds, (x & 1) * 32 + (lane & 31), (2 * bi + (x >> 1)) * 16 + half * 8);
                };
                fetch(fa[0], 0);
    #pragma unroll
                for (int bi = 0; bi < KS / 2; ++bi) {
                    if (bi + 1 < KS / 2) fetch(fa[(bi + 1) & 1], bi + 1);
                    lds_order();
    #pragma unroll
                    for (int x = 0; x < 4; ++x) mma(s[x & 1], fa[bi & 1][x], qf[2 * bi + (x >> 1)]);
                }
            }
            wg_barrier();                      // K buffer free
            if (has_next) kt.issue(k_lds, kb + nxt_off, wave);

            if (c_cur >= 0) {
                // padding keys of a cut cube: key of entry i of tile t2 is
                // 32 t2 + 16 (i / 8) + 8 half + i % 8
                if constexpr (PAD) {        // branch-free: a branch here costs registers
                    const uint64_t kmask = cube_real_mask(grid, c_cur, lane);
    #pragma unroll
                    for (int t2 = 0; t2 < 2; ++t2) {
                        const uint32_t lm = static_cast<uint32_t>(kmask >> (t2 * 32 + half * 8));
    #pragma unroll
                        for (int i = 0; i < 16; ++i)
                            s[t2][i] = ((lm >> ((i >> 3) * 16 + (i & 7))) & 1u) ? s[t2][i] : -INFINITY;
                    }
                }
                // Online softmax in log2 units with a lazily updated running max:
                // the accumulators are rescaled only when the block max exceeds
                // the running max m by more than 2^8 (any lane of the wave), so
                // p = 2^(s c - m) <= 256.  O = sum p V / sum p is exact for any m.
                float mx = -INFINITY;
    #pragma unroll
                for (int t2 = 0; t2 < 2; ++t2)
    #pragma unroll
                    for (int i = 0; i < 16; ++i) mx = fmaxf(mx, s[t2][i]);
                mx = fmaxf(mx, swap_half(mx)) * c_log2;
                if (__any(mx > m + 8.0f)) {
                    const float mn = fmaxf(m, mx);
                    const float alpha = fast_exp2(m - mn);
                    l *= alpha;
                    lr *= alpha;
    #pragma unroll
                    for (int mt = 0; mt < MT; ++mt)
    #pragma unroll
                        for (int i = 0; i < 16; ++i) oacc[mt][i] *= alpha;
                    m = mn;
                }
            }
            if (has_next) vm_wait<KT::PER_WAVE>(); else vm_wait<0>();   // V tile landed
            wg_barrier();
            if (c_cur >= 0) {
                // O^T += V^T P^T over 4 k-steps of 16 keys: keys 16kk + 8half + (0..7).
                // The probabilities of k-step kk + 1 (exponentials, row sum,
                // bf16 packing) are formed after the products of k-step kk in
                // program order, so they issue while those MFMAs run; V^T
                // fragments are requested one k-step ahead of their products.
                // On a flagged pair P is split into hi + lo = bf16(P - hi), and a
                // second pass adds V^T lo (its fragments read again).
                F pb[4], pl[SPLIT ? 4 : 1];
                constexpr bool two = SPLIT && TWO;
                float ps = 0.f, pr = 0.f;
                // Two row sums: ps of the probabilities themselves (for the
                // LSE, which the backward's recomputed P relies on) and pr of
                // the probabilities as the products take them (rounded to the
                // input dtype; hi + lo on a two-term pair).  O = sum p V / pr
                // is a weighted mean of V with exactly the weights the MFMAs
                // used, so a component that all value rows share passes
                // through without P's rounding error (which would otherwise
                // reach Delta = dO . O in the backward).
                auto make_p = [&](int kk) {
                    float pv8[8];
    #pragma unroll
                    for (int i = 0; i < 8; ++i) {
                        const float p = fast_exp2(fmaf(s[kk >> 1][(kk & 1) * 8 + i], c_log2, -m));
                        pv8[i] = p;
                        ps += p;
                    }
                    if (two) {
                        pack_frag_hilo(pb[kk], pl[SPLIT ? kk : 0], pv8);
                        pr = frag_sum(pl[SPLIT ? kk : 0], pr);
                    } else {
                        pack_frag(pb[kk], pv8);
                    }
                    pr = frag_sum(pb[kk], pr);
                };
                F fa[2][MT];
                auto fetch = [&](F* f, int kk) {
    #pragma unroll
                    for (int mt = 0; mt < MT; ++mt) lds_frag_tr<KRB, true>(f[mt], v_lds, mt * 32, kk * 16);
                };
                make_p(0);
                fetch(fa[0], 0);
    #pragma unroll
                for (int kk = 0; kk < 4; ++kk) {
                    if (kk + 1 < 4) fetch(fa[(kk + 1) & 1], kk + 1);
                    lds_order();
    #pragma unroll
                    for (int mt = 0; mt < MT; ++mt) mma(oacc[mt], fa[kk & 1][mt], pb[kk]);
                    if (kk + 1 < 4) make_p(kk + 1);
                }
                l += ps;
                lr += pr;
                if constexpr (SPLIT) {
                    if (two) {
                        fetch(fa[0], 0);
    #pragma unroll
                        for (int kk = 0; kk < 4; ++kk) {
                            if (kk + 1 < 4) fetch(fa[(kk + 1) & 1], kk + 1);
                            lds_order();
    #pragma unroll
                            for (int mt = 0; mt < MT; ++mt) mma(oacc[mt], fa[kk & 1][mt], pl[kk]);
                        }
                    }
                }
            }
            wg_barrier();                      // V buffer free
            if (has_next) vt_.issue(v_lds, vb + nxt_off, wave);
            c_cur = c_next;
        }
    };
    if (SPLIT && big) walk(std::true_type{});
    else walk(std::false_type{});

    const float lt = q_real ? l + swap_half(l) : 0.f;     // a padding query has no output
    const float lrt = q_real ? lr + swap_half(lr) : 0.f;
    const float inv = lrt > 0.f ? 1.0f / lrt : 0.f;
    T* orow = o + qtok * D;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
            const int d0 = mt * 32 + g4 * 8 + half * 4;
            float ov[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) ov[j] = q_real ? oacc[mt][g4 * 4 + j] * inv : 0.f;
            if constexpr (E == 2) {
                const uint32_t w0 = pack2_bf16(ov[0], ov[1]);
                const uint32_t w1 = pack2_bf16(ov[2], ov[3]);
                *reinterpret_cast<uint2*>(orow + d0) = make_uint2(w0, w1);
                if constexpr (COMP) {
                    const uint32_t r0 = pack2_bf16(ov[0] - __uint_as_float(w0 << 16),
                                                   ov[1] - __uint_as_float(w0 & 0xffff0000u));
                    const uint32_t r1 = pack2_bf16(ov[2] - __uint_as_float(w1 << 16),
                                                   ov[3] - __uint_as_float(w1 & 0xffff0000u));
                    *reinterpret_cast<uint2*>(o_lo + qtok * D + d0) = make_uint2(r0, r1);
                }
            } else {
                *reinterpret_cast<float4*>(orow + d0) = make_float4(ov[0], ov[1], ov[2], ov[3]);
                if constexpr (COMP)
                    *reinterpret_cast<float4*>(o_lo + qtok * D + d0) = make_float4(0.f, 0.f, 0.f, 0.f);
            }
        }
    if (half == 0) lse[qtok] = lt > 0.f ? (m + log2f(lt)) * 0.6931471805599453f : -INFINITY;
}

template <typename T, int D, bool COMP, bool PAD>
static void launch_fwd_k(const void* q, const void* k, const void* v, const int32_t* row_ptr, const int32_t* col_idx,
                         int64_t col_cap, void* o, float* lse, void* o_lo, const int32_t* order, int64_t rows, int Hq,
                         int Hkv, int N, const cube_grid& cg, const block_flag_layout& fl, hipStream_t s) {
    const float c = 1.4426950408889634f / sqrtf(static_cast<float>(D));
    hipLaunchKernelGGL((attn_fwd_kernel<T, D, COMP, PAD>), dim3(static_cast<unsigned>(rows)), dim3(AF_NT), 0, s,
                       static_cast<const T*>(q), static_cast<const T*>(k), static_cast<const T*>(v), row_ptr,
                       col_idx, col_cap, static_cast<T*>(o), lse, static_cast<T*>(o_lo), Hq, Hkv, N, c,
                       resident_per_xcd<attn_fwd_kernel<T, D, COMP, PAD>>(AF_NT), order, cg, fl);
}

// Forward workspace: the work order of the CSR rows (one int32 per row), then
// the block magnitude flags (used when the call keeps O's remainder).
static size_t align256f(size_t x) { return (x + 255) / 256 * 256; }

size_t fwd_workspace_bytes(int batch, int Hq, int Hkv, int N) {
    const int64_t rq = static_cast<int64_t>(batch) * Hq * N, rkv = static_cast<int64_t>(batch) * Hkv * N;
    return align256f(4 * static_cast<size_t>(rq)) + block_flags_bytes(rq, rkv, static_cast<int64_t>(batch) * Hkv);
}

template <typename T, int D>
static hipError_t launch_fwd_t(const void* q, const void* k, const void* v, const int32_t* row_ptr,
                               const int32_t* col_idx, int64_t col_cap, void* o, float* lse, void* o_lo,
                               void* ws, int batch, int Hq, int Hkv, int N, const cube_grid& cg,
                               hipStream_t s) {
    const int64_t rows = static_cast<int64_t>(batch) * Hq * N;
    if (rows == 0) return hipSuccess;
    const int64_t rows_kv = static_cast<int64_t>(batch) * Hkv * N;
    int32_t* order = static_cast<int32_t*>(ws);
    const block_flag_layout fl = block_flags_at(static_cast<char*>(ws) + align256f(4 * static_cast<size_t>(rows)),
                                                rows, rows_kv, static_cast<int64_t>(batch) * Hkv);
    hipError_t e = launch_lpt_order(row_ptr, rows, N, col_cap, order, s);
    if (e != hipSuccess) return e;
    if (o_lo) {
        if constexpr (sizeof(T) == 2) {
            e = launch_block_flags(q, k, v, fl, rows, rows_kv, N, D, Hq, Hkv, cg, s);
            if (e != hipSuccess) return e;
        }
        if (cg.padded) launch_fwd_k<T, D, true, true>(q, k, v, row_ptr, col_idx, col_cap, o, lse, o_lo, order, rows, Hq, Hkv, N, cg, fl, s);
        else launch_fwd_k<T, D, true, false>(q, k, v, row_ptr, col_idx, col_cap, o, lse, o_lo, order, rows, Hq, Hkv, N, cg, fl, s);
    } else {
        if (cg.padded) launch_fwd_k<T, D, false, true>(q, k, v, row_ptr, col_idx, col_cap, o, lse, nullptr, order, rows, Hq, Hkv, N, cg, fl, s);
        else launch_fwd_k<T, D, false, false>(q, k, v, row_ptr, col_idx, col_cap, o, lse, nullptr, order, rows, Hq, Hkv, N, cg, fl, s);
    }
    return hipGetLastError();
}

hipError_t launch_attn_fwd(int dtype, int D, const void* q, const void* k, const void* v,
                           const int32_t* row_ptr, const int32_t* col_idx, int64_t col_cap, void* o,
                           float* lse, void* o_lo, void* ws, int batch, int Hq, int Hkv, int N,
                           const cube_grid& cg, hipStream_t s) {
    if (dtype == 1) {
        if (D == 64) return launch_fwd_t<bf16_t, 64>(q, k, v, row_ptr, col_idx, col_cap, o, lse, o_lo, ws, batch, Hq, Hkv, N, cg, s);
        if (D == 128) return launch_fwd_t<bf16_t, 128>(q, k, v, row_ptr, col_idx, col_cap, o, lse, o_lo, ws, batch, Hq, Hkv, N, cg, s);
    } else {
        if (D == 64) return launch_fwd_t<float, 64>(q, k, v, row_ptr, col_idx, col_cap, o, lse, o_lo, ws, batch, Hq, Hkv, N, cg, s);
        if (D == 128) return launch_fwd_t<float, 128>(q, k, v, row_ptr, col_idx, col_cap, o, lse, o_lo, ws, batch, Hq, Hkv, N, cg, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace vsa2
