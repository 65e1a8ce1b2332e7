// Block-sparse attention backward for gfx950.  The block mask is a constant
// (routing carries no gradient, VSA2 Sec. 2.1), so the gradients are those of
// masked softmax attention restricted to the selected block pairs:
//   Delta_l = dO_l . O_l
//   P = exp(S/sqrt(D) - LSE),  dP = dO V^T,  dS = P o (dP - Delta)
//   dV = P^T dO,  dK = dS^T Q / sqrt(D),  dQ = dS K / sqrt(D)
// Kernels, all deterministic (no atomics):
//   stat_kernel      per query token: LSE * log2(e) and -Delta
//   dkdv_kernel      key-block stationary: one workgroup per key block walks
//                    the transposed (CSC) list of query blocks that selected
//                    it; a wave owns 32 keys and accumulates dV^T and dK^T
//                    in registers
//   dq_kernel        query-block stationary: one workgroup per query block
//                    walks its CSR row; a wave owns 32 queries
// Products are arranged so that each lane owns one column (a key in dkdv, a
// query in dq) and its 16 accumulator rows form two runs of 8 consecutive
// rows (tiles stored with the bit-2/3 slot swap): a lane's P / dS values are
// directly the B operand of the next MFMA.  Every tile is a row-major
// [64 tokens][D] copy; the transposed operands (Q^T, dO^T, K^T) are read from
// the same tiles with transposing LDS reads.  Tiles stream into LDS with
// asynchronous global_load_lds copies; each buffer is refilled as soon as
// its last reader is done.
#include <type_traits>

#include "common.hpp"
#include "internal.hpp"

namespace vsa2 {

constexpr int AB_NT = 128;
constexpr float kLog2e = 1.4426950408889634f;

// ---------------------------------------------------------------------------
// Per query token l: LSE_l * log2(e) and -Delta_l = -(dO_l . O_l); 16 lanes
// per token (D <= 128).  With the forward's rounding remainder o_lo,
// O_l = o_l + o_lo_l.  A token without attention mass (LSE = -inf: a
// padding query, or an empty row) gets +inf, so every probability
// 2^(s - LSE log2 e) the backward forms for it is 0.
// Layout: per block of 64 tokens, the 64 scaled LSE values, then the 64
// negated Deltas (stat_at gives the element offsets), so one query block's
// statistics are one 512-byte copy and a lane's run of 8 consecutive
// queries is one 32-byte read of each.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int64_t stat_lse_at(int64_t tok) { return (tok >> 6) * 128 + (tok & 63); }
__device__ __forceinline__ int64_t stat_nd_at(int64_t tok) { return (tok >> 6) * 128 + 64 + (tok & 63); }

template <typename T, int D>
__global__ __launch_bounds__(256) void stat_kernel(const T* __restrict__ o, const T* __restrict__ o_lo,
                                                   const T* __restrict__ dout,
                                                   const float* __restrict__ lse, float* __restrict__ stat,
                                                   int64_t ntok) {
    constexpr int LPT = D / 8;   // lanes per token, 8 elements each
    const int64_t t = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    const int64_t tok = t / LPT;
    const int part = static_cast<int>(t % LPT);
    float s = 0.f;
    if (tok < ntok) {
        const T* a = o + tok * D + part * 8;
        const T* b = dout + tok * D + part * 8;
#pragma unroll
        for (int i = 0; i < 8; ++i) s += to_f32(a[i]) * to_f32(b[i]);
        if (o_lo) {
            const T* c = o_lo + tok * D + part * 8;
#pragma unroll
            for (int i = 0; i < 8; ++i) s += to_f32(c[i]) * to_f32(b[i]);
        }
    }
#pragma unroll
    for (int off = LPT / 2; off >= 1; off >>= 1) s += __shfl_xor(s, off, 64);
    if (tok < ntok && part == 0) {
        const float x = lse[tok];
        stat[stat_lse_at(tok)] = x == -INFINITY ? INFINITY : x * kLog2e;
        stat[stat_nd_at(tok)] = -s;
    }
}

// ---------------------------------------------------------------------------
// dK and dV: one workgroup (2 waves) per key block of head (b, hkv); a wave
// owns 32 keys and keeps both accumulators (dV^T, dK^T) in registers.  Per
// selecting query block:
//   S = Q K^T, dP = dO V^T   (Q, dO rows from LDS; K, V in registers)
//   P = exp2(S c - LSE log2 e), dS = P (dP - Delta)
//   dV^T += dO^T P,  dK^T += Q^T dS   (dO^T, Q^T read transposed from LDS)
// The Q / dO / stat tiles are double-buffered: the copies of the next query
// block stream in during the whole of the current one.  On a padded grid,
// padding keys get dK = dV = 0 and padding queries (scaled LSE = +inf) add
// nothing.  (PAD: the grid is padded; the masking is compiled only into
// that variant.)  bf16: on block pairs that touch a large-magnitude block
// (this key block's flag or the query block's) P enters the dV product as
// two bf16 terms (hi + lo); dS enters the dK product as two terms on those
// pairs and on every pair of a query block with the row flag (its row
// touches a flagged block, or one of its queries has |Delta| above
// DELTA_FLAG).
// ---------------------------------------------------------------------------
template <typename T, int D, bool PAD>
__global__ __launch_bounds__(AB_NT, 1) void dkdv_kernel(
    const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ v,
    const T* __restrict__ dout, const float* __restrict__ stat,
    const int32_t* __restrict__ kv_ptr, const int32_t* __restrict__ kv_idx, int64_t col_cap,
    T* __restrict__ dk, T* __restrict__ dv, int Hq, int Hkv, int N, float c_log2, float scale,
    const int32_t* __restrict__ order, cube_grid grid, block_flag_layout fl) {
    using F = typename frag_of<T>::type;
    constexpr int E = sizeof(T);
    constexpr int KS = D / 16;
    constexpr int MT = D / 32;
    constexpr int RB = D * E;                    // tile row bytes
    constexpr bool SPLIT = sizeof(T) == 2;       // two-term P and dS possible (bf16 only)
    using RT = async_tile<64, RB, 2, true, E == 2>;      // Q, dO rows (slot-swapped)
    __shared__ __align__(1024) char q_lds[2][RT::BYTES];
    __shared__ __align__(1024) char o_lds[2][RT::BYTES];
    __shared__ __align__(1024) float st_lds[2][128];   // 64 scaled LSE, then 64 -Delta

    const int tid = threadIdx.x, lane = tid & 63, wave = wave_id(), half = lane >> 5;
    const int64_t krow = work_row(order, xcd_item(blockIdx.x, gridDim.x), gridDim.x);   // (b*Hkv + hkv)*N + nk
    const int64_t bkv = krow / N;
    const int nk = static_cast<int>(krow % N);
    const int b = static_cast<int>(bkv / Hkv), hkv = static_cast<int>(bkv % Hkv);
    const int grp = Hq / Hkv;
    const int64_t L = static_cast<int64_t>(N) * 64;
    const int64_t ktok = bkv * L + static_cast<int64_t>(nk) * 64 + wave * 32 + (lane & 31);
    bool k_real = true;
    if constexpr (PAD) k_real = (cube_real_mask(grid, nk, lane) >> (wave * 32 + (lane & 31))) & 1;

    int64_t e0 = kv_ptr[krow], e1 = kv_ptr[krow + 1];
    e0 = e0 < 0 ? 0 : (e0 > col_cap ? col_cap : e0);
    e1 = e1 < e0 ? e0 : (e1 > col_cap ? col_cap : e1);

    // K and V rows of this lane's key as B operands (column = key, k = d)
    F kf[KS], vf[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
        load_frag(kf[ks], k + ktok * D + ks * 16 + half * 8);
        load_frag(vf[ks], v + ktok * D + ks * 16 + half * 8);
    }
    f32x16_t acc_v[MT], acc_k[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int i = 0; i < 16; ++i) { acc_v[mt][i] = 0.f; acc_k[mt][i] = 0.f; }

    // query-block row of entry value ent ((b*Hq + h)*N + n_q), or -1 for a
    // malformed entry; its first token is row * 64
    const int64_t qrow0 = (static_cast<int64_t>(b) * Hq + hkv * grp) * N;
    const int ent_end = grp * N;
    auto qrow_of = [&](int ent) -> int64_t {
        if (ent < 0 || ent >= ent_end) return -1;
        return qrow0 + ent;
    };
    // two-term operands on every pair of a flagged key block; otherwise P on
    // the pairs whose query block is flagged and dS on the pairs whose query
    // block has the row flag (per-pair flags are read only when some query
    // block of the KV group has the row flag, which its own flag implies)
    bool all_big = false, some_big = false;
    if constexpr (SPLIT) {
        all_big = byte_of(scalar_load_i32(byte_word(fl.kv, krow)), krow);
        some_big = !all_big && scalar_load_i32(fl.any_row + bkv) != 0;
    }
    const RT rt(wave, lane);
    // Q, dO and the statistics of the 64 queries of query-block row qr (512
    // bytes, 16 lanes of each wave)
    auto issue = [&](int64_t qr, int buf) {
        const int64_t o0 = qr < 0 ? 0 : qr * 64;
        rt.issue(q_lds[buf], reinterpret_cast<const char*>(q + o0 * D), wave);
        rt.issue(o_lds[buf], reinterpret_cast<const char*>(dout + o0 * D), wave);
        if (lane < 16)
            dma16(static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_void_t*)st_lds[buf])) + wave * 256,
                  reinterpret_cast<const char*>(stat + 2 * o0) + wave * 256, lane * 16);
    };

#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {   // fragments in registers before the copies start
        settle(kf[ks]);
        settle(vf[ks]);
    }
    // With 256-byte rows and up, the K, V fragments stay in AGPRs for the
    // whole walk (the MFMAs read them there; in VGPRs the accumulators would
    // push them out and every use would copy them back).  Smaller ones fit
    // in VGPRs next to everything else.
    if constexpr (RB >= 256) {
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            pin_agpr(kf[ks]);
            pin_agpr(vf[ks]);
        }
    }
    // Ascending sweep over the query blocks (values hq_local*N + n_q).  With
    // the longest-first order of the key blocks, the workgroups resident
    // together have lists of about the same length and move through the
    // query range together, so the Q / dO tiles they gather are shared
    // through L2 (measured at 720p: 122 GB of L2 misses; 164 GB with the
    // phased start of the query-stationary kernels, which needs equal
    // lengths from rows that are not reordered).
    const int64_t cnt = e1 - e0;
    auto entry = [&](int64_t j) -> int64_t { return e0 + j; };
    int64_t q_cur = -1;
    if (cnt > 0) {
        q_cur = qrow_of(scalar_load_i32(kv_idx + entry(0)));
        issue(q_cur, 0);
    }
    // The walk over the list, in three versions: a flagged key block takes
    // two-term P and dS on every pair (no flag reads, no branches); FL (some
    // pair may touch a large-magnitude block or a flagged row) reads per-pair
    // flags and branches to the two-term steps; the third has neither, so
    // its pipeline is scheduled as one piece.
    auto walk = [&](auto mode) {
        constexpr int MODE = decltype(mode)::value;
        constexpr bool FL = MODE == 1;
        for (int64_t j = 0; j < cnt; ++j) {
            const int buf = static_cast<int>(j & 1);
            const bool has_next = j + 1 < cnt;
            // the next list entry, and the current query block's flags with it
            int64_t q_next = -1;
            bool big_p = FL && all_big, big_s = FL && all_big;
            if (FL && some_big && q_cur >= 0) {
                int32_t ent = -1, w = 0;
                if (has_next) scalar_load2_i32(kv_idx + entry(j + 1), byte_word(fl.qrow, q_cur), ent, w);
                else w = scalar_load_i32(byte_word(fl.qrow, q_cur));
                q_next = has_next ? qrow_of(ent) : -1;
                const int code = byte_val(w, q_cur);
                big_p = (code & 1) != 0;
                big_s = (code & 2) != 0;
            } else if (has_next) {
                q_next = qrow_of(scalar_load_i32(kv_idx + entry(j + 1)));
            }
            // One barrier per block: after it, this block's copies (the only
            // ones outstanding) are visible and both waves are done with the
            // previous block, whose buffer then receives the next block's copies.
            vm_wait<0>();
            wg_barrier();
            if (has_next) issue(q_next, buf ^ 1);
            const char* qt = q_lds[buf];
            const char* ot = o_lds[buf];
            const float* st = st_lds[buf];
            // Software pipeline over the two 32-query tiles of the block:
            //   S/dP(tile 0) | S/dP(tile 1) + P,dS(tile 0) |
            //   dV/dK(tile 0) + P,dS(tile 1) | dV/dK(tile 1)
            // so the exponentials and the dS arithmetic of one tile issue
            // while the other tile's MFMAs run (one wave per SIMD: the wave's
            // own independent work is all there is to overlap).  LDS operand
            // fragments are requested one step ahead of their MFMAs;
            // lds_order keeps the compiler from moving work across steps.
            // two_p, two_s (wave-uniform): P (dS) as hi + lo, a second dV (dK)
            // product with the lo terms.  One code path with the lo steps behind
            // scalar branches: inlined variants of the loop raise the kernel's
            // register allocation for all of them.
            auto pair = [&](bool two_p, bool two_s) {
                constexpr int NB = KS / 2;           // S/dP steps per tile (2 k-steps each)
                constexpr int NU = 2 * MT;           // dV/dK steps per tile
                constexpr int EV = 16 / NB;          // P,dS elements per S/dP step
                constexpr int EU = 16 / NU;          // P,dS elements per dV/dK step
                // S starts from 0; dP starts from -Delta of its query (element i
                // of tile t is query 32t + 16(i/8) + 8half + i%8), so the product
                // leaves dP - Delta
                f32x16_t s[2], dp[2];
    #pragma unroll
                for (int t = 0; t < 2; ++t)
    #pragma unroll
                    for (int i = 0; i < 16; ++i) s[t][i] = 0.f;
                auto dp_init = [&](int t) {
    #pragma unroll
                    for (int i = 0; i < 16; ++i) dp[t][i] = st[64 + t * 32 + (i >> 3) * 16 + half * 8 + (i & 7)];
                };
                dp_init(0);
                F pb[2][2], db[2][2], pl[2][SPLIT ? 2 : 1], dl[2][SPLIT ? 2 : 1];
                // scaled LSE of the elements of softmax_grad call c (calls
                // 0..NB-1: tile 0 in groups of EV; NB..NB+NU-1: tile 1 in groups
                // of EU), read one step ahead into a double buffer
                constexpr int EMAX = EV > EU ? EV : EU;
                float stv[2][EMAX];
                auto st_load = [&](int c) {
                    const int t = c < NB ? 0 : 1;
                    const int i0 = c < NB ? c * EV : (c - NB) * EU;
                    const int n = c < NB ? EV : EU;
    #pragma unroll
                    for (int i = i0; i < i0 + n; ++i) stv[c & 1][i - i0] = st[t * 32 + (i >> 3) * 16 + half * 8 + (i & 7)];
                };
                // P and dS of elements [i0, i0 + n) of tile t, in place (s <- P,
                // dp <- dS); element i is query 32t + 16(i/8) + 8half + i%8.
                // A group of 8 finished elements becomes a fragment pair.
                auto softmax_grad = [&](int t, int i0, int n) {
                    const int c = t == 0 ? i0 / EV : NB + i0 / EU;
                    if (c + 1 < NB + NU) st_load(c + 1);
    #pragma unroll
                    for (int i = i0; i < i0 + n; ++i) {
                        const float pv = fast_exp2(s[t][i] * c_log2 - stv[c & 1][i - i0]);
                        s[t][i] = pv;
                        dp[t][i] = pv * dp[t][i];
                    }
                    if (((i0 + n) & 7) == 0) {
                        const int h = (i0 + n - 1) >> 3;
                        float xp[8], xd[8];
    #pragma unroll
                        for (int i = 0; i < 8; ++i) { xp[i] = s[t][8 * h + i]; xd[i] = dp[t][8 * h + i]; }
                        if (SPLIT && two_p) pack_frag_hilo(pb[t][h], pl[t][SPLIT ? h : 0], xp);
                        else pack_frag(pb[t][h], xp);
                        if (SPLIT && two_s) pack_frag_hilo(db[t][h], dl[t][SPLIT ? h : 0], xd);
                        else pack_frag(db[t][h], xd);
                    }
                };
                F fa[2][4];
                auto fetch_sd = [&](F* f, int t, int bi) {
                    const int row = t * 32 + (lane & 31);
                    lds_frag_s<RB>(f[0], qt, row, 32 * bi + half * 8);
                    lds_frag_s<RB>(f[1], ot, row, 32 * bi + half * 8);
                    lds_frag_s<RB>(f[2], qt, row, 32 * bi + 16 + half * 8);
                    lds_frag_s<RB>(f[3], ot, row, 32 * bi + 16 + half * 8);
                };
                F ta[2][2];
                auto fetch_dk = [&](F* f, int t, int u) {
                    const int kk = 2 * t + u / MT, mt = u % MT;
                    lds_frag_tr<RB, true>(f[0], ot, mt * 32, kk * 16);
                    lds_frag_tr<RB, true>(f[1], qt, mt * 32, kk * 16);
                };
                // S = Q K^T and dP = dO V^T, both tiles
                fetch_sd(fa[0], 0, 0);
    #pragma unroll
                for (int k = 0; k < 2 * NB; ++k) {
                    const int t = k / NB, bi = k % NB;
                    if (k + 1 < 2 * NB) fetch_sd(fa[(k + 1) & 1], (k + 1) / NB, (k + 1) % NB);
                    else fetch_dk(ta[0], 0, 0);
                    if (k == NB - 1) dp_init(1);
                    lds_order();
                    mma(s[t], fa[k & 1][0], kf[2 * bi]);
                    mma(dp[t], fa[k & 1][1], vf[2 * bi]);
                    mma(s[t], fa[k & 1][2], kf[2 * bi + 1]);
                    mma(dp[t], fa[k & 1][3], vf[2 * bi + 1]);
                    if (k == NB - 1) st_load(0);
                    if (t == 1) softmax_grad(0, bi * EV, EV);
                }
                // dV^T += dO^T P and dK^T += Q^T dS, tile by tile (dO^T and Q^T
                // read transposed from the row-major tiles)
    #pragma unroll
                for (int k = 0; k < 2 * NU; ++k) {
                    const int t = k / NU, u = k % NU;
                    if (k + 1 < 2 * NU) fetch_dk(ta[(k + 1) & 1], (k + 1) / NU, (k + 1) % NU);
                    lds_order();
                    const int h = u / MT, mt = u % MT;
                    mma(acc_v[mt], ta[k & 1][0], pb[t][h]);
                    if (SPLIT && two_p) mma(acc_v[mt], ta[k & 1][0], pl[t][SPLIT ? h : 0]);
                    mma(acc_k[mt], ta[k & 1][1], db[t][h]);
                    if (SPLIT && two_s) mma(acc_k[mt], ta[k & 1][1], dl[t][SPLIT ? h : 0]);
                    if (t == 0) softmax_grad(1, u * EU, EU);
                }
            };
            if (q_cur >= 0) {
                if constexpr (MODE == 2) pair(true, true);
                else pair(FL && big_p, FL && big_s);
            }
            q_cur = q_next;
        }
    };
    if (SPLIT && all_big) walk(std::integral_constant<int, 2>{});
    else if (SPLIT && some_big) walk(std::integral_constant<int, 1>{});
    else walk(std::integral_constant<int, 0>{});

    // lane holds key column (lane & 31) and d = 32mt + 8(v/4) + 4half + v%4
    T* krow_k = dk + ktok * D;
    T* krow_v = dv + ktok * D;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
            const int d0 = mt * 32 + g4 * 8 + half * 4;
            float av[4], kx[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                av[i] = k_real ? acc_v[mt][g4 * 4 + i] : 0.f;
                kx[i] = k_real ? acc_k[mt][g4 * 4 + i] * scale : 0.f;
            }
            if constexpr (E == 2) {
                *reinterpret_cast<uint2*>(krow_v + d0) =
                    make_uint2(pack2_bf16(av[0], av[1]), pack2_bf16(av[2], av[3]));
                *reinterpret_cast<uint2*>(krow_k + d0) =
                    make_uint2(pack2_bf16(kx[0], kx[1]), pack2_bf16(kx[2], kx[3]));
            } else {
                *reinterpret_cast<float4*>(krow_v + d0) = make_float4(av[0], av[1], av[2], av[3]);
                *reinterpret_cast<float4*>(krow_k + d0) = make_float4(kx[0], kx[1], kx[2], kx[3]);
            }
        }
}

// ---------------------------------------------------------------------------
// dQ: one workgroup (2 waves) per query block; wave owns 32 queries.
// Tiles K (for S^T and, read transposed, K^T) and V (for dP^T).  On a
// padded grid, padding keys get P = 0 and padding queries dQ = 0 (PAD
// variant only).  bf16: when this query block's row touches a
// large-magnitude block (its own flag or a listed key block's) or one of
// its queries has |Delta| above DELTA_FLAG, dS enters every dQ product of
// the row as two bf16 terms (hi + lo).
// ---------------------------------------------------------------------------
template <typename T, int D, bool PAD>
__global__ __launch_bounds__(AB_NT, 2) void dq_kernel(
    const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ v,
    const T* __restrict__ dout, const float* __restrict__ stat,
    const int32_t* __restrict__ row_ptr, const int32_t* __restrict__ col_idx, int64_t col_cap,
    T* __restrict__ dq, int Hq, int Hkv, int N, float c_log2, float scale, int period,
    const int32_t* __restrict__ order, cube_grid grid, block_flag_layout fl) {
    using F = typename frag_of<T>::type;
    constexpr int E = sizeof(T);
    constexpr int KS = D / 16;
    constexpr int MT = D / 32;
    constexpr int RB = D * E;
    constexpr bool SPLIT = sizeof(T) == 2;       // two-term dS possible (bf16 only)
    using RT = async_tile<64, RB, 2, true, E == 2>;     // K, V rows (slot-swapped)
    __shared__ __align__(1024) char k_lds[RT::BYTES];
    __shared__ __align__(1024) char v_lds[RT::BYTES];

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

    F qf[KS], of[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
        load_frag(qf[ks], q + qtok * D + ks * 16 + half * 8);
        load_frag(of[ks], dout + qtok * D + ks * 16 + half * 8);
    }
    if constexpr (PAD) {
        if (!q_real) {          // a padding query computes with zero vectors
            const float z[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                pack_frag(qf[ks], z);
                pack_frag(of[ks], z);
            }
        }
    }
    const float st_lse = stat[stat_lse_at(qtok)], st_nd = stat[stat_nd_at(qtok)];   // LSE log2 e, -Delta
    f32x16_t dqa[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int i = 0; i < 16; ++i) dqa[mt][i] = 0.f;

    auto block_of = [&](int64_t e) -> int {
        const int c = scalar_load_i32(col_idx + e);
        return (c >= 0 && c < N) ? c : -1;
    };
    // two-term dS on every pair of a row that touches a flagged block or
    // has a large Delta: the query block's own flag, else a query of the
    // block with |Delta| above DELTA_FLAG (and attention mass: scaled LSE
    // below +inf), else (only when the head holds a flagged key block) a
    // scan of the listed key blocks' flags, 64 entries per step.  Both waves
    // read the same values, so the decision is the workgroup's.
    const int64_t kvrow0 = static_cast<int64_t>(b * Hkv + hkv) * N;
    bool big = false;
    if constexpr (SPLIT) {
        big = byte_of(scalar_load_i32(byte_word(fl.q, row)), row);
        if (!big) {
            const float ls = stat[row * 128 + lane], nd = stat[row * 128 + 64 + lane];
            big = __any(ls != INFINITY && fabsf(nd) > DELTA_FLAG);
        }
        if (!big && scalar_load_i32(fl.any_kv + b * Hkv + hkv) != 0) {
            bool hit = false;
            for (int64_t e = e0 + lane; e < e1; e += 64) {
                const int c = col_idx[e];
                if (c >= 0 && c < N && fl.kv[kvrow0 + c]) hit = true;
            }
            big = __any(hit);
        }
    }
    constexpr int64_t TILE = 64 * RB;
    const RT rt(wave, lane);
    auto issue_k = [&](int c) { rt.issue(k_lds, kb + static_cast<int64_t>(c < 0 ? 0 : c) * TILE, wave); };
    auto issue_v = [&](int c) { rt.issue(v_lds, vb + static_cast<int64_t>(c < 0 ? 0 : c) * TILE, wave); };

#pragma unroll
    for (int ks = 0; ks < KS; ++ks) { settle(qf[ks]); settle(of[ks]); }   // before the copies start
    settle(st_lse);
    settle(st_nd);
    const int64_t cnt = e1 - e0;
    const int64_t s0 = sweep_start(col_idx, e0, cnt, blockIdx.x >> 3, period, N);
    auto entry = [&](int64_t j) -> int64_t {
        const int64_t t = s0 + j;
        return e0 + (t >= cnt ? t - cnt : t);
    };
    int c_cur = -1;
    if (cnt > 0) {
        c_cur = block_of(entry(0));
        issue_k(c_cur);
        issue_v(c_cur);
    }
    for (int64_t j = 0; j < cnt; ++j) {
        const bool has_next = j + 1 < cnt;
        const int c_next = has_next ? block_of(entry(j + 1)) : -1;

        vm_wait<0>();                   // K and V landed
        wg_barrier();
        // padding keys of a cut cube (bit = key within the block)
        const uint64_t kmask = PAD && c_cur >= 0 ? cube_real_mask(grid, c_cur, lane) : ~0ull;
        F sb[2][2];
        F sl[SPLIT ? 2 : 1][2];
#pragma unroll
        for (int t2 = 0; t2 < 2; ++t2) {
            // S^T = K Q^T, dP^T = V dO^T: 32 keys x this lane's query; K and V
            // fragments requested one k-step pair ahead of their products
            const int row = t2 * 32 + (lane & 31);
            // dP^T starts at -Delta (this lane's query), so the products
            // accumulate dP - Delta directly
            f32x16_t s, dp;
#pragma unroll
            for (int i = 0; i < 16; ++i) { s[i] = 0.f; dp[i] = st_nd; }
            F fa[2][4];
            auto fetch = [&](F* f, int bi) {
                lds_frag_s<RB>(f[0], k_lds, row, 32 * bi + half * 8);
                lds_frag_s<RB>(f[1], v_lds, row, 32 * bi + half * 8);
                lds_frag_s<RB>(f[2], k_lds, row, 32 * bi + 16 + half * 8);
                lds_frag_s<RB>(f[3], v_lds, row, 32 * bi + 16 + half * 8);
            };
            fetch(fa[0], 0);
#pragma unroll
            for (int bi = 0; bi < KS / 2; ++bi) {
                if (bi + 1 < KS / 2) fetch(fa[(bi + 1) & 1], bi + 1);
                lds_order();
                mma(s, fa[bi & 1][0], qf[2 * bi]);
                mma(dp, fa[bi & 1][1], of[2 * bi]);
                mma(s, fa[bi & 1][2], qf[2 * bi + 1]);
                mma(dp, fa[bi & 1][3], of[2 * bi + 1]);
            }
            float ds[16];
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const float p = fast_exp2(s[i] * c_log2 - st_lse);
                ds[i] = p * dp[i];
            }
            if constexpr (PAD) {        // branch-free: a branch here costs registers
                const uint32_t lm = static_cast<uint32_t>(kmask >> (t2 * 32 + half * 8));
#pragma unroll
                for (int i = 0; i < 16; ++i) ds[i] = ((lm >> ((i >> 3) * 16 + (i & 7))) & 1u) ? ds[i] : 0.f;
            }
            if (SPLIT && big) {
                pack_frag_hilo(sb[t2][0], sl[SPLIT ? t2 : 0][0], ds);
                pack_frag_hilo(sb[t2][1], sl[SPLIT ? t2 : 0][1], ds + 8);
            } else {
                pack_frag(sb[t2][0], ds);
                pack_frag(sb[t2][1], ds + 8);
            }
        }
        wg_barrier();                   // V buffer free: stream the next one during dQ
        if (has_next) issue_v(c_next);
        if (c_cur >= 0) {
            // dQ^T += K^T dS^T over the 64 keys (4 k-steps of 16); K^T read
            // transposed, one k-step ahead of its products.  On a flagged
            // pair a second pass adds K^T times the lo terms of dS.
            auto dq_product = [&](F (*sf)[2]) {
                F fa[2][MT];
                auto fetch = [&](F* f, int kk) {
#pragma unroll
                    for (int mt = 0; mt < MT; ++mt) lds_frag_tr<RB, true>(f[mt], k_lds, mt * 32, kk * 16);
                };
                fetch(fa[0], 0);
#pragma unroll
                for (int kk = 0; kk < 4; ++kk) {
                    if (kk + 1 < 4) fetch(fa[(kk + 1) & 1], kk + 1);
                    lds_order();
#pragma unroll
                    for (int mt = 0; mt < MT; ++mt) mma(dqa[mt], fa[kk & 1][mt], sf[kk >> 1][kk & 1]);
                }
            };
            dq_product(sb);
            if constexpr (SPLIT) {
                if (big) dq_product(sl);
            }
        }
        wg_barrier();                   // K buffer free
        if (has_next) issue_k(c_next);
        c_cur = c_next;
    }
    T* dqrow = dq + qtok * D;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
            const int d0 = mt * 32 + g4 * 8 + half * 4;
            float x[4];                                    // a padding query has dQ = 0
#pragma unroll
            for (int i = 0; i < 4; ++i) x[i] = q_real ? dqa[mt][g4 * 4 + i] * scale : 0.f;
            if constexpr (E == 2) {
                *reinterpret_cast<uint2*>(dqrow + d0) = make_uint2(pack2_bf16(x[0], x[1]), pack2_bf16(x[2], x[3]));
            } else {
                *reinterpret_cast<float4*>(dqrow + d0) = make_float4(x[0], x[1], x[2], x[3]);
            }
        }
}

// Workspace of the backward call: per query token LSE * log2(e) and -Delta,
// then the work orders of the CSR rows (dQ) and of the CSC rows (dK/dV),
// then the block magnitude flags.
static size_t align256(size_t x) { return (x + 255) / 256 * 256; }

size_t bwd_ws_csr_order_offset(int batch, int Hq, int N) {
    return align256(8 * static_cast<size_t>(batch) * Hq * N * 64);
}

size_t bwd_ws_csc_order_offset(int batch, int Hq, int N) {
    return bwd_ws_csr_order_offset(batch, Hq, N) + align256(4 * static_cast<size_t>(batch) * Hq * N);
}

static size_t bwd_ws_flags_offset(int batch, int Hq, int Hkv, int N) {
    return bwd_ws_csc_order_offset(batch, Hq, N) + align256(4 * static_cast<size_t>(batch) * Hkv * N);
}

static block_flag_layout bwd_flags(void* ws, int batch, int Hq, int Hkv, int N) {
    return block_flags_at(static_cast<char*>(ws) + bwd_ws_flags_offset(batch, Hq, Hkv, N),
                          static_cast<int64_t>(batch) * Hq * N, static_cast<int64_t>(batch) * Hkv * N,
                          static_cast<int64_t>(batch) * Hkv);
}

size_t bwd_workspace_bytes(int dtype, int D, int batch, int Hq, int Hkv, int N) {
    (void)dtype;
    (void)D;
    return bwd_ws_flags_offset(batch, Hq, Hkv, N) +
           block_flags_bytes(static_cast<int64_t>(batch) * Hq * N, static_cast<int64_t>(batch) * Hkv * N,
                             static_cast<int64_t>(batch) * Hkv);
}

// Stage 1: per query token LSE * log2(e) and -Delta into ws.
template <typename T, int D>
static hipError_t launch_prep_t(const void* o, const float* lse, const void* o_lo, const void* dout, void* ws,
                                int64_t ntok, hipStream_t s) {
    if (ntok == 0) return hipSuccess;
    const int64_t sthreads = ntok * (D / 8);
    hipLaunchKernelGGL((stat_kernel<T, D>), dim3(static_cast<unsigned>((sthreads + 255) / 256)), dim3(256), 0,
                       s, static_cast<const T*>(o), static_cast<const T*>(o_lo), static_cast<const T*>(dout),
                       lse, static_cast<float*>(ws), ntok);
    return hipGetLastError();
}

// Stage 2: dK and dV (key-block stationary, transposed lists).
template <typename T, int D>
static hipError_t launch_dkdv_t(const void* q, const void* k, const void* v, const void* dout,
                                const int32_t* kv_ptr, const int32_t* kv_idx, int64_t col_cap, void* dk,
                                void* dv, void* ws, int batch, int Hq, int Hkv, int N, const cube_grid& cg,
                                hipStream_t s) {
    const int64_t krows = static_cast<int64_t>(batch) * Hkv * N;
    if (krows == 0) return hipSuccess;
    int32_t* order = reinterpret_cast<int32_t*>(static_cast<char*>(ws) + bwd_ws_csc_order_offset(batch, Hq, N));
    hipError_t e = launch_lpt_order(kv_ptr, krows, N, col_cap, order, s);
    if (e != hipSuccess) return e;
    const float c = kLog2e / sqrtf(static_cast<float>(D));
    const float scale = 1.0f / sqrtf(static_cast<float>(D));
    const block_flag_layout fl = bwd_flags(ws, batch, Hq, Hkv, N);
    if constexpr (sizeof(T) == 2) {   // the row flags of the query blocks (two-term dS)
        e = launch_row_flags(fl, static_cast<const float*>(ws), kv_ptr, kv_idx, col_cap,
                             static_cast<int64_t>(batch) * Hq * N, krows, N, Hq, Hkv, s);
        if (e != hipSuccess) return e;
    }
    auto go = [&](auto pad) {
        hipLaunchKernelGGL((dkdv_kernel<T, D, decltype(pad)::value>), dim3(static_cast<unsigned>(krows)),
                           dim3(AB_NT), 0, s, static_cast<const T*>(q), static_cast<const T*>(k),
                           static_cast<const T*>(v), static_cast<const T*>(dout), static_cast<const float*>(ws),
                           kv_ptr, kv_idx, col_cap, static_cast<T*>(dk), static_cast<T*>(dv), Hq, Hkv, N, c, scale,
                           order, cg, fl);
    };
    if (cg.padded) go(std::true_type{}); else go(std::false_type{});
    return hipGetLastError();
}

// Stage 3: dQ (query-block stationary, CSR rows).
template <typename T, int D>
static hipError_t launch_dq_t(const void* q, const void* k, const void* v, const void* dout,
                              const int32_t* row_ptr, const int32_t* col_idx, int64_t col_cap, void* dq,
                              void* ws, int batch, int Hq, int Hkv, int N, const cube_grid& cg, hipStream_t s) {
    const int64_t qrows = static_cast<int64_t>(batch) * Hq * N;
    if (qrows == 0) return hipSuccess;
    int32_t* order = reinterpret_cast<int32_t*>(static_cast<char*>(ws) + bwd_ws_csr_order_offset(batch, Hq, N));
    hipError_t e = launch_lpt_order(row_ptr, qrows, N, col_cap, order, s);
    if (e != hipSuccess) return e;
    const float c = kLog2e / sqrtf(static_cast<float>(D));
    const float scale = 1.0f / sqrtf(static_cast<float>(D));
    const block_flag_layout fl = bwd_flags(ws, batch, Hq, Hkv, N);
    auto go = [&](auto pad) {
        constexpr bool P = decltype(pad)::value;
        hipLaunchKernelGGL((dq_kernel<T, D, P>), dim3(static_cast<unsigned>(qrows)), dim3(AB_NT), 0, s,
                           static_cast<const T*>(q), static_cast<const T*>(k), static_cast<const T*>(v),
                           static_cast<const T*>(dout), static_cast<const float*>(ws), row_ptr, col_idx, col_cap,
                           static_cast<T*>(dq), Hq, Hkv, N, c, scale,
                           resident_per_xcd<dq_kernel<T, D, P>>(AB_NT), order, cg, fl);
    };
    if (cg.padded) go(std::true_type{}); else go(std::false_type{});
    return hipGetLastError();
}

#define VSA2_DISPATCH_TD(...)                               \
    if (dtype == 1) {                                       \
        if (D == 64) { using T = bf16_t; constexpr int DD = 64; __VA_ARGS__; }   \
        if (D == 128) { using T = bf16_t; constexpr int DD = 128; __VA_ARGS__; } \
    } else {                                                \
        if (D == 64) { using T = float; constexpr int DD = 64; __VA_ARGS__; }    \
        if (D == 128) { using T = float; constexpr int DD = 128; __VA_ARGS__; }  \
    }                                                       \
    return hipErrorInvalidValue

hipError_t launch_attn_bwd_prep_tokens(int dtype, int D, const void* o, const float* lse, const void* o_lo,
                                       const void* dout, void* ws, int64_t ntok, hipStream_t s) {
    VSA2_DISPATCH_TD(return (launch_prep_t<T, DD>(o, lse, o_lo, dout, ws, ntok, s)));
}

// Stage 1 of the backward: the per-token statistics and (bf16) the block
// magnitude flags of Q, K, V.
hipError_t launch_attn_bwd_prep(int dtype, int D, const void* q, const void* k, const void* v, const void* o,
                                const float* lse, const void* o_lo, const void* dout, void* ws, int batch, int Hq,
                                int Hkv, int N, const cube_grid& cg, hipStream_t s) {
    hipError_t e = launch_attn_bwd_prep_tokens(dtype, D, o, lse, o_lo, dout, ws,
                                               static_cast<int64_t>(batch) * Hq * N * 64, s);
    if (e != hipSuccess || dtype != 1) return e;
    return launch_block_flags(q, k, v, bwd_flags(ws, batch, Hq, Hkv, N), static_cast<int64_t>(batch) * Hq * N,
                              static_cast<int64_t>(batch) * Hkv * N, N, D, Hq, Hkv, cg, s);
}

hipError_t launch_attn_bwd_dkdv(int dtype, int D, const void* q, const void* k, const void* v,
                                const void* dout, const int32_t* kv_ptr, const int32_t* kv_idx, int64_t col_cap,
                                void* dk, void* dv, void* ws, int batch, int Hq, int Hkv, int N,
                                const cube_grid& cg, hipStream_t s) {
    VSA2_DISPATCH_TD(return (launch_dkdv_t<T, DD>(q, k, v, dout, kv_ptr, kv_idx, col_cap, dk, dv, ws, batch, Hq,
                                                  Hkv, N, cg, s)));
}

hipError_t launch_attn_bwd_dq(int dtype, int D, const void* q, const void* k, const void* v,
                              const void* dout, const int32_t* row_ptr, const int32_t* col_idx, int64_t col_cap,
                              void* dq, void* ws, int batch, int Hq, int Hkv, int N, const cube_grid& cg,
                              hipStream_t s) {
    VSA2_DISPATCH_TD(return (launch_dq_t<T, DD>(q, k, v, dout, row_ptr, col_idx, col_cap, dq, ws, batch, Hq, Hkv,
                                                N, cg, s)));
}
#undef VSA2_DISPATCH_TD

// The whole backward: prep, dK/dV, dQ on one stream.
hipError_t launch_attn_bwd(int dtype, int D, const void* q, const void* k, const void* v, const void* o,
                           const float* lse, const void* o_lo, const void* dout, const int32_t* row_ptr,
                           const int32_t* col_idx, const int32_t* kv_ptr, const int32_t* kv_idx,
                           int64_t col_cap, void* dq, void* dk, void* dv, void* ws, int batch,
                           int Hq, int Hkv, int N, const cube_grid& cg, hipStream_t s) {
    hipError_t e = launch_attn_bwd_prep(dtype, D, q, k, v, o, lse, o_lo, dout, ws, batch, Hq, Hkv, N, cg, s);
    if (e != hipSuccess) return e;
    e = launch_attn_bwd_dkdv(dtype, D, q, k, v, dout, kv_ptr, kv_idx, col_cap, dk, dv, ws, batch, Hq, Hkv, N, cg,
                             s);
    if (e != hipSuccess) return e;
    return launch_attn_bwd_dq(dtype, D, q, k, v, dout, row_ptr, col_idx, col_cap, dq, ws, batch, Hq, Hkv, N, cg,
                              s);
}

}  // namespace vsa2
