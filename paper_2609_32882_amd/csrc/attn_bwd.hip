// Block-sparse attention backward for gfx950.  The block mask is a constant
// (routing carries no gradient, VSA2 Sec. 2.1), so the gradients are those of
// masked softmax attention restricted to the selected block pairs:
//   Delta_l = dO_l . O_l
//   P = exp(S/sqrt(D) - LSE),  dP = dO V^T,  dS = P o (dP - Delta)
//   dV = P^T dO,  dK = dS^T Q / sqrt(D),  dQ = dS K / sqrt(D)
// Kernels, all deterministic (no atomics):
//   stat_kernel      per query token: (LSE * log2(e), Delta)
//   block transposes Q^T, dO^T and K^T per 64-token block (workspace)
//   dkdv_kernel      key-block stationary: one workgroup per key block walks
//                    the transposed (CSC) list of query blocks that selected
//                    it; a wave owns 32 keys; one launch accumulates dV^T,
//                    a second dK^T, in registers
//   dq_kernel        query-block stationary: one workgroup per query block
//                    walks its CSR row; a wave owns 32 queries
// Products are arranged so that each lane owns one column (a key in dkdv, a
// query in dq) and its 16 accumulator rows form two runs of 8 consecutive
// rows (tiles stored with the bit-2/3 slot swap): a lane's P / dS values are
// directly the B operand of the next MFMA.  Tiles stream into LDS with
// global_load_lds; each buffer is refilled as soon as its last reader is done.
#include "common.hpp"
#include "internal.hpp"

namespace vsa2 {

constexpr int AB_NT = 128;
constexpr float kLog2e = 1.4426950408889634f;

// ---------------------------------------------------------------------------
// stat[l] = (LSE_l * log2(e), dO_l . O_l); 16 lanes per token (D <= 128).
// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ __launch_bounds__(256) void stat_kernel(const T* __restrict__ o, const T* __restrict__ dout,
                                                   const float* __restrict__ lse, float2* __restrict__ stat,
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
    }
#pragma unroll
    for (int off = LPT / 2; off >= 1; off >>= 1) s += __shfl_xor(s, off, 64);
    if (tok < ntok && part == 0) stat[tok] = make_float2(lse[tok] * kLog2e, s);
}

// ---------------------------------------------------------------------------
// dV (GRAD = 0) or dK (GRAD = 1): one workgroup (2 waves) per key block of
// head (b, hkv); a wave owns 32 keys.  The two gradients run as separate
// launches so each keeps one accumulator set (64 registers) and two waves
// fit per SIMD; the price is recomputing S once more per block pair.
//   dV^T += dO^T P            (tiles: Q rows for S, dO^T)
//   dK^T += Q^T dS            (tiles: Q and dO rows for S and dP, Q^T)
// ---------------------------------------------------------------------------
template <typename T, int D, int GRAD>
__global__ __launch_bounds__(AB_NT, 2) void dkdv_kernel(
    const T* __restrict__ q, const T* __restrict__ qt, const T* __restrict__ k, const T* __restrict__ v,
    const T* __restrict__ dout, const T* __restrict__ doutt, const float2* __restrict__ stat,
    const int32_t* __restrict__ kv_ptr, const int32_t* __restrict__ kv_idx, int64_t col_cap,
    T* __restrict__ dgrad, int Hq, int Hkv, int N, float c_log2, float scale) {
    using F = typename frag_of<T>::type;
    constexpr int E = sizeof(T);
    constexpr int KS = D / 16;
    constexpr int MT = D / 32;
    constexpr int RRB = D * E;      // row-major tile row bytes
    constexpr int TRB = 64 * E;     // transposed tile row bytes
    using RT = async_tile<64, RRB, 2, true>;     // Q, dO rows (slot-swapped)
    using TT = async_tile<D, TRB, 2, false>;     // dO^T (dV) or Q^T (dK)
    __shared__ __align__(1024) char q_lds[RT::BYTES];
    __shared__ __align__(1024) char o_lds[GRAD == 1 ? RT::BYTES : 16];
    __shared__ __align__(1024) char t_lds[TT::BYTES];
    __shared__ __align__(1024) float2 st_lds[64];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, half = lane >> 5;
    const int64_t krow = blockIdx.x;                 // (b*Hkv + hkv)*N + nk
    const int64_t bkv = krow / N;
    const int nk = static_cast<int>(krow % N);
    const int b = static_cast<int>(bkv / Hkv), hkv = static_cast<int>(bkv % Hkv);
    const int grp = Hq / Hkv;
    const int64_t L = static_cast<int64_t>(N) * 64;
    const int64_t ktok = bkv * L + static_cast<int64_t>(nk) * 64 + wave * 32 + (lane & 31);

    int64_t e0 = kv_ptr[krow], e1 = kv_ptr[krow + 1];
    e0 = e0 < 0 ? 0 : (e0 > col_cap ? col_cap : e0);
    e1 = e1 < e0 ? e0 : (e1 > col_cap ? col_cap : e1);

    // K (and for dK also V) rows of this lane's key as B operands (column = key, k = d)
    F kf[KS], vf[GRAD == 1 ? KS : 1];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
        load_frag(kf[ks], k + ktok * D + ks * 16 + half * 8);
        if constexpr (GRAD == 1) load_frag(vf[ks], v + ktok * D + ks * 16 + half * 8);
    }
    f32x16_t acc[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[mt][i] = 0.f;

    // query-block token offset of entry e, or -1 for a malformed entry
    auto q0_of = [&](int64_t e) -> int64_t {
        const int ent = scalar_load_i32(kv_idx + e);
        const int hl = ent / N;
        if (ent < 0 || hl >= grp) return -1;
        const int64_t bh = static_cast<int64_t>(b) * Hq + hkv * grp + hl;
        return bh * L + static_cast<int64_t>(ent % N) * 64;
    };
    const RT rt(wave, lane);
    const TT tt(wave, lane);
    auto issue_rows = [&](int64_t q0) {
        const int64_t o0 = q0 < 0 ? 0 : q0;
        rt.issue(q_lds, reinterpret_cast<const char*>(q + o0 * D), wave);
        if constexpr (GRAD == 1) rt.issue(o_lds, reinterpret_cast<const char*>(dout + o0 * D), wave);
        // (LSE, Delta) of the 64 queries: 512 bytes, 16 lanes of each wave
        if (lane < 16)
            dma16(static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_void_t*)st_lds)) + wave * 256,
                  reinterpret_cast<const char*>(stat + o0) + wave * 256, lane * 16);
    };
    auto issue_tr = [&](int64_t q0) {
        const int64_t o0 = q0 < 0 ? 0 : q0;
        tt.issue(t_lds, reinterpret_cast<const char*>((GRAD == 1 ? qt : doutt) + o0 * D), wave);
    };
    constexpr int ROWS_OPS = (GRAD == 1 ? 2 : 1) * RT::PER_WAVE + 1;
    constexpr int TR_OPS = TT::PER_WAVE;

#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {   // fragments in registers before the copies start
        settle(kf[ks]);
        if constexpr (GRAD == 1) settle(vf[ks]);
    }
    int64_t q_cur = -1;
    if (e0 < e1) {
        q_cur = q0_of(e0);
        issue_rows(q_cur);
        issue_tr(q_cur);
    }
    for (int64_t e = e0; e < e1; ++e) {
        const bool has_next = e + 1 < e1;
        const int64_t q_next = has_next ? q0_of(e + 1) : -1;
        const bool valid = q_cur >= 0;

        vm_wait<TR_OPS>();              // rows and stats landed
        wg_barrier();
        F fb[2][2];                     // P (dV) or dS (dK) by [query tile][k-step half]
#pragma unroll
        for (int qtile = 0; qtile < 2; ++qtile) {
            // S = Q K^T (and dP = dO V^T) for 32 queries x this lane's key
            f32x16_t s, dp;
#pragma unroll
            for (int i = 0; i < 16; ++i) { s[i] = 0.f; dp[i] = 0.f; }
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                F a;
                lds_frag_s<RRB>(a, q_lds, qtile * 32 + (lane & 31), ks * 16 + half * 8);
                mma(s, a, kf[ks]);
                if constexpr (GRAD == 1) {
                    lds_frag_s<RRB>(a, o_lds, qtile * 32 + (lane & 31), ks * 16 + half * 8);
                    mma(dp, a, vf[ks]);
                    // bound how far the scheduler hoists LDS reads (register pressure)
                    __builtin_amdgcn_sched_barrier(0);
                }
            }
            // entry i is query 32qtile + 16(i/8) + 8half + i%8
            float x[16];
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const float2 st = st_lds[qtile * 32 + (i >> 3) * 16 + half * 8 + (i & 7)];
                const float p = fast_exp2(s[i] * c_log2 - st.x);
                x[i] = GRAD == 1 ? p * (dp[i] - st.y) : p;
            }
            pack_frag(fb[qtile][0], x);
            pack_frag(fb[qtile][1], x + 8);
        }
        wg_barrier();                   // row buffers free
        if (has_next) issue_rows(q_next);
        if (has_next) vm_wait<ROWS_OPS>(); else vm_wait<0>();   // transposed tile landed
        wg_barrier();
        if (valid) {
            // acc^T += X^T F over the 64 queries (4 k-steps), X = dO (dV) or Q (dK)
#pragma unroll
            for (int kk = 0; kk < 4; ++kk)
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) {
                    F a;
                    lds_frag_s<TRB>(a, t_lds, mt * 32 + (lane & 31), kk * 16 + half * 8);
                    mma(acc[mt], a, fb[kk >> 1][kk & 1]);
                    if (GRAD == 1 && mt % 2 == 1) __builtin_amdgcn_sched_barrier(0);
                }
        }
        wg_barrier();                   // transposed buffer free
        if (has_next) issue_tr(q_next);
        q_cur = q_next;
    }

    // lane holds key column (lane & 31) and d = 32mt + 8(v/4) + 4half + v%4
    const float sc = GRAD == 1 ? scale : 1.0f;
    T* grow = dgrad + ktok * D;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
            const int d0 = mt * 32 + g4 * 8 + half * 4;
            if constexpr (E == 2) {
                const uint32_t w0 = pack2_bf16(acc[mt][g4 * 4] * sc, acc[mt][g4 * 4 + 1] * sc);
                const uint32_t w1 = pack2_bf16(acc[mt][g4 * 4 + 2] * sc, acc[mt][g4 * 4 + 3] * sc);
                *reinterpret_cast<uint2*>(grow + d0) = make_uint2(w0, w1);
            } else {
                *reinterpret_cast<float4*>(grow + d0) =
                    make_float4(acc[mt][g4 * 4] * sc, acc[mt][g4 * 4 + 1] * sc, acc[mt][g4 * 4 + 2] * sc,
                                acc[mt][g4 * 4 + 3] * sc);
            }
        }
}

// ---------------------------------------------------------------------------
// dQ: one workgroup (2 waves) per query block; wave owns 32 queries.
// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ __launch_bounds__(AB_NT, 2) void dq_kernel(
    const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ kt, const T* __restrict__ v,
    const T* __restrict__ dout, const float2* __restrict__ stat,
    const int32_t* __restrict__ row_ptr, const int32_t* __restrict__ col_idx, int64_t col_cap,
    T* __restrict__ dq, int Hq, int Hkv, int N, float c_log2, float scale) {
    using F = typename frag_of<T>::type;
    constexpr int E = sizeof(T);
    constexpr int KS = D / 16;
    constexpr int MT = D / 32;
    constexpr int RRB = D * E;
    constexpr int TRB = 64 * E;
    using RT = async_tile<64, RRB, 2, true>;     // K, V rows (slot-swapped)
    using TT = async_tile<D, TRB, 2, false>;     // K^T
    __shared__ __align__(1024) char k_lds[RT::BYTES];
    __shared__ __align__(1024) char v_lds[RT::BYTES];
    __shared__ __align__(1024) char kt_lds[TT::BYTES];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, half = lane >> 5;
    const int64_t row = blockIdx.x;
    const int64_t bh = row / N;
    const int n = static_cast<int>(row % N);
    const int b = static_cast<int>(bh / Hq), h = static_cast<int>(bh % Hq);
    const int hkv = h / (Hq / Hkv);
    const int64_t L = static_cast<int64_t>(N) * 64;
    const char* kb = reinterpret_cast<const char*>(k + static_cast<int64_t>(b * Hkv + hkv) * L * D);
    const char* ktb = reinterpret_cast<const char*>(kt + static_cast<int64_t>(b * Hkv + hkv) * L * D);
    const char* vb = reinterpret_cast<const char*>(v + static_cast<int64_t>(b * Hkv + hkv) * L * D);
    const int64_t qtok = bh * L + static_cast<int64_t>(n) * 64 + wave * 32 + (lane & 31);

    int64_t e0 = row_ptr[row], e1 = row_ptr[row + 1];
    e0 = e0 < 0 ? 0 : (e0 > col_cap ? col_cap : e0);
    e1 = e1 < e0 ? e0 : (e1 > col_cap ? col_cap : e1);

    F qf[KS], of[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
        load_frag(qf[ks], q + qtok * D + ks * 16 + half * 8);
        load_frag(of[ks], dout + qtok * D + ks * 16 + half * 8);
    }
    const float2 st = stat[qtok];
    f32x16_t dqa[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int i = 0; i < 16; ++i) dqa[mt][i] = 0.f;

    auto block_of = [&](int64_t e) -> int {
        const int c = scalar_load_i32(col_idx + e);
        return (c >= 0 && c < N) ? c : -1;
    };
    constexpr int64_t TILE = 64 * RRB;
    const RT rt(wave, lane);
    const TT tt(wave, lane);
    auto issue_rows = [&](int c) {
        const int64_t off = static_cast<int64_t>(c < 0 ? 0 : c) * TILE;
        rt.issue(k_lds, kb + off, wave);
        rt.issue(v_lds, vb + off, wave);
    };
    auto issue_tr = [&](int c) {
        tt.issue(kt_lds, ktb + static_cast<int64_t>(c < 0 ? 0 : c) * TILE, wave);
    };
    constexpr int ROWS_OPS = 2 * RT::PER_WAVE;
    constexpr int TR_OPS = TT::PER_WAVE;

#pragma unroll
    for (int ks = 0; ks < KS; ++ks) { settle(qf[ks]); settle(of[ks]); }   // before the copies start
    settle(st.x);
    settle(st.y);
    int c_cur = -1;
    if (e0 < e1) {
        c_cur = block_of(e0);
        issue_rows(c_cur);
        issue_tr(c_cur);
    }
    for (int64_t e = e0; e < e1; ++e) {
        const bool has_next = e + 1 < e1;
        const int c_next = has_next ? block_of(e + 1) : -1;

        vm_wait<TR_OPS>();              // K, V landed
        wg_barrier();
        F sb[2][2];
#pragma unroll
        for (int t2 = 0; t2 < 2; ++t2) {
            // S^T = K Q^T, dP^T = V dO^T: 32 keys x this lane's query
            f32x16_t s, dp;
#pragma unroll
            for (int i = 0; i < 16; ++i) { s[i] = 0.f; dp[i] = 0.f; }
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                F a;
                lds_frag_s<RRB>(a, k_lds, t2 * 32 + (lane & 31), ks * 16 + half * 8);
                mma(s, a, qf[ks]);
                lds_frag_s<RRB>(a, v_lds, t2 * 32 + (lane & 31), ks * 16 + half * 8);
                mma(dp, a, of[ks]);
            }
            float ds[16];
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const float p = fast_exp2(s[i] * c_log2 - st.x);
                ds[i] = p * (dp[i] - st.y);
            }
            pack_frag(sb[t2][0], ds);
            pack_frag(sb[t2][1], ds + 8);
        }
        wg_barrier();                   // K, V buffers free
        if (has_next) issue_rows(c_next);
        if (has_next) vm_wait<ROWS_OPS>(); else vm_wait<0>();   // K^T landed
        wg_barrier();
        if (c_cur >= 0) {
            // dQ^T += K^T dS^T over the 64 keys (4 k-steps of 16)
#pragma unroll
            for (int kk = 0; kk < 4; ++kk)
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) {
                    F a;
                    lds_frag_s<TRB>(a, kt_lds, mt * 32 + (lane & 31), kk * 16 + half * 8);
                    mma(dqa[mt], a, sb[kk >> 1][kk & 1]);
                }
        }
        wg_barrier();                   // K^T buffer free
        if (has_next) issue_tr(c_next);
        c_cur = c_next;
    }
    T* dqrow = dq + qtok * D;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
            const int d0 = mt * 32 + g4 * 8 + half * 4;
            if constexpr (E == 2) {
                const uint32_t w0 = pack2_bf16(dqa[mt][g4 * 4 + 0] * scale, dqa[mt][g4 * 4 + 1] * scale);
                const uint32_t w1 = pack2_bf16(dqa[mt][g4 * 4 + 2] * scale, dqa[mt][g4 * 4 + 3] * scale);
                *reinterpret_cast<uint2*>(dqrow + d0) = make_uint2(w0, w1);
            } else {
                *reinterpret_cast<float4*>(dqrow + d0) =
                    make_float4(dqa[mt][g4 * 4] * scale, dqa[mt][g4 * 4 + 1] * scale,
                                dqa[mt][g4 * 4 + 2] * scale, dqa[mt][g4 * 4 + 3] * scale);
            }
        }
}

// Workspace of the backward call: stat [ntok] float2, then Q^T, dO^T and K^T.
size_t bwd_workspace_bytes(int dtype, int D, int batch, int Hq, int Hkv, int N) {
    const size_t E = dtype == 1 ? 2 : 4;
    const size_t L = static_cast<size_t>(N) * 64;
    auto al = [](size_t x) { return (x + 255) / 256 * 256; };
    return al(8 * static_cast<size_t>(batch) * Hq * L) + 2 * al(E * batch * Hq * L * D) +
           al(E * batch * Hkv * L * D);
}

template <typename T, int D>
static hipError_t launch_bwd_t(const void* q, const void* k, const void* v, const void* o, const float* lse,
                               const void* dout, const int32_t* row_ptr, const int32_t* col_idx,
                               const int32_t* kv_ptr, const int32_t* kv_idx, int64_t col_cap, void* dq,
                               void* dk, void* dv, void* ws, int batch, int Hq, int Hkv, int N,
                               hipStream_t s) {
    const int64_t L = static_cast<int64_t>(N) * 64;
    const int64_t ntok = static_cast<int64_t>(batch) * Hq * L;
    auto al = [](size_t x) { return (x + 255) / 256 * 256; };
    char* w = static_cast<char*>(ws);
    float2* stat = reinterpret_cast<float2*>(w);
    w += al(8 * static_cast<size_t>(ntok));
    T* qt = reinterpret_cast<T*>(w);
    w += al(sizeof(T) * static_cast<size_t>(ntok) * D);
    T* dot = reinterpret_cast<T*>(w);
    w += al(sizeof(T) * static_cast<size_t>(ntok) * D);
    T* ktr = reinterpret_cast<T*>(w);

    const float c = kLog2e / sqrtf(static_cast<float>(D));
    const float scale = 1.0f / sqrtf(static_cast<float>(D));
    const T* Q = static_cast<const T*>(q);
    const T* K = static_cast<const T*>(k);
    const T* V = static_cast<const T*>(v);
    const T* dO = static_cast<const T*>(dout);
    const int64_t sthreads = ntok * (D / 8);
    hipLaunchKernelGGL((stat_kernel<T, D>), dim3(static_cast<unsigned>((sthreads + 255) / 256)), dim3(256), 0,
                       s, static_cast<const T*>(o), dO, lse, stat, ntok);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if ((e = launch_block_transpose(sizeof(T) == 2 ? 1 : 0, D, q, qt, ntok / 64, s)) != hipSuccess) return e;
    if ((e = launch_block_transpose(sizeof(T) == 2 ? 1 : 0, D, dout, dot, ntok / 64, s)) != hipSuccess) return e;
    if ((e = launch_block_transpose(sizeof(T) == 2 ? 1 : 0, D, k, ktr, static_cast<int64_t>(batch) * Hkv * N, s)) !=
        hipSuccess)
        return e;
    const int64_t krows = static_cast<int64_t>(batch) * Hkv * N;
    hipLaunchKernelGGL((dkdv_kernel<T, D, 0>), dim3(static_cast<unsigned>(krows)), dim3(AB_NT), 0, s, Q, qt, K, V,
                       dO, dot, stat, kv_ptr, kv_idx, col_cap, static_cast<T*>(dv), Hq, Hkv, N, c, scale);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL((dkdv_kernel<T, D, 1>), dim3(static_cast<unsigned>(krows)), dim3(AB_NT), 0, s, Q, qt, K, V,
                       dO, dot, stat, kv_ptr, kv_idx, col_cap, static_cast<T*>(dk), Hq, Hkv, N, c, scale);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    const int64_t qrows = static_cast<int64_t>(batch) * Hq * N;
    hipLaunchKernelGGL((dq_kernel<T, D>), dim3(static_cast<unsigned>(qrows)), dim3(AB_NT), 0, s, Q, K, ktr, V,
                       dO, stat, row_ptr, col_idx, col_cap, static_cast<T*>(dq), Hq, Hkv, N, c, scale);
    return hipGetLastError();
}

hipError_t launch_attn_bwd(int dtype, int D, const void* q, const void* k, const void* v, const void* o,
                           const float* lse, const void* dout, const int32_t* row_ptr,
                           const int32_t* col_idx, const int32_t* kv_ptr, const int32_t* kv_idx,
                           int64_t col_cap, void* dq, void* dk, void* dv, void* ws, int batch,
                           int Hq, int Hkv, int N, hipStream_t s) {
#define VSA2_BWD(T, DD) \
    return launch_bwd_t<T, DD>(q, k, v, o, lse, dout, row_ptr, col_idx, kv_ptr, kv_idx, col_cap, dq, dk, dv, \
                               ws, batch, Hq, Hkv, N, s)
    if (dtype == 1) {
        if (D == 64) VSA2_BWD(bf16_t, 64);
        if (D == 128) VSA2_BWD(bf16_t, 128);
    } else {
        if (D == 64) VSA2_BWD(float, 64);
        if (D == 128) VSA2_BWD(float, 128);
    }
#undef VSA2_BWD
    return hipErrorInvalidValue;
}

}  // namespace vsa2
