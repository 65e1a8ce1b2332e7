// Block-sparse attention backward for gfx950.  The block mask is a constant
// (routing carries no gradient, VSA2 Sec. 2.1), so the gradients are those of
// masked softmax attention restricted to the selected block pairs:
//   Delta_l = dO_l . O_l
//   P = exp(S/sqrt(D) - LSE),  dP = dO V^T,  dS = P o (dP - Delta)
//   dV = P^T dO,  dK = dS^T Q / sqrt(D),  dQ = dS K / sqrt(D)
// Three kernels, all deterministic (no atomics):
//   delta_kernel   Delta per query token
//   dkdv_kernel    key-block stationary: one workgroup per key block walks the
//                  transposed (CSC) list of query blocks that selected it;
//                  a wave owns 32 keys, dK^T and dV^T accumulate in registers
//   dq_kernel      query-block stationary: one workgroup per query block walks
//                  its CSR row; a wave owns 32 queries, dQ^T accumulates
// Layout tricks as in the forward: products are arranged so that each lane
// owns one column (a key in dkdv, a query in dq) and its 16 accumulator rows
// form two runs of 8 consecutive rows (tiles stored with the bit-2/3 slot
// swap), so a lane's P / dS values are directly the B operand of the next
// MFMA, and per-row statistics (LSE, Delta) are lane-local in dq.
#include "common.hpp"
#include "internal.hpp"

namespace vsa2 {

constexpr int AB_NT = 128;
constexpr float kLog2e = 1.4426950408889634f;

// ---------------------------------------------------------------------------
// Delta_l = sum_d dO[l][d] * O[l][d]; 16 lanes per token (D <= 128).
// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ __launch_bounds__(256) void delta_kernel(const T* __restrict__ o, const T* __restrict__ dout,
                                                    float* __restrict__ delta, int64_t ntok) {
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
    if (tok < ntok && part == 0) delta[tok] = s;
}

// ---------------------------------------------------------------------------
// dK, dV: one workgroup (2 waves) per key block of head (b, hkv).
// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ __launch_bounds__(AB_NT, 1) void dkdv_kernel(
    const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ v,
    const T* __restrict__ dout, const float* __restrict__ lse, const float* __restrict__ delta,
    const int32_t* __restrict__ kv_ptr, const int32_t* __restrict__ kv_idx, int64_t col_cap,
    T* __restrict__ dk, T* __restrict__ dv, int Hq, int Hkv, int N, float c_log2, float scale) {
    using F = typename frag_of<T>::type;
    constexpr int E = sizeof(T);
    constexpr int KS = D / 16;
    constexpr int MT = D / 32;
    constexpr int RRB = D * E;      // row-major tile row bytes
    constexpr int TRB = 64 * E;     // transposed tile row bytes
    using TL = tile_transposed<T, D, AB_NT>;
    __shared__ __align__(16) char q_lds[64 * RRB];
    __shared__ __align__(16) char qt_lds[D * TRB];
    __shared__ __align__(16) char o_lds[64 * RRB];   // dO
    __shared__ __align__(16) char ot_lds[D * TRB];   // dO^T
    __shared__ float lse_lds[64], del_lds[64];

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

    // K and V rows of this lane's key as B operands (column = key, k = d)
    F kf[KS], vf[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
        load_frag(kf[ks], k + ktok * D + ks * 16 + half * 8);
        load_frag(vf[ks], v + ktok * D + ks * 16 + half * 8);
    }
    f32x16_t dva[MT], dka[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int i = 0; i < 16; ++i) { dva[mt][i] = 0.f; dka[mt][i] = 0.f; }

    TL tq, to;
    for (int64_t e = e0; e < e1; ++e) {
        const int ent = kv_idx[e];
        const int hl = ent / N, nq = ent % N;
        if (ent < 0 || hl >= grp) continue;            // malformed entry: skipped
        const int64_t bh = static_cast<int64_t>(b) * Hq + hkv * grp + hl;
        const int64_t q0 = bh * L + static_cast<int64_t>(nq) * 64;
        tq.load(q, q0, tid);
        to.load(dout, q0, tid);
        __syncthreads();
        tq.store_rows(q_lds, true, tid);
        tq.store(qt_lds, tid);
        to.store_rows(o_lds, true, tid);
        to.store(ot_lds, tid);
        if (tid < 64) {
            lse_lds[tid] = lse[q0 + tid] * kLog2e;
            del_lds[tid] = delta[q0 + tid];
        }
        __syncthreads();

#pragma unroll
        for (int qt = 0; qt < 2; ++qt) {
            // S = Q K^T and dP = dO V^T for 32 queries x this lane's key
            f32x16_t s, dp;
#pragma unroll
            for (int i = 0; i < 16; ++i) { s[i] = 0.f; dp[i] = 0.f; }
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                F a;
                lds_frag<RRB>(a, q_lds, qt * 32 + (lane & 31), ks * 16 + half * 8);
                mma(s, a, kf[ks]);
                lds_frag<RRB>(a, o_lds, qt * 32 + (lane & 31), ks * 16 + half * 8);
                mma(dp, a, vf[ks]);
            }
            // entry v is query 32qt + 16(v/8) + 8half + v%8
            float p[16], ds[16];
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int qi = qt * 32 + (i >> 3) * 16 + half * 8 + (i & 7);
                p[i] = exp2f(s[i] * c_log2 - lse_lds[qi]);
                ds[i] = p[i] * (dp[i] - del_lds[qi]);
            }
            // dV^T += dO^T P and dK^T += Q^T dS over the 32 queries (2 k-steps)
#pragma unroll
            for (int kh = 0; kh < 2; ++kh) {
                F pb, sb;
                pack_frag(pb, p + kh * 8);
                pack_frag(sb, ds + kh * 8);
                const int kk = qt * 2 + kh;
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) {
                    F a;
                    lds_frag<TRB>(a, ot_lds, mt * 32 + (lane & 31), kk * 16 + half * 8);
                    mma(dva[mt], a, pb);
                    lds_frag<TRB>(a, qt_lds, mt * 32 + (lane & 31), kk * 16 + half * 8);
                    mma(dka[mt], a, sb);
                }
            }
        }
        __syncthreads();
    }

    // lane holds key column (lane & 31) and d = 32mt + 8(v/4) + 4half + v%4
    T* dkrow = dk + ktok * D;
    T* dvrow = dv + ktok * D;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
            const int d0 = mt * 32 + g4 * 8 + half * 4;
            if constexpr (E == 2) {
                uint32_t wk[2], wv[2];
#pragma unroll
                for (int j = 0; j < 2; ++j) {
                    wk[j] = static_cast<uint32_t>(f32_to_bf16(dka[mt][g4 * 4 + 2 * j] * scale)) |
                            (static_cast<uint32_t>(f32_to_bf16(dka[mt][g4 * 4 + 2 * j + 1] * scale)) << 16);
                    wv[j] = static_cast<uint32_t>(f32_to_bf16(dva[mt][g4 * 4 + 2 * j])) |
                            (static_cast<uint32_t>(f32_to_bf16(dva[mt][g4 * 4 + 2 * j + 1])) << 16);
                }
                *reinterpret_cast<uint2*>(dkrow + d0) = make_uint2(wk[0], wk[1]);
                *reinterpret_cast<uint2*>(dvrow + d0) = make_uint2(wv[0], wv[1]);
            } else {
                *reinterpret_cast<float4*>(dkrow + d0) =
                    make_float4(dka[mt][g4 * 4] * scale, dka[mt][g4 * 4 + 1] * scale,
                                dka[mt][g4 * 4 + 2] * scale, dka[mt][g4 * 4 + 3] * scale);
                *reinterpret_cast<float4*>(dvrow + d0) =
                    make_float4(dva[mt][g4 * 4], dva[mt][g4 * 4 + 1], dva[mt][g4 * 4 + 2], dva[mt][g4 * 4 + 3]);
            }
        }
}

// ---------------------------------------------------------------------------
// dQ: one workgroup (2 waves) per query block; wave owns 32 queries.
// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ __launch_bounds__(AB_NT, 1) void dq_kernel(
    const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ v,
    const T* __restrict__ dout, const float* __restrict__ lse, const float* __restrict__ delta,
    const int32_t* __restrict__ row_ptr, const int32_t* __restrict__ col_idx, int64_t col_cap,
    T* __restrict__ dq, int Hq, int Hkv, int N, float c_log2, float scale) {
    using F = typename frag_of<T>::type;
    constexpr int E = sizeof(T);
    constexpr int KS = D / 16;
    constexpr int MT = D / 32;
    constexpr int RRB = D * E;
    constexpr int TRB = 64 * E;
    using TL = tile_transposed<T, D, AB_NT>;
    using RL = tile_rows<T, D, AB_NT>;
    __shared__ __align__(16) char k_lds[64 * RRB];
    __shared__ __align__(16) char kt_lds[D * TRB];
    __shared__ __align__(16) char v_lds[64 * RRB];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, half = lane >> 5;
    const int64_t row = blockIdx.x;
    const int64_t bh = row / N;
    const int n = static_cast<int>(row % N);
    const int b = static_cast<int>(bh / Hq), h = static_cast<int>(bh % Hq);
    const int hkv = h / (Hq / Hkv);
    const int64_t L = static_cast<int64_t>(N) * 64;
    const T* kb = k + static_cast<int64_t>(b * Hkv + hkv) * L * D;
    const T* vb = v + static_cast<int64_t>(b * Hkv + hkv) * L * D;
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
    const float lse2 = lse[qtok] * kLog2e;
    const float del = delta[qtok];
    f32x16_t dqa[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int i = 0; i < 16; ++i) dqa[mt][i] = 0.f;

    TL tk;
    RL tv;
    for (int64_t e = e0; e < e1; ++e) {
        const int c = col_idx[e];
        if (c < 0 || c >= N) continue;
        tk.load(kb, static_cast<int64_t>(c) * 64, tid);
        tv.load(vb, static_cast<int64_t>(c) * 64, L, tid);
        __syncthreads();
        tk.store_rows(k_lds, true, tid);
        tk.store(kt_lds, tid);
        tv.store(v_lds, true, tid);
        __syncthreads();
#pragma unroll
        for (int t2 = 0; t2 < 2; ++t2) {
            // S^T = K Q^T, dP^T = V dO^T: 32 keys x this lane's query
            f32x16_t s, dp;
#pragma unroll
            for (int i = 0; i < 16; ++i) { s[i] = 0.f; dp[i] = 0.f; }
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                F a;
                lds_frag<RRB>(a, k_lds, t2 * 32 + (lane & 31), ks * 16 + half * 8);
                mma(s, a, qf[ks]);
                lds_frag<RRB>(a, v_lds, t2 * 32 + (lane & 31), ks * 16 + half * 8);
                mma(dp, a, of[ks]);
            }
            float ds[16];
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const float p = exp2f(s[i] * c_log2 - lse2);
                ds[i] = p * (dp[i] - del);
            }
            // dQ^T += K^T dS^T over these 32 keys (2 k-steps of 16)
#pragma unroll
            for (int kh = 0; kh < 2; ++kh) {
                F sb;
                pack_frag(sb, ds + kh * 8);
                const int kk = t2 * 2 + kh;
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) {
                    F a;
                    lds_frag<TRB>(a, kt_lds, mt * 32 + (lane & 31), kk * 16 + half * 8);
                    mma(dqa[mt], a, sb);
                }
            }
        }
        __syncthreads();
    }
    T* dqrow = dq + qtok * D;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
            const int d0 = mt * 32 + g4 * 8 + half * 4;
            if constexpr (E == 2) {
                const uint32_t w0 = static_cast<uint32_t>(f32_to_bf16(dqa[mt][g4 * 4 + 0] * scale)) |
                                    (static_cast<uint32_t>(f32_to_bf16(dqa[mt][g4 * 4 + 1] * scale)) << 16);
                const uint32_t w1 = static_cast<uint32_t>(f32_to_bf16(dqa[mt][g4 * 4 + 2] * scale)) |
                                    (static_cast<uint32_t>(f32_to_bf16(dqa[mt][g4 * 4 + 3] * scale)) << 16);
                *reinterpret_cast<uint2*>(dqrow + d0) = make_uint2(w0, w1);
            } else {
                *reinterpret_cast<float4*>(dqrow + d0) =
                    make_float4(dqa[mt][g4 * 4] * scale, dqa[mt][g4 * 4 + 1] * scale,
                                dqa[mt][g4 * 4 + 2] * scale, dqa[mt][g4 * 4 + 3] * scale);
            }
        }
}

template <typename T, int D>
static hipError_t launch_bwd_t(const void* q, const void* k, const void* v, const void* o, const float* lse,
                               const void* dout, const int32_t* row_ptr, const int32_t* col_idx,
                               const int32_t* kv_ptr, const int32_t* kv_idx, int64_t col_cap, void* dq,
                               void* dk, void* dv, float* delta, int batch, int Hq, int Hkv, int N,
                               hipStream_t s) {
    const int64_t L = static_cast<int64_t>(N) * 64;
    const int64_t ntok = static_cast<int64_t>(batch) * Hq * L;
    const float c = kLog2e / sqrtf(static_cast<float>(D));
    const float scale = 1.0f / sqrtf(static_cast<float>(D));
    const T* Q = static_cast<const T*>(q);
    const T* K = static_cast<const T*>(k);
    const T* V = static_cast<const T*>(v);
    const T* dO = static_cast<const T*>(dout);
    const int64_t dthreads = ntok * (D / 8);
    hipLaunchKernelGGL((delta_kernel<T, D>), dim3(static_cast<unsigned>((dthreads + 255) / 256)), dim3(256), 0,
                       s, static_cast<const T*>(o), dO, delta, ntok);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int64_t krows = static_cast<int64_t>(batch) * Hkv * N;
    hipLaunchKernelGGL((dkdv_kernel<T, D>), dim3(static_cast<unsigned>(krows)), dim3(AB_NT), 0, s, Q, K, V, dO,
                       lse, delta, kv_ptr, kv_idx, col_cap, static_cast<T*>(dk), static_cast<T*>(dv), Hq, Hkv,
                       N, c, scale);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    const int64_t qrows = static_cast<int64_t>(batch) * Hq * N;
    hipLaunchKernelGGL((dq_kernel<T, D>), dim3(static_cast<unsigned>(qrows)), dim3(AB_NT), 0, s, Q, K, V, dO, lse,
                       delta, row_ptr, col_idx, col_cap, static_cast<T*>(dq), Hq, Hkv, N, c, scale);
    return hipGetLastError();
}

hipError_t launch_attn_bwd(int dtype, int D, const void* q, const void* k, const void* v, const void* o,
                           const float* lse, const void* dout, const int32_t* row_ptr,
                           const int32_t* col_idx, const int32_t* kv_ptr, const int32_t* kv_idx,
                           int64_t col_cap, void* dq, void* dk, void* dv, float* delta, int batch,
                           int Hq, int Hkv, int N, hipStream_t s) {
#define VSA2_BWD(T, DD) \
    return launch_bwd_t<T, DD>(q, k, v, o, lse, dout, row_ptr, col_idx, kv_ptr, kv_idx, col_cap, dq, dk, dv, \
                               delta, batch, Hq, Hkv, N, s)
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
