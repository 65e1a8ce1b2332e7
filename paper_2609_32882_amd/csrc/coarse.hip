// Coarse branch and gated merge (VSA2 Sec. 2.2, "Coarse Branch" and
// "Gated Merge"):
//   [Q_c, K_c, V_c] = MeanPool_B([Q, K, V])            (vsa2_pool with P = B)
//   O_c_hat = Softmax(Q_c K_c^T / sqrt(D)) V_c          dense over N cube means
//   O = tanh(g) * Repeat_B(O_c_hat) + O_f               g = X W_g per token, head
// and the gradients of each step (the MeanPool adjoint adds the pooled
// gradients back onto the token gradients).
//
// The coarse attention is small (N x N per head, N = number of cubes, not a
// multiple of 64 in general), so its kernels favour simplicity: tiles of 64
// cube rows are loaded synchronously into padded, slot-permuted LDS rows
// (the layout the fragment readers of the fine kernels expect), rows past N
// read as zero and are masked out of every softmax.
#include "common.hpp"
#include "internal.hpp"

namespace vsa2 {

constexpr int CB_NT = 128;   // two waves, 32 rows each
constexpr float kLog2eC = 1.4426950408889634f;

// Rows row0 .. row0+63 of a [rows][D] tensor into a padded LDS tile, LDS row r
// holding global row row0 + tile_row_at(r) (bf16: column groups in the
// cgroup_pos order the fragment readers expect); rows >= nrows are zero.
template <int RB, bool CPERM>
__device__ __forceinline__ void load_rows_sync(char* lds, const char* g, int64_t row0, int64_t nrows, int tid) {
    constexpr int CH = RB / 16;
    for (int c = tid; c < 64 * CH; c += CB_NT) {
        const int r = c / CH, ch = c % CH;
        const int64_t gr = row0 + tile_row_at<RB>(r);
        uint4 v = make_uint4(0, 0, 0, 0);
        if (gr < nrows) v = *reinterpret_cast<const uint4*>(g + gr * RB + ch * 16);
        const int pc = CPERM ? cgroup_pos<RB>(ch >> 1) * 32 + (ch & 1) * 16 : ch * 16;
        *reinterpret_cast<uint4*>(lds + r * (RB + 16) + pc) = v;
    }
}

template <typename F>
__device__ __forceinline__ void zero_frag(F& f) {
    f = F{};
}

// ---------------------------------------------------------------------------
// Forward: one workgroup per (64 coarse queries, batch x query head).
// S^T = K_c Q_c^T per 64-key tile, online softmax over the keys < N,
// O^T += V_c^T P^T (the fine forward's transposed formulation), with P as
// two bf16 terms (hi + lo): V_c's rows are cube means, dominated by their
// common component, which would amplify one-term rounding of P; the branch
// is small enough that the second product costs little.
// STAT: the backward's statistics instead of O: per coarse query
// (LSE * log2 e, Delta = dO . O), Delta matching sum_j P_j dP_j to ~2^-17.
// ---------------------------------------------------------------------------
template <typename T, int D, bool STAT>
__global__ __launch_bounds__(CB_NT) void coarse_fwd_kernel(const T* __restrict__ qc, const T* __restrict__ kc,
                                                           const T* __restrict__ vc, T* __restrict__ oc,
                                                           float* __restrict__ lse, const T* __restrict__ doc,
                                                           float2* __restrict__ stat, int Hq, int Hkv, int N,
                                                           float c_log2) {
    using F = typename frag_of<T>::type;
    constexpr int E = sizeof(T);
    constexpr int KS = D / 16;
    constexpr int MT = D / 32;
    constexpr int RB = D * E;
    __shared__ __align__(16) char k_lds[64 * (RB + 16)];
    __shared__ __align__(16) char v_lds[64 * (RB + 16)];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, half = lane >> 5;
    const int64_t bh = blockIdx.y;
    const int64_t b = bh / Hq, h = bh % Hq;
    const int64_t kv = b * Hkv + h / (Hq / Hkv);
    const int64_t n = static_cast<int64_t>(blockIdx.x) * 64 + wave * 32 + (lane & 31);
    const bool live = n < N;
    const T* qrow = qc + (bh * N + n) * D;

    F qf[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
        if (live) load_frag(qf[ks], qrow + ks * 16 + half * 8);
        else zero_frag(qf[ks]);
    }
    f32x16_t oacc[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int i = 0; i < 16; ++i) oacc[mt][i] = 0.f;
    float m = -INFINITY, l = 0.f;

    const char* kb = reinterpret_cast<const char*>(kc + kv * N * D);
    const char* vb = reinterpret_cast<const char*>(vc + kv * N * D);
    const int ntiles = (N + 63) / 64;
    for (int kt = 0; kt < ntiles; ++kt) {
        __syncthreads();                  // previous tile's readers are done
        load_rows_sync<RB, E == 2>(k_lds, kb, static_cast<int64_t>(kt) * 64, N, tid);
        load_rows_sync<RB, E == 2>(v_lds, vb, static_cast<int64_t>(kt) * 64, N, tid);
        __syncthreads();
        f32x16_t s[2];
#pragma unroll
        for (int t2 = 0; t2 < 2; ++t2) {
#pragma unroll
            for (int i = 0; i < 16; ++i) s[t2][i] = 0.f;
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                F a;
                lds_frag_s<RB>(a, k_lds, t2 * 32 + (lane & 31), ks * 16 + half * 8);
                mma(s[t2], a, qf[ks]);
            }
        }
        // element i of s[t2] is key 64kt + 32t2 + 16(i/8) + 8half + i%8
        float mx = -INFINITY;
#pragma unroll
        for (int t2 = 0; t2 < 2; ++t2)
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int key = kt * 64 + t2 * 32 + (i >> 3) * 16 + half * 8 + (i & 7);
                s[t2][i] = key < N ? s[t2][i] * c_log2 : -INFINITY;
                mx = fmaxf(mx, s[t2][i]);
            }
        mx = fmaxf(mx, swap_half(mx));    // finite: every tile holds a key < N
        const float mn = fmaxf(m, mx);
        const float alpha = fast_exp2(m - mn);
        float ps = 0.f;
#pragma unroll
        for (int t2 = 0; t2 < 2; ++t2)
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const float pv = fast_exp2(s[t2][i] - mn);
                s[t2][i] = pv;
                ps += pv;
            }
        l = l * alpha + ps;
        m = mn;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int i = 0; i < 16; ++i) oacc[mt][i] *= alpha;
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
            F pb, pl;
            float pv[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) pv[i] = s[kk >> 1][(kk & 1) * 8 + i];
            pack_frag_hilo(pb, pl, pv);
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                F a;
                lds_frag_tr<RB, true>(a, v_lds, mt * 32, kk * 16);
                mma(oacc[mt], a, pb);
                mma(oacc[mt], a, pl);
            }
        }
    }
    const float lt = l + swap_half(l);
    const float inv = 1.0f / lt;
    if constexpr (STAT) {
        // lane holds d = 32mt + 8(v/4) + 4half + v%4 of its query
        float delta = 0.f;
        if (live) {
            const T* drow = doc + (bh * N + n) * D;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                for (int v = 0; v < 16; ++v)
                    delta = fmaf(to_f32(drow[mt * 32 + (v >> 2) * 8 + half * 4 + (v & 3)]), oacc[mt][v] * inv, delta);
        }
        delta += swap_half(delta);
        if (live && half == 0) stat[bh * N + n] = make_float2(m + log2f(lt), delta);
        return;
    }
    if (!live) return;
    T* orow = oc + (bh * N + n) * D;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
            const int d0 = mt * 32 + g4 * 8 + half * 4;
#pragma unroll
            for (int j = 0; j < 4; ++j) from_f32(orow[d0 + j], oacc[mt][g4 * 4 + j] * inv);
        }
    if (half == 0) lse[bh * N + n] = (m + log2f(lt)) * 0.6931471805599453f;
}

// ---------------------------------------------------------------------------
// Backward, key side: one workgroup per (64 coarse keys, batch x KV head); a
// wave owns 32 keys and accumulates dV_c^T and dK_c^T over every coarse
// query of the KV group (64-row tiles; rows past N have LSE = +inf, so
// their P and dS are 0).
// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ __launch_bounds__(CB_NT) void coarse_dkdv_kernel(const T* __restrict__ qc, const T* __restrict__ kc,
                                                            const T* __restrict__ vc, const T* __restrict__ doc,
                                                            const float2* __restrict__ stat, T* __restrict__ dkc,
                                                            T* __restrict__ dvc, int Hq, int Hkv, int N,
                                                            float c_log2, float scale) {
    using F = typename frag_of<T>::type;
    constexpr int E = sizeof(T);
    constexpr int KS = D / 16;
    constexpr int MT = D / 32;
    constexpr int RB = D * E;
    __shared__ __align__(16) char q_lds[64 * (RB + 16)];
    __shared__ __align__(16) char o_lds[64 * (RB + 16)];
    __shared__ float2 st_lds[64];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, half = lane >> 5;
    const int64_t kvh = blockIdx.y;                       // b * Hkv + hkv
    const int64_t b = kvh / Hkv, hkv = kvh % Hkv;
    const int grp = Hq / Hkv;
    const int64_t j = static_cast<int64_t>(blockIdx.x) * 64 + wave * 32 + (lane & 31);
    const bool live = j < N;
    F kf[KS], vf[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
        if (live) {
            load_frag(kf[ks], kc + (kvh * N + j) * D + ks * 16 + half * 8);
            load_frag(vf[ks], vc + (kvh * N + j) * D + ks * 16 + half * 8);
        } else {
            zero_frag(kf[ks]);
            zero_frag(vf[ks]);
        }
    }
    f32x16_t acc_v[MT], acc_k[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int i = 0; i < 16; ++i) { acc_v[mt][i] = 0.f; acc_k[mt][i] = 0.f; }

    const int ntiles = (N + 63) / 64;
    for (int hl = 0; hl < grp; ++hl) {
        const int64_t bh = b * Hq + hkv * grp + hl;
        const char* qb = reinterpret_cast<const char*>(qc + bh * N * D);
        const char* ob = reinterpret_cast<const char*>(doc + bh * N * D);
        for (int qt = 0; qt < ntiles; ++qt) {
            __syncthreads();
            load_rows_sync<RB, E == 2>(q_lds, qb, static_cast<int64_t>(qt) * 64, N, tid);
            load_rows_sync<RB, E == 2>(o_lds, ob, static_cast<int64_t>(qt) * 64, N, tid);
            if (tid < 64) {
                const int64_t i = static_cast<int64_t>(qt) * 64 + tid;
                st_lds[tid] = i < N ? stat[bh * N + i] : make_float2(INFINITY, 0.f);
            }
            __syncthreads();
#pragma unroll
            for (int qtile = 0; qtile < 2; ++qtile) {
                f32x16_t s, dp;
#pragma unroll
                for (int i = 0; i < 16; ++i) { s[i] = 0.f; dp[i] = 0.f; }
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) {
                    F a;
                    lds_frag_s<RB>(a, q_lds, qtile * 32 + (lane & 31), ks * 16 + half * 8);
                    mma(s, a, kf[ks]);
                    lds_frag_s<RB>(a, o_lds, qtile * 32 + (lane & 31), ks * 16 + half * 8);
                    mma(dp, a, vf[ks]);
                }
                // entry i is query 32qtile + 16(i/8) + 8half + i%8 of the tile
                float pv[16], dsv[16];
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const float2 sv = st_lds[qtile * 32 + (i >> 3) * 16 + half * 8 + (i & 7)];
                    pv[i] = fast_exp2(s[i] * c_log2 - sv.x);
                    dsv[i] = pv[i] * (dp[i] - sv.y);
                }
                // P and dS as hi + lo bf16 terms: Q_c (and K_c) carry a large
                // common component, which would amplify one-term rounding
                F pb[2], db[2], pl[2], dl[2];
                pack_frag_hilo(pb[0], pl[0], pv);
                pack_frag_hilo(pb[1], pl[1], pv + 8);
                pack_frag_hilo(db[0], dl[0], dsv);
                pack_frag_hilo(db[1], dl[1], dsv + 8);
#pragma unroll
                for (int h2 = 0; h2 < 2; ++h2)
#pragma unroll
                    for (int mt = 0; mt < MT; ++mt) {
                        F a;
                        lds_frag_tr<RB, true>(a, o_lds, mt * 32, (2 * qtile + h2) * 16);
                        mma(acc_v[mt], a, pb[h2]);
                        mma(acc_v[mt], a, pl[h2]);
                        lds_frag_tr<RB, true>(a, q_lds, mt * 32, (2 * qtile + h2) * 16);
                        mma(acc_k[mt], a, db[h2]);
                        mma(acc_k[mt], a, dl[h2]);
                    }
            }
        }
    }
    if (!live) return;
    T* gk = dkc + (kvh * N + j) * D;
    T* gv = dvc + (kvh * N + j) * D;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
            const int d0 = mt * 32 + g4 * 8 + half * 4;
#pragma unroll
            for (int x = 0; x < 4; ++x) {
                from_f32(gk[d0 + x], acc_k[mt][g4 * 4 + x] * scale);
                from_f32(gv[d0 + x], acc_v[mt][g4 * 4 + x]);
            }
        }
}

// ---------------------------------------------------------------------------
// Backward, query side: one workgroup per (64 coarse queries, batch x query
// head); dQ_c^T += K_c^T dS^T over the key tiles, keys past N masked.
// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ __launch_bounds__(CB_NT) void coarse_dq_kernel(const T* __restrict__ qc, const T* __restrict__ kc,
                                                          const T* __restrict__ vc, const T* __restrict__ doc,
                                                          const float2* __restrict__ stat, T* __restrict__ dqc,
                                                          int Hq, int Hkv, int N, float c_log2, float scale) {
    using F = typename frag_of<T>::type;
    constexpr int E = sizeof(T);
    constexpr int KS = D / 16;
    constexpr int MT = D / 32;
    constexpr int RB = D * E;
    __shared__ __align__(16) char k_lds[64 * (RB + 16)];
    __shared__ __align__(16) char v_lds[64 * (RB + 16)];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, half = lane >> 5;
    const int64_t bh = blockIdx.y;
    const int64_t b = bh / Hq, h = bh % Hq;
    const int64_t kv = b * Hkv + h / (Hq / Hkv);
    const int64_t n = static_cast<int64_t>(blockIdx.x) * 64 + wave * 32 + (lane & 31);
    const bool live = n < N;
    F qf[KS], of[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
        if (live) {
            load_frag(qf[ks], qc + (bh * N + n) * D + ks * 16 + half * 8);
            load_frag(of[ks], doc + (bh * N + n) * D + ks * 16 + half * 8);
        } else {
            zero_frag(qf[ks]);
            zero_frag(of[ks]);
        }
    }
    const float2 st = live ? stat[bh * N + n] : make_float2(INFINITY, 0.f);
    f32x16_t dqa[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int i = 0; i < 16; ++i) dqa[mt][i] = 0.f;

    const char* kb = reinterpret_cast<const char*>(kc + kv * N * D);
    const char* vb = reinterpret_cast<const char*>(vc + kv * N * D);
    const int ntiles = (N + 63) / 64;
    for (int kt = 0; kt < ntiles; ++kt) {
        __syncthreads();
        load_rows_sync<RB, E == 2>(k_lds, kb, static_cast<int64_t>(kt) * 64, N, tid);
        load_rows_sync<RB, E == 2>(v_lds, vb, static_cast<int64_t>(kt) * 64, N, tid);
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
                lds_frag_s<RB>(a, k_lds, t2 * 32 + (lane & 31), ks * 16 + half * 8);
                mma(s, a, qf[ks]);
                lds_frag_s<RB>(a, v_lds, t2 * 32 + (lane & 31), ks * 16 + half * 8);
                mma(dp, a, of[ks]);
            }
            float ds[16];
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int key = kt * 64 + t2 * 32 + (i >> 3) * 16 + half * 8 + (i & 7);
                const float p = key < N ? fast_exp2(s[i] * c_log2 - st.x) : 0.f;
                ds[i] = p * (dp[i] - st.y);
            }
            F sb[2], sl[2];
            pack_frag_hilo(sb[0], sl[0], ds);
            pack_frag_hilo(sb[1], sl[1], ds + 8);
#pragma unroll
            for (int h2 = 0; h2 < 2; ++h2)
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) {
                    F a;
                    lds_frag_tr<RB, true>(a, k_lds, mt * 32, (2 * t2 + h2) * 16);
                    mma(dqa[mt], a, sb[h2]);
                    mma(dqa[mt], a, sl[h2]);
                }
        }
    }
    if (!live) return;
    T* g = dqc + (bh * N + n) * D;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
            const int d0 = mt * 32 + g4 * 8 + half * 4;
#pragma unroll
            for (int x = 0; x < 4; ++x) from_f32(g[d0 + x], dqa[mt][g4 * 4 + x] * scale);
        }
}

// ---------------------------------------------------------------------------
// Gated merge: out[l] = tanh(g_l) * oc[cube(l)] + of[l] for the L video
// tokens of each sequence of Lj tokens; text tokens (l >= L) keep of[l].
// One thread per 8 elements.
// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ __launch_bounds__(256) void gate_merge_kernel(const float* __restrict__ gate, const T* __restrict__ oc,
                                                         const T* __restrict__ of, T* __restrict__ out,
                                                         int64_t ntok, int64_t L, int64_t Lj, int N) {
    constexpr int PARTS = D / 8;
    const int64_t t = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    const int64_t tok = t / PARTS;
    if (tok >= ntok) return;
    const int d0 = static_cast<int>(t % PARTS) * 8;
    const int64_t bh = tok / Lj, l = tok - bh * Lj;
    const T* f = of + tok * D + d0;
    T* o = out + tok * D + d0;
    if (l >= L) {               // a text token: no coarse branch
#pragma unroll
        for (int i = 0; i < 8; ++i) o[i] = f[i];
        return;
    }
    const float gv = tanhf(gate[tok]);
    const T* c = oc + (bh * N + l / 64) * D + d0;
#pragma unroll
    for (int i = 0; i < 8; ++i) from_f32(o[i], fmaf(gv, to_f32(c[i]), to_f32(f[i])));
}

// Backward of the merge: one workgroup of 256 per cube.  Four threads per
// token (D/4 elements each): dg_l = (1 - tanh(g_l)^2) (dout_l . oc_n);
// doc[n] = sum_l tanh(g_l) dout_l, summed over the cube's 64 tokens in LDS.
// Sequences hold N video cubes then M text blocks (Lj = (N + M) * 64
// tokens); the workgroups past the video cubes write dg = 0 for the text
// tokens, which have no coarse branch.
template <typename T, int D>
__global__ __launch_bounds__(256) void gate_merge_bwd_kernel(const float* __restrict__ gate,
                                                             const T* __restrict__ oc,
                                                             const T* __restrict__ dout, T* __restrict__ doc,
                                                             float* __restrict__ dgate, int64_t ncubes, int N,
                                                             int M, cube_grid grid) {
    constexpr int PER = D / 4;
    __shared__ float part[64][D + 1];
    const int tid = threadIdx.x;
    const int t = tid >> 2, q4 = tid & 3;
    const int64_t Lj = static_cast<int64_t>(N + M) * 64;
    if (blockIdx.x >= ncubes) {                      // text block (b * Hq + h) * M + m
        const int64_t tb = blockIdx.x - ncubes;
        if (q4 == 0) dgate[(tb / M) * Lj + static_cast<int64_t>(N) * 64 + (tb % M) * 64 + t] = 0.f;
        return;
    }
    const int64_t cube = blockIdx.x;                 // (b * Hq + h) * N + n
    const int64_t tok = (cube / N) * Lj + (cube % N) * 64 + t;
    // a padding token of a padded grid is not an output: gate 0, dgate 0
    bool real = true;
    if (grid.padded) real = token_in(grid, cube_extent(grid, static_cast<int>(cube % N)), t);
    const float gv = real ? tanhf(gate[tok]) : 0.f;
    const T* dl = dout + tok * D + q4 * PER;
    const T* c = oc + cube * D + q4 * PER;
    float dot = 0.f;
#pragma unroll 8
    for (int i = 0; i < PER; ++i) {
        const float x = to_f32(dl[i]);
        dot = fmaf(x, to_f32(c[i]), dot);
        part[t][q4 * PER + i] = real ? gv * x : 0.f;
    }
    dot += __shfl_xor(dot, 1, 64);
    dot += __shfl_xor(dot, 2, 64);
    if (q4 == 0) dgate[tok] = real ? (1.0f - gv * gv) * dot : 0.f;
    __syncthreads();
    for (int d = tid; d < D; d += 256) {
        float s = 0.f;
        for (int r = 0; r < 64; ++r) s += part[r][d];
        from_f32(doc[cube * D + d], s);
    }
}

// MeanPool adjoint: dx[token] += dxc[n * Gp + g(token)] / P, one thread per
// 8 elements of a token.  On a padded grid P counts the real tokens of the
// sub-cube and padding tokens receive nothing.
template <typename T, int D>
__global__ __launch_bounds__(256) void unpool_add_kernel(const T* __restrict__ dxc, T* __restrict__ dx,
                                                         int64_t ntok, int64_t L, int64_t Lj, int N, int Pt,
                                                         int Ph, int Pw, cube_grid grid) {
    constexpr int PARTS = D / 8;
    const int64_t t = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    const int64_t tok = t / PARTS;                   // video token (bh, l): bh * L + l
    if (tok >= ntok) return;
    const int Bt = grid.Bt, Bh = grid.Bh, Bw = grid.Bw;
    const int d0 = static_cast<int>(t % PARTS) * 8;
    const int B = Bt * Bh * Bw;
    const int64_t cube = tok / B;                    // bh * N + n (L = N * B)
    const int beta = static_cast<int>(tok % B);
    const int bw = beta % Bw, bhh = (beta / Bw) % Bh, bt = beta / (Bw * Bh);
    const int Gh = Bh / Ph, Gw = Bw / Pw, Gp = (Bt / Pt) * Gh * Gw;
    const int g = ((bt / Pt) * Gh + bhh / Ph) * Gw + bw / Pw;
    int cnt = Pt * Ph * Pw;
    if (grid.padded) {
        const int3 e = cube_extent(grid, static_cast<int>(cube % N));
        if (!token_in(grid, e, beta)) return;
        const int ot = (bt / Pt) * Pt, oh = (bhh / Ph) * Ph, ow = (bw / Pw) * Pw;   // sub-cube origin
        cnt = min(Pt, e.x - ot) * min(Ph, e.y - oh) * min(Pw, e.z - ow);
    }
    const float inv = 1.0f / static_cast<float>(cnt);
    const T* src = dxc + (cube * Gp + g) * D + d0;
    T* dst = dx + ((tok / L) * Lj + tok % L) * D + d0;   // sequences of Lj tokens (video first)
#pragma unroll
    for (int i = 0; i < 8; ++i) from_f32(dst[i], fmaf(to_f32(src[i]), inv, to_f32(dst[i])));
}

// ---------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------
#define VSA2_COARSE_DISPATCH(...)                                                   \
    if (dtype == 1) {                                                               \
        if (D == 64) { using T = bf16_t; constexpr int DD = 64; __VA_ARGS__; }      \
        if (D == 128) { using T = bf16_t; constexpr int DD = 128; __VA_ARGS__; }    \
    } else {                                                                        \
        if (D == 64) { using T = float; constexpr int DD = 64; __VA_ARGS__; }       \
        if (D == 128) { using T = float; constexpr int DD = 128; __VA_ARGS__; }     \
    }                                                                               \
    return hipErrorInvalidValue

hipError_t launch_coarse_fwd(int dtype, int D, const void* qc, const void* kc, const void* vc, void* oc,
                             float* lse, int batch, int Hq, int Hkv, int N, hipStream_t s) {
    const dim3 grid(static_cast<unsigned>((N + 63) / 64), static_cast<unsigned>(batch * Hq));
    const float c = kLog2eC / sqrtf(static_cast<float>(D));
    VSA2_COARSE_DISPATCH(hipLaunchKernelGGL((coarse_fwd_kernel<T, DD, false>), grid, dim3(CB_NT), 0, s,
                                            static_cast<const T*>(qc), static_cast<const T*>(kc),
                                            static_cast<const T*>(vc), static_cast<T*>(oc), lse, nullptr, nullptr,
                                            Hq, Hkv, N, c);
                         return hipGetLastError());
}

hipError_t launch_coarse_bwd(int dtype, int D, const void* qc, const void* kc, const void* vc, const void* doc,
                             void* dqc, void* dkc, void* dvc, void* ws, int batch, int Hq, int Hkv, int N,
                             hipStream_t s) {
    // (LSE log2 e, Delta) per coarse query from a recomputed forward, then
    // the key and query sides
    hipError_t e = hipSuccess;
    const float c = kLog2eC / sqrtf(static_cast<float>(D));
    const float scale = 1.0f / sqrtf(static_cast<float>(D));
    float2* st = static_cast<float2*>(ws);
    const dim3 kgrid(static_cast<unsigned>((N + 63) / 64), static_cast<unsigned>(batch * Hkv));
    const dim3 qgrid(static_cast<unsigned>((N + 63) / 64), static_cast<unsigned>(batch * Hq));
    VSA2_COARSE_DISPATCH(
        hipLaunchKernelGGL((coarse_fwd_kernel<T, DD, true>), qgrid, dim3(CB_NT), 0, s, static_cast<const T*>(qc),
                           static_cast<const T*>(kc), static_cast<const T*>(vc), nullptr, nullptr,
                           static_cast<const T*>(doc), st, Hq, Hkv, N, c);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        hipLaunchKernelGGL((coarse_dkdv_kernel<T, DD>), kgrid, dim3(CB_NT), 0, s, static_cast<const T*>(qc),
                           static_cast<const T*>(kc), static_cast<const T*>(vc), static_cast<const T*>(doc), st,
                           static_cast<T*>(dkc), static_cast<T*>(dvc), Hq, Hkv, N, c, scale);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        hipLaunchKernelGGL((coarse_dq_kernel<T, DD>), qgrid, dim3(CB_NT), 0, s, static_cast<const T*>(qc),
                           static_cast<const T*>(kc), static_cast<const T*>(vc), static_cast<const T*>(doc), st,
                           static_cast<T*>(dqc), Hq, Hkv, N, c, scale);
        return hipGetLastError());
}

hipError_t launch_gate_merge(int dtype, int D, const float* gate, const void* oc, const void* of, void* out,
                             int64_t ntok, int64_t L, int64_t Lj, int N, hipStream_t s) {
    if (ntok == 0) return hipSuccess;
    const unsigned blocks = static_cast<unsigned>((ntok * (D / 8) + 255) / 256);
    VSA2_COARSE_DISPATCH(hipLaunchKernelGGL((gate_merge_kernel<T, DD>), dim3(blocks), dim3(256), 0, s, gate,
                                            static_cast<const T*>(oc), static_cast<const T*>(of),
                                            static_cast<T*>(out), ntok, L, Lj, N);
                         return hipGetLastError());
}

hipError_t launch_gate_merge_bwd(int dtype, int D, const float* gate, const void* oc, const void* dout, void* doc,
                                 float* dgate, int64_t ncubes, int N, int M, const cube_grid& cg, hipStream_t s) {
    if (ncubes == 0) return hipSuccess;
    const int64_t blocks = ncubes + ncubes / N * M;     // video cubes, then the text blocks
    VSA2_COARSE_DISPATCH(hipLaunchKernelGGL((gate_merge_bwd_kernel<T, DD>), dim3(static_cast<unsigned>(blocks)),
                                            dim3(256), 0, s, gate, static_cast<const T*>(oc),
                                            static_cast<const T*>(dout), static_cast<T*>(doc), dgate, ncubes, N,
                                            M, cg);
                         return hipGetLastError());
}

hipError_t launch_unpool_add(int dtype, int D, const void* dxc, void* dx, int64_t ntok, int64_t L, int64_t Lj,
                             int N, const cube_grid& cg, int Pt, int Ph, int Pw, hipStream_t s) {
    if (ntok == 0) return hipSuccess;
    const unsigned blocks = static_cast<unsigned>((ntok * (D / 8) + 255) / 256);
    VSA2_COARSE_DISPATCH(hipLaunchKernelGGL((unpool_add_kernel<T, DD>), dim3(blocks), dim3(256), 0, s,
                                            static_cast<const T*>(dxc), static_cast<T*>(dx), ntok, L, Lj, N, Pt,
                                            Ph, Pw, cg);
                         return hipGetLastError());
}
#undef VSA2_COARSE_DISPATCH

}  // namespace vsa2
