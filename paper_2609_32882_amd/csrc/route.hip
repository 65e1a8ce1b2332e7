// Pooling and the fine-grained router (VSA2 Sec. 2.2, Eq. router_start ..
// Eq. router_end), selection and the sparse block lists.
//
//   pool_kernel          MeanPool over sub-cubes, fp64 sums, one rounding
//   route_pass_kernel    pass 1: row log-sum-exp of Q_r K_r^T / sqrt(D)
//                        pass 2: softmax + G x G pooling into block scores
//   select_kernel        per-row top-k / mass selection by bisection on the
//                        fp32 bit pattern, register resident, one wave a row
//   scan / CSC kernels   CSR offsets, and the transposed (key-block) lists
#include <type_traits>

#include "common.hpp"
#include "internal.hpp"

namespace vsa2 {

// ===========================================================================
// Pool
// ===========================================================================
// One thread per (output row, 8-element chunk of D).  Output row
// (bh*N + n)*G + g averages the real tokens of sub-cube g of cube n (of a
// sequence of Lj tokens: the N*B video tokens, then any text tokens): all
// Pt*Ph*Pw of them unless the grid is padded, where the real tokens of a
// sub-cube form a box and an all-padding sub-cube pools to 0.
// FP = 2: sub-cubes of 2 x 2 x 2 tokens (the router's pool), the eight
// loads unrolled and issued together; FP = 0: any sub-cube (runtime loops).
template <typename T, int FP>
__global__ __launch_bounds__(256) void pool_kernel(const T* __restrict__ x, T* __restrict__ out,
                                                   int64_t nthreads, int N, int64_t Lj, int D, int G, int Gh,
                                                   int Gw, int Pt, int Ph, int Pw, int B, cube_grid grid) {
    const int64_t t = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (t >= nthreads) return;
    const int chunks = D / 8;
    const int ch = static_cast<int>(t % chunks);
    const int64_t orow = t / chunks;                  // (bh*N + n)*G + g
    const int g = static_cast<int>(orow % G);
    const int64_t cube = orow / G;                   // bh*N + n
    const int gt = g / (Gh * Gw), gh = (g / Gw) % Gh, gw = g % Gw;
    const int Bh = grid.Bh, Bw = grid.Bw;
    const T* xc = x + ((cube / N) * Lj + (cube % N) * B) * D;   // the cube's first token
    // real part of the sub-cube: [0, et) x [0, eh) x [0, ew) of its offsets
    int et = Pt, eh = Ph, ew = Pw;
    if (grid.padded) {
        const int3 e = cube_extent(grid, static_cast<int>(cube % N));
        et = max(0, min(Pt, e.x - gt * Pt));
        eh = max(0, min(Ph, e.y - gh * Ph));
        ew = max(0, min(Pw, e.z - gw * Pw));
    }
    double acc[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[i] = 0.0;
    // adds token (rt, rh, rw) of the sub-cube when `in` (else reads it and
    // leaves the sums as they are: its contents never reach them)
    auto add_token = [&](int rt, int rh, int rw, bool in) {
        const int beta = ((gt * Pt + rt) * Bh + gh * Ph + rh) * Bw + gw * Pw + rw;
        const T* src = xc + beta * D + ch * 8;
        double f[8];
        if constexpr (sizeof(T) == 2) {
            const uint4 wv = *reinterpret_cast<const uint4*>(src);
            const uint32_t u[4] = {wv.x, wv.y, wv.z, wv.w};
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                f[2 * i] = static_cast<double>(bf16_to_f32(u[i] & 0xffffu));
                f[2 * i + 1] = static_cast<double>(bf16_to_f32(u[i] >> 16));
            }
        } else {
            const float4 a = reinterpret_cast<const float4*>(src)[0];
            const float4 b = reinterpret_cast<const float4*>(src)[1];
            const float g[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
#pragma unroll
            for (int i = 0; i < 8; ++i) f[i] = static_cast<double>(g[i]);
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[i] = in ? acc[i] + f[i] : acc[i];
    };
    if constexpr (FP > 0) {
        // fixed bounds, no branch: for a token outside the real part of a
        // cut sub-cube the sub-cube's first token is read (it exists in
        // memory) and not added, so the eight loads issue together
#pragma unroll
        for (int rt = 0; rt < FP; ++rt)
#pragma unroll
            for (int rh = 0; rh < FP; ++rh)
#pragma unroll
                for (int rw = 0; rw < FP; ++rw) {
                    const bool in = rt < et && rh < eh && rw < ew;
                    add_token(in ? rt : 0, in ? rh : 0, in ? rw : 0, in);
                }
    } else {
        for (int rt = 0; rt < et; ++rt)
            for (int rh = 0; rh < eh; ++rh)
                for (int rw = 0; rw < ew; ++rw) add_token(rt, rh, rw, true);
    }
    const int cnt = et * eh * ew;
    const double P = static_cast<double>(cnt > 0 ? cnt : 1);
    T* dst = out + orow * D + ch * 8;
    if constexpr (sizeof(T) == 2) {
        uint32_t u[4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
            u[i] = static_cast<uint32_t>(f64_to_bf16(acc[2 * i] / P)) |
                   (static_cast<uint32_t>(f64_to_bf16(acc[2 * i + 1] / P)) << 16);
        *reinterpret_cast<uint4*>(dst) = make_uint4(u[0], u[1], u[2], u[3]);
    } else {
        float f[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) f[i] = __double2float_rn(acc[i] / P);
        reinterpret_cast<float4*>(dst)[0] = make_float4(f[0], f[1], f[2], f[3]);
        reinterpret_cast<float4*>(dst)[1] = make_float4(f[4], f[5], f[6], f[7]);
    }
}

hipError_t launch_pool(int dtype, const void* x, void* out, int64_t nbh, int N, int64_t Lj, int D,
                       const cube_grid& grid, int Pt, int Ph, int Pw, hipStream_t s) {
    const int Bt = grid.Bt, Bh = grid.Bh, Bw = grid.Bw;
    const int Gt = Bt / Pt, Gh = Bh / Ph, Gw = Bw / Pw, G = Gt * Gh * Gw;
    const int64_t nthreads = nbh * N * G * (D / 8);
    if (nthreads == 0) return hipSuccess;
    const int64_t blocks = (nthreads + 255) / 256;
    const int B = Bt * Bh * Bw;
    auto go = [&](auto elem, auto fixed) {
        using E = decltype(elem);
        hipLaunchKernelGGL((pool_kernel<E, decltype(fixed)::value>), dim3(blocks), dim3(256), 0, s,
                           static_cast<const E*>(x), static_cast<E*>(out), nthreads, N, Lj, D, G, Gh, Gw, Pt, Ph,
                           Pw, B, grid);
    };
    const bool two = Pt == 2 && Ph == 2 && Pw == 2;
    if (dtype == 1) {
        if (two) go(bf16_t{}, std::integral_constant<int, 2>{}); else go(bf16_t{}, std::integral_constant<int, 0>{});
    } else {
        if (two) go(0.f, std::integral_constant<int, 2>{}); else go(0.f, std::integral_constant<int, 0>{});
    }
    return hipGetLastError();
}

// ===========================================================================
// Router passes
// ===========================================================================
// Grid: x = tiles of 256 pooled queries, y = batch*Hq.  Four waves, each
// owning 64 pooled queries (two 32-column tiles).  The transposed product
// S^T = K_r Q_r^T puts one pooled query per accumulator column, so a lane
// holds 16 keys of one query: per-query reductions are lane-local plus one
// exchange with the other half-wave.  K_r streams through LDS in 64-key
// tiles, stored with the bit-2/3 slot swap so each lane's 16 keys form runs
// of 8 consecutive keys (G | 8 keys of a run make whole key blocks).
//   PASS 1: lse2[i] = log2 sum_j 2^(s_ij * log2(e)/sqrt(D))  (log2 units)
//   PASS 2: P_r[nq][nk] = (1/G^2) sum_{gq,gk} 2^(t - lse2)
// On a padded grid, pooled tokens whose sub-cube holds no real token are
// masked: such keys get no mass, such queries add nothing, and the G x G
// pooling averages over the G' pooled queries of the cube that do hold one
// (weight 1/(G G')), so every row still sums to 1/G.
constexpr int RT_Q = 256;   // pooled queries per workgroup
constexpr int RT_NT = 256;  // threads per workgroup

// Sub-cube gk (pool Rt x Rh x Rw) of a cube with real extent e holds a real
// token iff its first token is real (the real tokens form a box).
__device__ __forceinline__ bool subcube_real(const cube_grid& g, int3 e, int gk, int Rt, int Rh, int Rw) {
    const int Gh = g.Bh / Rh, Gw = g.Bw / Rw;
    const int gw = gk % Gw, r = gk / Gw;
    const int gh = r % Gh, gt = r / Gh;
    return gt * Rt < e.x && gh * Rh < e.y && gw * Rw < e.z;
}

// Sub-cubes of a cube with real extent e that hold a real token.
__device__ __forceinline__ int subcubes_real(int3 e, int Rt, int Rh, int Rw) {
    return ((e.x + Rt - 1) / Rt) * ((e.y + Rh - 1) / Rh) * ((e.z + Rw - 1) / Rw);
}

template <typename T, int D, int G, int PASS, bool PAD>
__global__ __launch_bounds__(RT_NT) void route_pass_kernel(
    const T* __restrict__ qr, const T* __restrict__ kr, float* __restrict__ lse2,
    float* __restrict__ scores, int Hq, int Hkv, int N, float c_log2, cube_grid grid, int Rt, int Rh, int Rw) {
    using F = typename frag_of<T>::type;
    constexpr int E = sizeof(T);
    constexpr int KS = D / 16;
    static_assert(G == 1 || G == 2 || G == 4 || G == 8, "pooled tokens per cube: 1, 2, 4 or 8");
    using AT = async_tile<64, D * E, RT_NT / 64, true, E == 2>;   // K_r rows (slot-swapped)
    __shared__ __align__(1024) char kt_lds[2][AT::BYTES];           // double buffer

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, half = lane >> 5;
    const int bh = blockIdx.y;
    const int b = bh / Hq, h = bh % Hq, hkv = h / (Hq / Hkv);
    const int64_t NG = static_cast<int64_t>(N) * G;
    const T* qbase = qr + static_cast<int64_t>(bh) * NG * D;
    const T* kbase = kr + static_cast<int64_t>(b * Hkv + hkv) * NG * D;
    const int64_t q0 = static_cast<int64_t>(blockIdx.x) * RT_Q + wave * 64;   // wave's first query

    F qf[2][KS];
#pragma unroll
    for (int qt = 0; qt < 2; ++qt) {
        const int64_t qi = q0 + qt * 32 + (lane & 31);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            if (qi < NG) load_frag(qf[qt][ks], qbase + qi * D + ks * 16 + half * 8);
            else {
                float z[8] = {0, 0, 0, 0, 0, 0, 0, 0};
                pack_frag(qf[qt][ks], z);
            }
        }
    }
    float m[2] = {-INFINITY, -INFINITY}, l[2] = {0.f, 0.f};
    float lq[2] = {0.f, 0.f};
    float qw[2] = {0.f, 0.f};          // pooling weight of the lane's pooled query
    if constexpr (PASS == 2) {
#pragma unroll
        for (int qt = 0; qt < 2; ++qt) {
            const int64_t qi = q0 + qt * 32 + (lane & 31);
            lq[qt] = qi < NG ? lse2[static_cast<int64_t>(bh) * NG + qi] : 0.f;
            qw[qt] = 1.0f / static_cast<float>(G * G);
            if (PAD && qi < NG) {
                const int3 e = cube_extent(grid, static_cast<int>(qi / G));
                qw[qt] = subcube_real(grid, e, static_cast<int>(qi % G), Rt, Rh, Rw)
                             ? 1.0f / static_cast<float>(G * subcubes_real(e, Rt, Rh, Rw))
                             : 0.f;
            }
        }
    }

    // K_r tiles stream through two LDS buffers with asynchronous copies: the
    // next tile's copy is issued before this tile's products
    const AT at(wave, lane);
    const int64_t ntiles = (NG + 63) / 64;
    auto issue_tile = [&](int64_t t) {
        const char* src = reinterpret_cast<const char*>(kbase + t * 64 * D);
        const int64_t rows = NG - t * 64;
        if (rows >= 64) at.issue(kt_lds[t & 1], src, wave);
        else at.issue_rows(kt_lds[t & 1], src, wave, lane, rows);
    };
    for (int qt = 0; qt < 2; ++qt)
        for (int ks = 0; ks < KS; ++ks) settle(qf[qt][ks]);   // fragments in registers before the copies start
    issue_tile(0);
    for (int64_t t = 0; t < ntiles; ++t) {
        const int64_t j0 = t * 64;
        const bool has_next = t + 1 < ntiles;
        if (has_next) issue_tile(t + 1);
        if (has_next) vm_wait<AT::PER_WAVE>(); else vm_wait<0>();   // tile t landed
        wg_barrier();
        const char* kt_l = kt_lds[t & 1];
        // bit jl: key j0 + jl exists (and, on a padded grid, holds a real
        // token); a tile without a missing key takes the mask-free path
        uint64_t kmask;
        if constexpr (PAD) {
            const int64_t j = j0 + lane;
            bool ok = j < NG;
            if (ok)
                ok = subcube_real(grid, cube_extent(grid, static_cast<int>(j / G)), static_cast<int>(j % G), Rt, Rh,
                                  Rw);
            kmask = __ballot(ok);
        } else {
            const int64_t nv = NG - j0;
            kmask = nv >= 64 ? ~0ull : ((1ull << nv) - 1);
        }
        f32x16_t acc[2][2];
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
            for (int qt = 0; qt < 2; ++qt)
#pragma unroll
                for (int v = 0; v < 16; ++v) acc[kt][qt][v] = 0.f;
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                F a;
                lds_frag_s<D * E>(a, kt_l, kt * 32 + (lane & 31), ks * 16 + half * 8);
                mma(acc[kt][0], a, qf[0][ks]);
                mma(acc[kt][1], a, qf[1][ks]);
            }
        }
        // key of accumulator entry v in key tile kt: j0 + 32kt + 16(v/8) + 8*half + v%8.
        // Keys that are not there get score -inf, i.e. probability 0 below
        // (a tile with a missing key is the last one or holds padding).
        if (kmask != ~0ull) {
#pragma unroll
            for (int kt = 0; kt < 2; ++kt)
#pragma unroll
                for (int qt = 0; qt < 2; ++qt)
#pragma unroll
                    for (int v = 0; v < 16; ++v) {
                        const int jl = kt * 32 + (v >> 3) * 16 + half * 8 + (v & 7);
                        acc[kt][qt][v] = ((kmask >> jl) & 1) ? acc[kt][qt][v] : -INFINITY;
                    }
        }
        {
            if constexpr (PASS == 1) {
#pragma unroll
                for (int qt = 0; qt < 2; ++qt) {
                    // the max of the raw scores scales to the max of the
                    // scaled ones (c > 0, rounding is monotonic)
                    float mt = -INFINITY;
#pragma unroll
                    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
                        for (int v = 0; v < 16; ++v) mt = fmaxf(mt, acc[kt][qt][v]);
                    mt = fmaxf(mt, swap_half(mt)) * c_log2;
                    const float mn = fmaxf(m[qt], mt);
                    float s = 0.f;
#pragma unroll
                    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
                        for (int v = 0; v < 16; ++v) s += fast_exp2(fmaf(acc[kt][qt][v], c_log2, -mn));
                    l[qt] = l[qt] * fast_exp2(m[qt] - mn) + s;
                    m[qt] = mn;
                }
            } else {
                // block sums bsv[qt][kt][run][i] of the lane's pooled query over
                // the G keys j0 + 32kt + 16run + 8half + iG + (0..G-1), weighted,
                // then summed over the G pooled queries of the block (G adjacent
                // lanes, within a row of 16): swap neighbours, then pairs, then
                // the two quads of 8 (mirror: lane i meets lane 7 - i).  All
                // sums first, so the lane exchanges of different blocks overlap.
                float bsv[2][2][2][8 / G];
#pragma unroll
                for (int qt = 0; qt < 2; ++qt)
#pragma unroll
                    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
                        for (int run = 0; run < 2; ++run)
#pragma unroll
                            for (int i = 0; i < 8 / G; ++i) {
                                float x = 0.f;
#pragma unroll
                                for (int u = 0; u < G; ++u)
                                    x += fast_exp2(fmaf(acc[kt][qt][run * 8 + i * G + u], c_log2, -lq[qt]));
                                bsv[qt][kt][run][i] = x * qw[qt];
                            }
#pragma unroll
                for (int qt = 0; qt < 2; ++qt)
#pragma unroll
                    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
                        for (int run = 0; run < 2; ++run)
#pragma unroll
                            for (int i = 0; i < 8 / G; ++i) {
                                float& x = bsv[qt][kt][run][i];
                                if constexpr (G >= 2) x += dpp_f32<0xB1>(x);     // quad_perm [1,0,3,2]
                                if constexpr (G >= 4) x += dpp_f32<0x4E>(x);     // quad_perm [2,3,0,1]
                                if constexpr (G >= 8) x += dpp_f32<0x141>(x);    // row_half_mirror
                            }
                if ((lane % G) == 0) {
#pragma unroll
                    for (int qt = 0; qt < 2; ++qt) {
                        const int64_t qi = q0 + qt * 32 + (lane & 31);
                        if (qi < NG) {
                            float* srow = scores + (static_cast<int64_t>(bh) * N + qi / G) * N;
#pragma unroll
                            for (int kt = 0; kt < 2; ++kt)
#pragma unroll
                                for (int run = 0; run < 2; ++run)
#pragma unroll
                                    for (int i = 0; i < 8 / G; ++i) {
                                        const int64_t j = j0 + kt * 32 + run * 16 + half * 8 + i * G;
                                        if (j < NG) srow[j / G] = bsv[qt][kt][run][i];
                                    }
                        }
                    }
                }
            }
        }
        wg_barrier();                      // buffer t & 1 is free for tile t + 2
    }
    if constexpr (PASS == 1) {
#pragma unroll
        for (int qt = 0; qt < 2; ++qt) {
            const float lt = l[qt] + swap_half(l[qt]);
            const int64_t qi = q0 + qt * 32 + (lane & 31);
            if (half == 0 && qi < NG) lse2[static_cast<int64_t>(bh) * NG + qi] = m[qt] + log2f(lt);
        }
    }
}

template <typename T, int D, int G>
static hipError_t launch_route_passes_t(const void* qr, const void* kr, float* lse2, float* scores,
                                        int batch, int Hq, int Hkv, int N, const cube_grid& cg, int Rt, int Rh,
                                        int Rw, hipStream_t s) {
    const int64_t NG = static_cast<int64_t>(N) * G;
    dim3 grid(static_cast<unsigned>((NG + RT_Q - 1) / RT_Q), static_cast<unsigned>(batch * Hq));
    const float c = 1.4426950408889634f / sqrtf(static_cast<float>(D));
    auto go = [&](auto pad) {
        constexpr bool P = decltype(pad)::value;
        hipLaunchKernelGGL((route_pass_kernel<T, D, G, 1, P>), grid, dim3(RT_NT), 0, s, static_cast<const T*>(qr),
                           static_cast<const T*>(kr), lse2, scores, Hq, Hkv, N, c, cg, Rt, Rh, Rw);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL((route_pass_kernel<T, D, G, 2, P>), grid, dim3(RT_NT), 0, s, static_cast<const T*>(qr),
                           static_cast<const T*>(kr), lse2, scores, Hq, Hkv, N, c, cg, Rt, Rh, Rw);
        return hipGetLastError();
    };
    return cg.padded ? go(std::true_type{}) : go(std::false_type{});
}

template <typename T, int D>
static hipError_t launch_route_passes_d(int G, const void* qr, const void* kr, float* lse2,
                                        float* scores, int batch, int Hq, int Hkv, int N, const cube_grid& cg,
                                        int Rt, int Rh, int Rw, hipStream_t s) {
    switch (G) {
        case 1: return launch_route_passes_t<T, D, 1>(qr, kr, lse2, scores, batch, Hq, Hkv, N, cg, Rt, Rh, Rw, s);
        case 2: return launch_route_passes_t<T, D, 2>(qr, kr, lse2, scores, batch, Hq, Hkv, N, cg, Rt, Rh, Rw, s);
        case 4: return launch_route_passes_t<T, D, 4>(qr, kr, lse2, scores, batch, Hq, Hkv, N, cg, Rt, Rh, Rw, s);
        case 8: return launch_route_passes_t<T, D, 8>(qr, kr, lse2, scores, batch, Hq, Hkv, N, cg, Rt, Rh, Rw, s);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_route_passes(int dtype, int D, int G, const void* qr, const void* kr, float* lse2,
                               float* scores, int batch, int Hq, int Hkv, int N, const cube_grid& cg, int Rt,
                               int Rh, int Rw, hipStream_t s) {
    if (dtype == 1) {
        if (D == 64) return launch_route_passes_d<bf16_t, 64>(G, qr, kr, lse2, scores, batch, Hq, Hkv, N, cg, Rt, Rh, Rw, s);
        if (D == 128) return launch_route_passes_d<bf16_t, 128>(G, qr, kr, lse2, scores, batch, Hq, Hkv, N, cg, Rt, Rh, Rw, s);
    } else {
        if (D == 64) return launch_route_passes_d<float, 64>(G, qr, kr, lse2, scores, batch, Hq, Hkv, N, cg, Rt, Rh, Rw, s);
        if (D == 128) return launch_route_passes_d<float, 128>(G, qr, kr, lse2, scores, batch, Hq, Hkv, N, cg, Rt, Rh, Rw, s);
    }
    return hipErrorInvalidValue;
}

// ===========================================================================
// Selection
// ===========================================================================
// One wave per query-block row of N scores (N <= 64*PER), held in registers:
// element j = 64*i + lane.  Scores are >= 0, so float order equals the order
// of their bit patterns and a 31-step bisection on the bits finds exact
// thresholds.  Ties at the threshold go to the lowest block indices, which
// reproduces the order (score desc, index asc).
__device__ __forceinline__ int wave_sum_i(int x) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) x += __shfl_xor(x, off, 64);
    return x;
}
__device__ __forceinline__ double wave_sum_d(double x) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) x += __shfl_xor(x, off, 64);
    return x;
}

// Number of the wave's entries with x > t (STRICT) or x >= t: one ballot
// per register and a population count, no lane exchanges.
template <int PER, bool STRICT>
__device__ __forceinline__ int wave_count(const float (&x)[PER], float t) {
    int c = 0;
#pragma unroll
    for (int i = 0; i < PER; ++i) c += __popcll(__ballot(STRICT ? x[i] > t : x[i] >= t));
    return c;
}

// Largest threshold t (as bits) with count(x >= t) >= k: the k-th largest value.
template <int PER>
__device__ __forceinline__ uint32_t kth_largest_bits(const float (&x)[PER], int k) {
    uint32_t tau = 0;
    for (int bit = 30; bit >= 0; --bit) {
        const uint32_t cand = tau | (1u << bit);
        if (wave_count<PER, false>(x, __uint_as_float(cand)) >= k) tau = cand;
    }
    return tau;
}

struct row_rule {
    float tau;      // threshold value
    int need;       // how many of the entries equal to tau are kept (lowest indices)
    int count;      // total kept
};

template <int PER>
__device__ row_rule decide_row(const float (&x)[PER], int N, int mode, int k, float mass, int cap) {
    row_rule r;
    int keep;
    if (mode == 0) {
        keep = k < N ? k : N;
    } else {
        double tot = 0.0;
#pragma unroll
        for (int i = 0; i < PER; ++i) tot += x[i] > 0.f ? static_cast<double>(x[i]) : 0.0;
        tot = wave_sum_d(tot);
        const double thr = static_cast<double>(mass) * tot;
        if (!(thr > 0.0)) {
            keep = 1;
        } else {
            // largest t with S(t) = sum_{x >= t} x >= thr
            uint32_t tau = 0;
            for (int bit = 30; bit >= 0; --bit) {
                const uint32_t cand = tau | (1u << bit);
                const float cf = __uint_as_float(cand);
                double s = 0.0;
#pragma unroll
                for (int i = 0; i < PER; ++i) s += x[i] >= cf ? static_cast<double>(x[i]) : 0.0;
                if (wave_sum_d(s) >= thr) tau = cand;
            }
            const float tf = __uint_as_float(tau);
            double sg = 0.0;
            int gt = 0, eq = 0;
#pragma unroll
            for (int i = 0; i < PER; ++i) {
                if (x[i] > tf) { sg += static_cast<double>(x[i]); ++gt; }
                else if (x[i] == tf) ++eq;
            }
            sg = wave_sum_d(sg);
            gt = wave_sum_i(gt);
            eq = wave_sum_i(eq);
            // ties added one at a time, lowest index first, until the sum reaches thr
            int m = 0;
            double cum = sg;
            while (m < eq && cum < thr) { cum += static_cast<double>(tf); ++m; }
            keep = gt + (m > 0 ? m : (eq > 0 ? 1 : 0));
            if (keep > N) keep = N;
        }
        if (keep > cap) keep = cap;
    }
    const uint32_t tau = kth_largest_bits<PER>(x, keep);
    const float tf = __uint_as_float(tau);
    const int gt = wave_count<PER, true>(x, tf);
    r.tau = tf;
    r.need = keep - gt;
    r.count = keep;
    return r;
}

// PHASE 0: counts[row] = number kept.  PHASE 1: write the kept block indices,
// ascending, at col_idx[row_ptr[row] ...].
template <int PER, int PHASE>
__global__ __launch_bounds__(256) void select_kernel(const float* __restrict__ scores, int64_t nrows,
                                                     int N, int mode, int k, float mass, int cap,
                                                     int32_t* __restrict__ counts,
                                                     const int32_t* __restrict__ row_ptr,
                                                     int32_t* __restrict__ col_idx, int64_t col_cap) {
    const int lane = threadIdx.x & 63;
    const int64_t row = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
    if (row >= nrows) return;
    float x[PER];
    const float* src = scores + row * N;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
        const int j = i * 64 + lane;
        x[i] = j < N ? src[j] : -1.0f;   // padding never reaches a threshold >= 0
    }
    const row_rule r = decide_row<PER>(x, N, mode, k, mass, cap);
    if constexpr (PHASE == 0) {
        if (lane == 0) counts[row] = r.count;
    } else {
        int64_t pos = row_ptr[row];
        int ties = 0;
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const bool eq = x[i] == r.tau;
            const uint64_t eqm = __ballot(eq);
            const int rank = ties + __popcll(eqm & ((1ull << lane) - 1ull));
            const bool sel = x[i] > r.tau || (eq && rank < r.need);
            const uint64_t sm = __ballot(sel);
            if (sel) {
                const int64_t at = pos + __popcll(sm & ((1ull << lane) - 1ull));
                if (at < col_cap) col_idx[at] = i * 64 + lane;
            }
            pos += __popcll(sm);
            ties += __popcll(eqm);
        }
    }
}

template <int PER>
static hipError_t launch_select_per(int phase, const float* scores, int64_t nrows, int N, int mode,
                                    int k, float mass, int cap, int32_t* counts,
                                    const int32_t* row_ptr, int32_t* col_idx, int64_t col_cap,
                                    hipStream_t s) {
    dim3 grid(static_cast<unsigned>((nrows + 3) / 4));
    if (phase == 0)
        hipLaunchKernelGGL((select_kernel<PER, 0>), grid, dim3(256), 0, s, scores, nrows, N, mode, k,
                           mass, cap, counts, row_ptr, col_idx, col_cap);
    else
        hipLaunchKernelGGL((select_kernel<PER, 1>), grid, dim3(256), 0, s, scores, nrows, N, mode, k,
                           mass, cap, counts, row_ptr, col_idx, col_cap);
    return hipGetLastError();
}

hipError_t launch_select(int phase, const float* scores, int64_t nrows, int N, int mode, int k,
                         float mass, int cap, int32_t* counts, const int32_t* row_ptr,
                         int32_t* col_idx, int64_t col_cap, hipStream_t s) {
    if (nrows == 0) return hipSuccess;
    const int per = (N + 63) / 64;
#define VSA2_SEL(P) \
    if (per <= P) return launch_select_per<P>(phase, scores, nrows, N, mode, k, mass, cap, counts, row_ptr, col_idx, col_cap, s)
    VSA2_SEL(2);
    VSA2_SEL(4);
    VSA2_SEL(8);
    VSA2_SEL(12);
    VSA2_SEL(16);
    VSA2_SEL(20);
    VSA2_SEL(24);
    VSA2_SEL(32);
    VSA2_SEL(40);
    VSA2_SEL(48);
    VSA2_SEL(64);
#undef VSA2_SEL
    return hipErrorInvalidValue;
}

// ===========================================================================
// Sequence-level selection: TopK_{N k} over each (batch, head)'s flattened
// N x N map of block scores (Sec. 2.2, the selection over all query-block /
// key-block pairs of a sequence).  Keeps the keep = min(N k, N^2) best pairs,
// order (score desc, flat index n_q N + n_k asc), decided on the fp32 scores.
//
//   1. threshold: radix select of the keep-th largest score per sequence,
//      8 bits at a time from the top (scores are >= 0: bit patterns order
//      like the values).  Each pass histograms the digit of the entries that
//      match the prefix found so far (chunked over many workgroups, LDS
//      histograms merged with integer atomics), then one thread per sequence
//      picks the digit.  Result: tau and need = how many entries equal to
//      tau are kept (the ones with the lowest flat indices).
//   2. per row: gt = #(> tau), eq = #(== tau); per sequence, an exclusive
//      scan of eq in row order gives each row's share of the need.
//   3. offsets (scan_kernel) and the kept indices, ascending per row.
// ===========================================================================
struct seq_state {
    uint32_t prefix;   // digits of tau found so far
    int32_t rem;       // rank of the target among the entries matching prefix
};

constexpr int SEQ_NT = 256;
constexpr int SEQ_CHUNK = SEQ_NT * 64;   // entries per histogram workgroup
constexpr int SEQ_HSTRIDE = 257;         // per-lane-group histogram stride (words)

__global__ void seq_init_kernel(seq_state* __restrict__ st, uint32_t* __restrict__ ghist, int64_t nseq,
                                int64_t keep) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i < nseq) {
        st[i].prefix = 0;
        st[i].rem = static_cast<int32_t>(keep);
    }
    if (i < nseq * 256) ghist[i] = 0;
}

// grid (chunks, nseq).  Histogram of digit (v >> shift) & 255 over the
// entries of chunk blockIdx.x of sequence blockIdx.y that match the prefix.
__global__ __launch_bounds__(SEQ_NT) void seq_hist_kernel(const float* __restrict__ scores, int64_t nn,
                                                          const seq_state* __restrict__ st,
                                                          uint32_t* __restrict__ ghist, int pass) {
    // four sub-histograms per wave (lane & 3), padded so one bin of the four
    // sits in four different banks
    __shared__ uint32_t h[SEQ_NT / 64][4][SEQ_HSTRIDE];
    const int tid = threadIdx.x, wave = tid >> 6, sub = tid & 3;
    const int64_t seq = blockIdx.y;
    const int shift = 24 - 8 * pass;
    const uint32_t hi_mask = pass == 0 ? 0u : (0xffffffffu << (shift + 8));
    const uint32_t want = pass == 0 ? 0u : (st[seq].prefix << (shift + 8));
    for (int i = tid; i < (SEQ_NT / 64) * 4 * SEQ_HSTRIDE; i += SEQ_NT) (&h[0][0][0])[i] = 0;
    __syncthreads();
    const uint32_t* u = reinterpret_cast<const uint32_t*>(scores + seq * nn);
    const int64_t c0 = static_cast<int64_t>(blockIdx.x) * SEQ_CHUNK;
    const int64_t c1 = c0 + SEQ_CHUNK < nn ? c0 + SEQ_CHUNK : nn;
    for (int64_t i = c0 + tid; i < c1; i += SEQ_NT) {
        const uint32_t v = u[i];
        if ((v & hi_mask) == want) atomicAdd(&h[wave][sub][(v >> shift) & 255u], 1u);
    }
    __syncthreads();
    uint32_t sum = 0;
#pragma unroll
    for (int w = 0; w < SEQ_NT / 64; ++w)
#pragma unroll
        for (int k = 0; k < 4; ++k) sum += h[w][k][tid];
    if (sum) atomicAdd(&ghist[seq * 256 + tid], sum);
}

// One thread per sequence: the digit holding the target rank; clears the
// histogram for the next pass.  After the last pass prefix = tau's bits and
// rem = the number of entries equal to tau that are kept.
__global__ void seq_pick_kernel(seq_state* __restrict__ st, uint32_t* __restrict__ ghist, int64_t nseq) {
    const int64_t seq = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (seq >= nseq) return;
    uint32_t* h = ghist + seq * 256;
    int64_t r = st[seq].rem;
    int d = 255;
    for (; d > 0; --d) {
        if (static_cast<int64_t>(h[d]) >= r) break;
        r -= h[d];
    }
    st[seq].prefix = (st[seq].prefix << 8) | static_cast<uint32_t>(d);
    st[seq].rem = static_cast<int32_t>(r);
    for (int b = 0; b < 256; ++b) h[b] = 0;
}

// One wave per row (N <= 64*PER).  PHASE 0: gt[row], eq[row].  PHASE 1:
// write the kept indices ascending at col_idx[row_ptr[row] ...]: every entry
// > tau and the first take[row] entries == tau.
template <int PER, int PHASE>
__global__ __launch_bounds__(256) void seq_rows_kernel(const float* __restrict__ scores, int64_t nrows, int N,
                                                       const seq_state* __restrict__ st,
                                                       int32_t* __restrict__ gt, int32_t* __restrict__ eq,
                                                       const int32_t* __restrict__ take,
                                                       const int32_t* __restrict__ row_ptr,
                                                       int32_t* __restrict__ col_idx, int64_t col_cap) {
    const int lane = threadIdx.x & 63;
    const int64_t row = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
    if (row >= nrows) return;
    const float tau = __uint_as_float(st[row / N].prefix);
    float x[PER];
    const float* src = scores + row * N;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
        const int j = i * 64 + lane;
        x[i] = j < N ? src[j] : -1.0f;
    }
    if constexpr (PHASE == 0) {
        int g = 0, e = 0;
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            g += x[i] > tau ? 1 : 0;
            e += x[i] == tau ? 1 : 0;
        }
        g = wave_sum_i(g);
        e = wave_sum_i(e);
        if (lane == 0) {
            gt[row] = g;
            eq[row] = e;
        }
    } else {
        const int need = take[row];
        int64_t pos = row_ptr[row];
        int ties = 0;
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const bool is_eq = x[i] == tau;
            const uint64_t eqm = __ballot(is_eq);
            const int rank = ties + __popcll(eqm & ((1ull << lane) - 1ull));
            const bool sel = x[i] > tau || (is_eq && rank < need);
            const uint64_t sm = __ballot(sel);
            if (sel) {
                const int64_t at = pos + __popcll(sm & ((1ull << lane) - 1ull));
                if (at < col_cap) col_idx[at] = i * 64 + lane;
            }
            pos += __popcll(sm);
            ties += __popcll(eqm);
        }
    }
}

// One workgroup (1024) per sequence: take[row] = the row's share of the
// sequence's need, in row order; counts[row] = gt + take.
__global__ __launch_bounds__(1024) void seq_take_kernel(const seq_state* __restrict__ st, int N,
                                                        const int32_t* __restrict__ gt,
                                                        const int32_t* __restrict__ eq,
                                                        int32_t* __restrict__ take, int32_t* __restrict__ counts) {
    __shared__ int32_t part[1024];
    const int tid = threadIdx.x;
    const int64_t base = static_cast<int64_t>(blockIdx.x) * N;
    const int per = (N + 1023) / 1024;
    const int lo = tid * per < N ? tid * per : N;
    const int hi = lo + per < N ? lo + per : N;
    int32_t sum = 0;
    for (int i = lo; i < hi; ++i) sum += eq[base + i];
    part[tid] = sum;
    __syncthreads();
    for (int off = 1; off < 1024; off <<= 1) {
        const int32_t v = tid >= off ? part[tid - off] : 0;
        __syncthreads();
        part[tid] += v;
        __syncthreads();
    }
    int64_t before = part[tid] - sum;
    const int64_t need = st[blockIdx.x].rem;
    for (int i = lo; i < hi; ++i) {
        const int64_t e = eq[base + i];
        int64_t t = need - before;
        t = t < 0 ? 0 : (t > e ? e : t);
        take[base + i] = static_cast<int32_t>(t);
        counts[base + i] = gt[base + i] + static_cast<int32_t>(t);
        before += e;
    }
}

template <int PER>
static hipError_t launch_seq_rows(int phase, const float* scores, int64_t nrows, int N, const seq_state* st,
                                  int32_t* gt, int32_t* eq, const int32_t* take, const int32_t* row_ptr,
                                  int32_t* col_idx, int64_t col_cap, hipStream_t s) {
    dim3 grid(static_cast<unsigned>((nrows + 3) / 4));
    if (phase == 0)
        hipLaunchKernelGGL((seq_rows_kernel<PER, 0>), grid, dim3(256), 0, s, scores, nrows, N, st, gt, eq, take,
                           row_ptr, col_idx, col_cap);
    else
        hipLaunchKernelGGL((seq_rows_kernel<PER, 1>), grid, dim3(256), 0, s, scores, nrows, N, st, gt, eq, take,
                           row_ptr, col_idx, col_cap);
    return hipGetLastError();
}

static hipError_t launch_seq_rows_any(int phase, const float* scores, int64_t nrows, int N, const seq_state* st,
                                      int32_t* gt, int32_t* eq, const int32_t* take, const int32_t* row_ptr,
                                      int32_t* col_idx, int64_t col_cap, hipStream_t s) {
    const int per = (N + 63) / 64;
#define VSA2_SEQ(P) \
    if (per <= P) return launch_seq_rows<P>(phase, scores, nrows, N, st, gt, eq, take, row_ptr, col_idx, col_cap, s)
    VSA2_SEQ(2);
    VSA2_SEQ(4);
    VSA2_SEQ(8);
    VSA2_SEQ(16);
    VSA2_SEQ(24);
    VSA2_SEQ(32);
    VSA2_SEQ(40);
    VSA2_SEQ(48);
    VSA2_SEQ(64);
#undef VSA2_SEQ
    return hipErrorInvalidValue;
}

size_t seq_workspace_bytes(int64_t nseq, int64_t nrows) {
    auto a = [](size_t x) { return (x + 255) / 256 * 256; };
    return a(sizeof(seq_state) * nseq) + a(4 * 256 * nseq) + 3 * a(4 * nrows);
}

hipError_t launch_select_seq(const float* scores, int64_t nseq, int N, int k, void* ws, int32_t* counts,
                             int32_t* row_ptr, int32_t* col_idx, int64_t col_cap, hipStream_t s) {
    if (nseq == 0) return hipSuccess;
    auto a = [](size_t x) { return (x + 255) / 256 * 256; };
    const int64_t nn = static_cast<int64_t>(N) * N;
    const int64_t nrows = nseq * N;
    const int64_t keep = static_cast<int64_t>(N) * k < nn ? static_cast<int64_t>(N) * k : nn;
    char* w = static_cast<char*>(ws);
    seq_state* st = reinterpret_cast<seq_state*>(w);
    w += a(sizeof(seq_state) * nseq);
    uint32_t* ghist = reinterpret_cast<uint32_t*>(w);
    w += a(4 * 256 * nseq);
    int32_t* gt = reinterpret_cast<int32_t*>(w);
    w += a(4 * nrows);
    int32_t* eq = reinterpret_cast<int32_t*>(w);
    w += a(4 * nrows);
    int32_t* take = reinterpret_cast<int32_t*>(w);

    hipLaunchKernelGGL(seq_init_kernel, dim3(static_cast<unsigned>((nseq * 256 + 255) / 256)), dim3(256), 0, s, st,
                       ghist, nseq, keep);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const dim3 hgrid(static_cast<unsigned>((nn + SEQ_CHUNK - 1) / SEQ_CHUNK), static_cast<unsigned>(nseq));
    for (int pass = 0; pass < 4; ++pass) {
        hipLaunchKernelGGL(seq_hist_kernel, hgrid, dim3(SEQ_NT), 0, s, scores, nn, st, ghist, pass);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        hipLaunchKernelGGL(seq_pick_kernel, dim3(static_cast<unsigned>((nseq + 63) / 64)), dim3(64), 0, s, st,
                           ghist, nseq);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    if ((e = launch_seq_rows_any(0, scores, nrows, N, st, gt, eq, nullptr, nullptr, nullptr, 0, s)) != hipSuccess)
        return e;
    hipLaunchKernelGGL(seq_take_kernel, dim3(static_cast<unsigned>(nseq)), dim3(1024), 0, s, st, N, gt, eq, take,
                       counts);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = launch_scan(counts, nrows, row_ptr, s)) != hipSuccess) return e;
    return launch_seq_rows_any(1, scores, nrows, N, st, gt, eq, take, row_ptr, col_idx, col_cap, s);
}

// ===========================================================================
// Offsets and the transposed lists
// ===========================================================================
// Exclusive scan of counts[0..n) into ptr[0..n] by one workgroup of 16
// waves.  Wave w owns the contiguous segment [w seg, (w + 1) seg) and reads
// it 64 consecutive counts at a time (coalesced): a first pass sums each
// segment, the 16 totals give each wave its starting carry, and a second
// pass writes the offsets with a wave prefix sum per 64 counts.
__global__ __launch_bounds__(1024) void scan_kernel(const int32_t* __restrict__ counts, int64_t n,
                                                    int32_t* __restrict__ ptr) {
    __shared__ int32_t tot[16];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int64_t seg = (n + 15) / 16;
    const int64_t lo = w * seg, hi = lo + seg < n ? lo + seg : n;
    int32_t s = 0;
#pragma unroll 8
    for (int64_t i = lo + lane; i < hi; i += 64) s += counts[i];
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) s += __shfl_xor(s, off, 64);
    if (lane == 0) tot[w] = s;
    __syncthreads();
    int32_t carry = 0;
    for (int j = 0; j < w; ++j) carry += tot[j];
#pragma unroll 4
    for (int64_t base = lo; base < hi; base += 64) {
        const int64_t i = base + lane;
        const int32_t x = i < hi ? counts[i] : 0;
        int32_t incl = x;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const int32_t y = __shfl_up(incl, off, 64);
            if (lane >= off) incl += y;
        }
        if (i < hi) ptr[i] = carry + incl - x;
        carry += __shfl(incl, 63, 64);
    }
    if (threadIdx.x == 0) {
        int32_t t = 0;
        for (int j = 0; j < 16; ++j) t += tot[j];
        ptr[n] = t;
    }
}

hipError_t launch_scan(const int32_t* counts, int64_t n, int32_t* ptr, hipStream_t s) {
    hipLaunchKernelGGL(scan_kernel, dim3(1), dim3(1024), 0, s, counts, n, ptr);
    return hipGetLastError();
}

// Offsets of uniform rows: ptr[i] = i * k.
__global__ void uniform_ptr_kernel(int32_t* __restrict__ ptr, int64_t n, int k) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i <= n) ptr[i] = static_cast<int32_t>(i * k);
}

hipError_t launch_uniform_ptr(int32_t* ptr, int64_t n, int k, hipStream_t s) {
    hipLaunchKernelGGL(uniform_ptr_kernel, dim3(static_cast<unsigned>((n + 1 + 255) / 256)), dim3(256), 0, s,
                       ptr, n, k);
    return hipGetLastError();
}

__global__ void fill_u32_kernel(uint32_t* __restrict__ p, int64_t n, uint32_t v) {
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n;
         i += static_cast<int64_t>(gridDim.x) * blockDim.x)
        p[i] = v;
}

hipError_t launch_fill_u32(uint32_t* p, int64_t n, uint32_t v, hipStream_t s) {
    if (n == 0) return hipSuccess;
    int64_t blocks = (n + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    hipLaunchKernelGGL(fill_u32_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, s, p, n, v);
    return hipGetLastError();
}

// Mark every CSR entry in the key-block bitmask: bit (hq_local*N + nq) of
// key-block row (b*Hkv + hkv)*N + nk.  One thread per query-block row.
__global__ void csc_mark_kernel(const int32_t* __restrict__ row_ptr, const int32_t* __restrict__ col_idx,
                                int64_t nrows, int N, int Hq, int Hkv, int words, int64_t col_cap,
                                uint32_t* __restrict__ mask) {
    const int64_t row = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (row >= nrows) return;
    const int grp = Hq / Hkv;
    const int64_t bh = row / N;
    const int nq = static_cast<int>(row % N);
    const int b = static_cast<int>(bh / Hq), h = static_cast<int>(bh % Hq);
    const int hkv = h / grp, hl = h % grp;
    const int bit = hl * N + nq;
    int64_t s0 = row_ptr[row], s1 = row_ptr[row + 1];
    s0 = s0 < 0 ? 0 : (s0 > col_cap ? col_cap : s0);
    s1 = s1 < s0 ? s0 : (s1 > col_cap ? col_cap : s1);
    for (int64_t e = s0; e < s1; ++e) {
        const int nk = col_idx[e];
        if (nk < 0 || nk >= N) continue;
        const int64_t krow = static_cast<int64_t>(b * Hkv + hkv) * N + nk;
        atomicOr(mask + krow * words + (bit >> 5), 1u << (bit & 31));
    }
}

// The same marks built per (KV group, 32-bit word of its query-block bits):
// the workgroup's 32 query-block rows (8 threads each) set their bits of
// every key block in LDS (N words), then the workgroup writes those N words.
// Every mask word is written exactly once, by one workgroup, so neither
// global atomics nor a zero fill are needed.  Grid: groups x words.
constexpr int CSC_LDS_MAX_N = 16384;   // N words of LDS (64 KB)
constexpr int CSC_NT = 256;            // 32 rows x 8 threads
__global__ __launch_bounds__(CSC_NT) void csc_mark_lds_kernel(const int32_t* __restrict__ row_ptr,
                                                           const int32_t* __restrict__ col_idx, int N, int Hq,
                                                           int Hkv, int words, int64_t col_cap,
                                                           uint32_t* __restrict__ mask) {
    extern __shared__ uint32_t marks[];
    const int grp = Hq / Hkv;
    const int64_t g = blockIdx.x / words;             // b*Hkv + hkv
    const int w = static_cast<int>(blockIdx.x % words);
    const int b = static_cast<int>(g / Hkv), hkv = static_cast<int>(g % Hkv);
    for (int i = threadIdx.x; i < N; i += CSC_NT) marks[i] = 0u;
    __syncthreads();
    const int r = threadIdx.x >> 3, sub = threadIdx.x & 7;   // r < 32
    const int bit = w * 32 + r;                       // hl*N + nq
    if (bit < grp * N) {
        const int hl = bit / N, nq = bit % N;
        const int64_t row = (static_cast<int64_t>(b) * Hq + hkv * grp + hl) * N + nq;
        int64_t s0 = row_ptr[row], s1 = row_ptr[row + 1];
        s0 = s0 < 0 ? 0 : (s0 > col_cap ? col_cap : s0);
        s1 = s1 < s0 ? s0 : (s1 > col_cap ? col_cap : s1);
        for (int64_t e = s0 + sub; e < s1; e += 8) {
            const int nk = col_idx[e];
            if (nk >= 0 && nk < N) atomicOr(&marks[nk], 1u << r);
        }
    }
    __syncthreads();
    uint32_t* out = mask + g * N * words + w;         // mask[(g*N + nk)*words + w]
    for (int i = threadIdx.x; i < N; i += CSC_NT) out[static_cast<int64_t>(i) * words] = marks[i];
}

__global__ void csc_count_kernel(const uint32_t* __restrict__ mask, int64_t nkrows, int words,
                                 int32_t* __restrict__ counts) {
    const int64_t r = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (r >= nkrows) return;
    int c = 0;
    for (int w = 0; w < words; ++w) c += __popc(mask[r * words + w]);
    counts[r] = c;
}

__global__ void csc_emit_kernel(const uint32_t* __restrict__ mask, int64_t nkrows, int words,
                                const int32_t* __restrict__ kv_ptr, int32_t* __restrict__ kv_idx,
                                int64_t col_cap) {
    const int64_t r = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (r >= nkrows) return;
    int64_t pos = kv_ptr[r];
    for (int w = 0; w < words; ++w) {
        uint32_t m = mask[r * words + w];
        while (m) {
            const int bit = __ffs(m) - 1;
            m &= m - 1;
            if (pos < col_cap) kv_idx[pos] = w * 32 + bit;
            ++pos;
        }
    }
}

hipError_t launch_csc(const int32_t* row_ptr, const int32_t* col_idx, int batch, int Hq, int Hkv, int N,
                      int64_t col_cap, uint32_t* mask, int32_t* kv_counts, int32_t* kv_ptr,
                      int32_t* kv_idx, hipStream_t s) {
    const int words = (Hq / Hkv * N + 31) / 32;
    const int64_t nkrows = static_cast<int64_t>(batch) * Hkv * N;
    const int64_t nrows = static_cast<int64_t>(batch) * Hq * N;
    hipError_t e;
    const int64_t wgs = static_cast<int64_t>(batch) * Hkv * words;
    if (N <= CSC_LDS_MAX_N && wgs <= 0x7fffffff) {
        hipLaunchKernelGGL(csc_mark_lds_kernel, dim3(static_cast<unsigned>(wgs)), dim3(CSC_NT),
                           static_cast<size_t>(N) * 4, s, row_ptr, col_idx, N, Hq, Hkv, words, col_cap, mask);
    } else {
        if ((e = launch_fill_u32(mask, nkrows * words, 0u, s)) != hipSuccess) return e;
        hipLaunchKernelGGL(csc_mark_kernel, dim3(static_cast<unsigned>((nrows + 255) / 256)), dim3(256), 0, s,
                           row_ptr, col_idx, nrows, N, Hq, Hkv, words, col_cap, mask);
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(csc_count_kernel, dim3(static_cast<unsigned>((nkrows + 255) / 256)), dim3(256), 0, s,
                       mask, nkrows, words, kv_counts);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = launch_scan(kv_counts, nkrows, kv_ptr, s)) != hipSuccess) return e;
    hipLaunchKernelGGL(csc_emit_kernel, dim3(static_cast<unsigned>((nkrows + 255) / 256)), dim3(256), 0, s,
                       mask, nkrows, words, kv_ptr, kv_idx, col_cap);
    return hipGetLastError();
}

// ===========================================================================
// Joint video + text lists (MMDiT joint attention)
// ===========================================================================
// Joint row r = bh*(N+M) + n.  A video row (n < N) lists the routed video
// blocks of row bh*N + n in their order (entries outside [0, N) become -1,
// which the attention skips) and then the M text blocks N .. N+M-1; a text
// row (n >= N) lists every block 0 .. N+M-1.
__global__ void joint_count_kernel(const int32_t* __restrict__ row_ptr, int64_t col_cap, int64_t nrows_j, int N,
                                   int M, int32_t* __restrict__ counts) {
    const int64_t r = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (r >= nrows_j) return;
    const int Nj = N + M;
    const int64_t bh = r / Nj;
    const int n = static_cast<int>(r % Nj);
    if (n >= N) {
        counts[r] = Nj;
        return;
    }
    const int64_t row = bh * N + n;
    int64_t s0 = row_ptr[row], s1 = row_ptr[row + 1];
    s0 = s0 < 0 ? 0 : (s0 > col_cap ? col_cap : s0);
    s1 = s1 < s0 ? s0 : (s1 > col_cap ? col_cap : s1);
    counts[r] = static_cast<int32_t>(s1 - s0) + M;
}

// One wave per joint row; writes stay below j_cap.
__global__ __launch_bounds__(256) void joint_emit_kernel(const int32_t* __restrict__ row_ptr,
                                                         const int32_t* __restrict__ col_idx, int64_t col_cap,
                                                         int64_t nrows_j, int N, int M,
                                                         const int32_t* __restrict__ j_row_ptr,
                                                         int32_t* __restrict__ j_col_idx, int64_t j_cap) {
    const int64_t r = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (r >= nrows_j) return;
    const int Nj = N + M;
    const int64_t bh = r / Nj;
    const int n = static_cast<int>(r % Nj);
    int64_t o = j_row_ptr[r];
    o = o < 0 ? 0 : (o > j_cap ? j_cap : o);
    auto put = [&](int64_t pos, int32_t v) {
        if (pos < j_cap) j_col_idx[pos] = v;
    };
    if (n >= N) {
        for (int i = lane; i < Nj; i += 64) put(o + i, i);
        return;
    }
    const int64_t row = bh * N + n;
    int64_t s0 = row_ptr[row], s1 = row_ptr[row + 1];
    s0 = s0 < 0 ? 0 : (s0 > col_cap ? col_cap : s0);
    s1 = s1 < s0 ? s0 : (s1 > col_cap ? col_cap : s1);
    for (int64_t e = s0 + lane; e < s1; e += 64) {
        const int32_t c = col_idx[e];
        put(o + (e - s0), (c >= 0 && c < N) ? c : -1);
    }
    for (int i = lane; i < M; i += 64) put(o + (s1 - s0) + i, N + i);
}

static size_t align256b(size_t x) { return (x + 255) / 256 * 256; }

size_t joint_workspace_bytes(int batch, int Hq, int Hkv, int N, int M) {
    const int64_t Nj = static_cast<int64_t>(N) + M;
    const int64_t words = (static_cast<int64_t>(Hq / Hkv) * Nj + 31) / 32;
    const int64_t rows_q = static_cast<int64_t>(batch) * Hq * Nj, rows_kv = static_cast<int64_t>(batch) * Hkv * Nj;
    return align256b(4 * static_cast<size_t>(rows_q)) + align256b(4 * static_cast<size_t>(rows_kv * words)) +
           align256b(4 * static_cast<size_t>(rows_kv));
}

hipError_t launch_joint_lists(const int32_t* row_ptr, const int32_t* col_idx, int64_t col_cap, int batch, int Hq,
                              int Hkv, int N, int M, int32_t* j_row_ptr, int32_t* j_col_idx, int64_t j_cap,
                              int32_t* j_kv_ptr, int32_t* j_kv_idx, void* ws, hipStream_t s) {
    const int Nj = N + M;
    const int64_t nrows_j = static_cast<int64_t>(batch) * Hq * Nj;
    const int64_t rows_kv = static_cast<int64_t>(batch) * Hkv * Nj;
    const int64_t words = (static_cast<int64_t>(Hq / Hkv) * Nj + 31) / 32;
    char* base = static_cast<char*>(ws);
    int32_t* counts = reinterpret_cast<int32_t*>(base);
    uint32_t* mask = reinterpret_cast<uint32_t*>(base + align256b(4 * static_cast<size_t>(nrows_j)));
    int32_t* kv_counts = reinterpret_cast<int32_t*>(base + align256b(4 * static_cast<size_t>(nrows_j)) +
                                                    align256b(4 * static_cast<size_t>(rows_kv * words)));
    if (nrows_j == 0) return hipSuccess;
    hipLaunchKernelGGL(joint_count_kernel, dim3(static_cast<unsigned>((nrows_j + 255) / 256)), dim3(256), 0, s,
                       row_ptr, col_cap, nrows_j, N, M, counts);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if ((e = launch_scan(counts, nrows_j, j_row_ptr, s)) != hipSuccess) return e;
    hipLaunchKernelGGL(joint_emit_kernel, dim3(static_cast<unsigned>((nrows_j + 3) / 4)), dim3(256), 0, s, row_ptr,
                       col_idx, col_cap, nrows_j, N, M, j_row_ptr, j_col_idx, j_cap);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    return launch_csc(j_row_ptr, j_col_idx, batch, Hq, Hkv, Nj, j_cap, mask, kv_counts, j_kv_ptr, j_kv_idx, s);
}

}  // namespace vsa2
