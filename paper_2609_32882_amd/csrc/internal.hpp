// Host-side launchers of the gfx950 kernels (internal to the library; the
// public C-ABI in vsa2.h validates arguments and calls these).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>

namespace vsa2 {

// A T x H x W grid cut into Bt x Bh x Bw cubes (Sec. 2.2).  An axis that
// is not a multiple of its cube size is padded up to one, so the grid holds
// Nt x Nh x Nw cubes in cube-major order (n = (nt*Nh + nh)*Nw + nw, tokens
// of a cube in (bt, bh, bw) raster order).  The real tokens of a cube form
// the box [0, rt) x [0, rh) x [0, rw) of its in-cube coordinates; only the
// last cube along a padded axis is cut, and every cube holds a real token.
// With text tokens (MMDiT joint attention) a sequence continues after the
// Nv video cubes with text blocks of B tokens, the first text_len real.
struct cube_grid {
    int T, H, W;
    int Bt, Bh, Bw;
    int Nh, Nw;
    int Nv;         // video cubes per sequence
    int text_len;   // real text tokens after them
    int padded;     // some block holds padding (a cut cube or text tail)
};

inline cube_grid make_cube_grid(int T, int H, int W, int Bt, int Bh, int Bw, int text_len) {
    cube_grid g;
    g.T = T; g.H = H; g.W = W;
    g.Bt = Bt; g.Bh = Bh; g.Bw = Bw;
    g.Nh = (H + Bh - 1) / Bh;
    g.Nw = (W + Bw - 1) / Bw;
    g.Nv = ((T + Bt - 1) / Bt) * g.Nh * g.Nw;
    g.text_len = text_len;
    g.padded = (T % Bt) || (H % Bh) || (W % Bw) || (text_len % (Bt * Bh * Bw));
    return g;
}

// Number of workgroups of kernel `Kern` (block threads, static LDS) resident
// per XCD at once: occupancy per CU times CUs / 8.  Used as the period of the
// phased block-list sweep.  Cached per kernel (one instantiation each) and
// per device.
template <auto Kern>
int resident_per_xcd(int block) {
    static std::atomic<int> cache[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 1;
    std::atomic<int>& slot = cache[dev & 63];
    int v = slot.load(std::memory_order_relaxed);
    if (v > 0) return v;
    int per_cu = 0, cus = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void*>(Kern), block, 0) !=
            hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
        return 1;
    v = per_cu * cus / 8;
    if (v < 1) v = 1;
    slot.store(v, std::memory_order_relaxed);
    return v;
}

hipError_t launch_pool(int dtype, const void* x, void* out, int64_t nbh, int N, int64_t Lj, int D,
                       const cube_grid& cg, int Pt, int Ph, int Pw, hipStream_t s);
hipError_t launch_route_passes(int dtype, int D, int G, const void* qr, const void* kr, float* lse2,
                               float* scores, int batch, int Hq, int Hkv, int N, const cube_grid& cg, int Rt,
                               int Rh, int Rw, hipStream_t s);
hipError_t launch_select(int phase, const float* scores, int64_t nrows, int N, int mode, int k,
                         float mass, int cap, int32_t* counts, const int32_t* row_ptr,
                         int32_t* col_idx, int64_t col_cap, hipStream_t s);
hipError_t launch_scan(const int32_t* counts, int64_t n, int32_t* ptr, hipStream_t s);
// Sequence-level top-(N k) selection over nseq maps of N x N scores.
size_t seq_workspace_bytes(int64_t nseq, int64_t nrows);
hipError_t launch_select_seq(const float* scores, int64_t nseq, int N, int k, void* ws, int32_t* counts,
                             int32_t* row_ptr, int32_t* col_idx, int64_t col_cap, hipStream_t s);
hipError_t launch_uniform_ptr(int32_t* ptr, int64_t n, int k, hipStream_t s);
hipError_t launch_fill_u32(uint32_t* p, int64_t n, uint32_t v, hipStream_t s);
hipError_t launch_csc(const int32_t* row_ptr, const int32_t* col_idx, int batch, int Hq, int Hkv, int N,
                      int64_t col_cap, uint32_t* mask, int32_t* kv_counts, int32_t* kv_ptr,
                      int32_t* kv_idx, hipStream_t s);
hipError_t launch_mfma_peak(int iters, float* sink, int64_t* flops, hipStream_t s);
// fp32 atomic adds of one 64 x D tile per transposed-list entry (a fused
// backward's dQ accumulation, without its arithmetic).
hipError_t launch_dq_atomic_probe(const int32_t* kv_ptr, const int32_t* kv_idx, int64_t col_cap, float* acc,
                                  int batch, int Hq, int Hkv, int N, int D, hipStream_t s);
hipError_t launch_attn_fwd(int dtype, int D, const void* q, const void* k, const void* v,
                           const int32_t* row_ptr, const int32_t* col_idx, int64_t col_cap, void* o,
                           float* lse, void* o_lo, void* ws, int batch, int Hq, int Hkv, int N,
                           const cube_grid& cg, hipStream_t s);
// Forward workspace: the work order of the CSR rows (int32 per row), then the
// block magnitude flags.
size_t fwd_workspace_bytes(int batch, int Hq, int Hkv, int N);
// Backward workspace: (LSE*log2 e, Delta) per query token, then the work
// orders of the CSR rows (dQ) and of the CSC rows (dK/dV).
size_t bwd_workspace_bytes(int dtype, int D, int batch, int Hq, int Hkv, int N);
size_t bwd_ws_csr_order_offset(int batch, int Hq, int N);
size_t bwd_ws_csc_order_offset(int batch, int Hq, int N);
// Longest-first work order of the rows of ptr within each piece of a head
// (n_per_head rows) that falls into one XCD range.
hipError_t launch_lpt_order(const int32_t* ptr, int64_t nrows, int64_t n_per_head, int64_t cap, int32_t* order,
                            hipStream_t s);
// Magnitude flags of the 64-token blocks of bf16 Q, K, V: q[row] for the
// query blocks, kv[row] for the key blocks (K and V combined), 1 when a real
// token holds a value above 7 in magnitude; any_q[g] / any_kv[g] per KV group
// g = b*Hkv + hkv: some flagged query block among the group's query heads /
// some flagged key block of the head.  The attention kernels take two-term
// P / dS operands where these flags (and the row flags) say so.
struct block_flag_layout {
    uint8_t* q;
    uint8_t* kv;
    int32_t* any_q;
    int32_t* any_kv;
    // per query block: bit 0 its own flag; bit 1 two-term dS for its row
    // (its list touches a flagged block, its own flag included, or one of
    // its queries has |Delta| above DELTA_FLAG)
    uint8_t* qrow;
    int32_t* any_row;    // per KV group: some query block of the group has bit 1
};
// Rows whose Delta = dO . O exceeds this in magnitude at some query take
// two-term dS: dS = P (dP - Delta) is then a small difference of large
// terms whose one-term rounding the gradients amplify.
constexpr float DELTA_FLAG = 16.0f;
block_flag_layout block_flags_at(void* base, int64_t rows_q, int64_t rows_kv, int64_t groups);
size_t block_flags_bytes(int64_t rows_q, int64_t rows_kv, int64_t groups);
hipError_t launch_block_flags(const void* q, const void* k, const void* v, const block_flag_layout& f, int64_t rows_q,
                              int64_t rows_kv, int N, int D, int Hq, int Hkv, const cube_grid& cg, hipStream_t s);
hipError_t launch_row_flags(const block_flag_layout& f, const float* stat, const int32_t* kv_ptr,
                            const int32_t* kv_idx, int64_t col_cap, int64_t rows_q, int64_t rows_kv, int N, int Hq,
                            int Hkv, hipStream_t s);
hipError_t launch_attn_bwd(int dtype, int D, const void* q, const void* k, const void* v, const void* o,
                           const float* lse, const void* o_lo, const void* dout, const int32_t* row_ptr,
                           const int32_t* col_idx, const int32_t* kv_ptr, const int32_t* kv_idx,
                           int64_t col_cap, void* dq, void* dk, void* dv, void* ws, int batch,
                           int Hq, int Hkv, int N, const cube_grid& cg, hipStream_t s);
hipError_t launch_attn_bwd_prep(int dtype, int D, const void* q, const void* k, const void* v, const void* o,
                                const float* lse, const void* o_lo, const void* dout, void* ws, int batch, int Hq,
                                int Hkv, int N, const cube_grid& cg, hipStream_t s);
// (LSE * log2 e, dO . O) for ntok rows of D elements.
hipError_t launch_attn_bwd_prep_tokens(int dtype, int D, const void* o, const float* lse, const void* o_lo,
                                       const void* dout, void* ws, int64_t ntok, hipStream_t s);
// Coarse branch and gated merge.
hipError_t launch_coarse_fwd(int dtype, int D, const void* qc, const void* kc, const void* vc, void* oc,
                             float* lse, int batch, int Hq, int Hkv, int N, hipStream_t s);
hipError_t launch_coarse_bwd(int dtype, int D, const void* qc, const void* kc, const void* vc, const void* doc,
                             void* dqc, void* dkc, void* dvc, void* ws, int batch, int Hq, int Hkv, int N,
                             hipStream_t s);
hipError_t launch_gate_merge(int dtype, int D, const float* gate, const void* oc, const void* of, void* out,
                             int64_t ntok, int64_t L, int64_t Lj, int N, hipStream_t s);
hipError_t launch_gate_merge_bwd(int dtype, int D, const float* gate, const void* oc, const void* dout, void* doc,
                                 float* dgate, int64_t ncubes, int N, int M, const cube_grid& cg, hipStream_t s);
hipError_t launch_unpool_add(int dtype, int D, const void* dxc, void* dx, int64_t ntok, int64_t L, int64_t Lj,
                             int N, const cube_grid& cg, int Pt, int Ph, int Pw, hipStream_t s);
// Joint video + text lists from the router's video lists (rows of N video
// cubes; M text blocks per sequence).  ws: int32 counts per joint row, then
// the CSC workspace.
size_t joint_workspace_bytes(int batch, int Hq, int Hkv, int N, int M);
hipError_t launch_joint_lists(const int32_t* row_ptr, const int32_t* col_idx, int64_t col_cap, int batch, int Hq,
                              int Hkv, int N, int M, int32_t* j_row_ptr, int32_t* j_col_idx, int64_t j_cap,
                              int32_t* j_kv_ptr, int32_t* j_kv_idx, void* ws, hipStream_t s);
hipError_t launch_attn_bwd_dkdv(int dtype, int D, const void* q, const void* k, const void* v,
                                const void* dout, const int32_t* kv_ptr, const int32_t* kv_idx, int64_t col_cap,
                                void* dk, void* dv, void* ws, int batch, int Hq, int Hkv, int N,
                                const cube_grid& cg, hipStream_t s);
hipError_t launch_attn_bwd_dq(int dtype, int D, const void* q, const void* k, const void* v,
                              const void* dout, const int32_t* row_ptr, const int32_t* col_idx, int64_t col_cap,
                              void* dq, void* ws, int batch, int Hq, int Hkv, int N, const cube_grid& cg,
                              hipStream_t s);

}  // namespace vsa2
