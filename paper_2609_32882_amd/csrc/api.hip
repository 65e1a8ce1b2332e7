// The public C-ABI (vsa2.h): argument validation, workspace layout and the
// launch sequence of each call.  Every check runs on the host before any
// device work is enqueued; no call allocates, synchronises or reads device
// memory.
#include "vsa2.h"

#include <math.h>

#include <mutex>

#include "internal.hpp"

namespace {

constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// N, L, rows_*: video cubes / tokens / query- and key-block rows; the
// joint sequence (video, then M text blocks) has Nj = N + M blocks of B
// tokens, Lj tokens, rows_qj / rows_kvj block rows (= the video ones
// without text).
struct shape {
    int64_t N, L, B, G, rows_q, rows_kv;
    int64_t M, Nj, Lj, rows_qj, rows_kvj;
};

// Structural checks shared by all calls.
vsa2_status check_problem(const vsa2_problem* p, shape* out) {
    if (!p) return VSA2_ERR_NULL;
    if (p->dtype != VSA2_F32 && p->dtype != VSA2_BF16) return VSA2_ERR_DTYPE;
    if (p->batch < 1 || p->heads_q < 1 || p->heads_kv < 1 || p->head_dim < 1) return VSA2_ERR_SHAPE;
    if (p->heads_q % p->heads_kv) return VSA2_ERR_SHAPE;
    if (p->T < 1 || p->H < 1 || p->W < 1 || p->Bt < 1 || p->Bh < 1 || p->Bw < 1) return VSA2_ERR_SHAPE;
    if (p->Rt < 1 || p->Rh < 1 || p->Rw < 1) return VSA2_ERR_SHAPE;
    if (p->text_len < 0) return VSA2_ERR_SHAPE;
    if (p->Bt % p->Rt || p->Bh % p->Rh || p->Bw % p->Rw) return VSA2_ERR_SHAPE;
    shape s;
    s.B = static_cast<int64_t>(p->Bt) * p->Bh * p->Bw;
    // a grid axis that is not a multiple of its cube size is padded up to one
    s.N = static_cast<int64_t>((p->T + p->Bt - 1) / p->Bt) * ((p->H + p->Bh - 1) / p->Bh) *
          ((p->W + p->Bw - 1) / p->Bw);
    s.L = s.N * s.B;
    s.G = static_cast<int64_t>(p->Bt / p->Rt) * (p->Bh / p->Rh) * (p->Bw / p->Rw);
    s.rows_q = static_cast<int64_t>(p->batch) * p->heads_q * s.N;
    s.rows_kv = static_cast<int64_t>(p->batch) * p->heads_kv * s.N;
    s.M = (p->text_len + s.B - 1) / s.B;
    s.Nj = s.N + s.M;
    s.Lj = s.Nj * s.B;
    s.rows_qj = static_cast<int64_t>(p->batch) * p->heads_q * s.Nj;
    s.rows_kvj = static_cast<int64_t>(p->batch) * p->heads_kv * s.Nj;
    if (s.Nj > (1 << 26) || s.rows_qj > (int64_t(1) << 31) - 2) return VSA2_ERR_SHAPE;
    *out = s;
    return VSA2_OK;
}

vsa2::cube_grid grid_of(const vsa2_problem* p) {
    return vsa2::make_cube_grid(p->T, p->H, p->W, p->Bt, p->Bh, p->Bw, p->text_len);
}

// Shapes the attention and router kernels are built for.
vsa2_status check_kernel_shape(const vsa2_problem* p, const shape& s) {
    if (s.B != 64) return VSA2_ERR_UNSUPPORTED;
    if (p->head_dim != 64 && p->head_dim != 128) return VSA2_ERR_UNSUPPORTED;
    return VSA2_OK;
}

vsa2_status check_select(const vsa2_select* sel) {
    if (!sel) return VSA2_ERR_NULL;
    if (sel->mode == VSA2_SEL_TOPK || sel->mode == VSA2_SEL_SEQ_TOPK) return sel->k >= 1 ? VSA2_OK : VSA2_ERR_SELECT;
    if (sel->mode == VSA2_SEL_MASS) {
        if (!(sel->mass > 0.f && sel->mass <= 1.f)) return VSA2_ERR_SELECT;
        return sel->cap >= 1 ? VSA2_OK : VSA2_ERR_SELECT;
    }
    return VSA2_ERR_SELECT;
}

int64_t keep_per_row(const vsa2_select* sel, int64_t N) {
    // SEQ_TOPK keeps N*min(k, N) pairs per sequence: the same total as TOPK,
    // spread unevenly over the rows (a row holds at most N)
    const int64_t k = sel->mode == VSA2_SEL_MASS ? sel->cap : sel->k;
    return k < N ? k : N;
}

struct route_ws {
    size_t lse2, scores, counts, mask, kv_counts, seq, total;
};

route_ws route_layout(const vsa2_problem* p, const shape& s, const vsa2_select* sel) {
    route_ws w;
    size_t at = 0;
    const int64_t words = (static_cast<int64_t>(p->heads_q / p->heads_kv) * s.N + 31) / 32;
    w.lse2 = at;      at = align_up(at + sizeof(float) * static_cast<size_t>(s.rows_q * s.G));
    w.scores = at;    at = align_up(at + sizeof(float) * static_cast<size_t>(s.rows_q * s.N));
    w.counts = at;    at = align_up(at + sizeof(int32_t) * static_cast<size_t>(s.rows_q));
    w.mask = at;      at = align_up(at + sizeof(uint32_t) * static_cast<size_t>(s.rows_kv * words));
    w.kv_counts = at; at = align_up(at + sizeof(int32_t) * static_cast<size_t>(s.rows_kv));
    w.seq = at;
    if (sel->mode == VSA2_SEL_SEQ_TOPK)
        at = align_up(at + vsa2::seq_workspace_bytes(static_cast<int64_t>(p->batch) * p->heads_q, s.rows_q));
    w.total = at;
    return w;
}

// the forward's workspace holds its work order (one int32 per query-block row)
// and the block magnitude flags
size_t fwd_ws_bytes(const shape& s, const vsa2_problem* p) {
    return vsa2::fwd_workspace_bytes(p->batch, p->heads_q, p->heads_kv, static_cast<int>(s.Nj));
}

size_t bwd_ws_bytes(const shape& s, const vsa2_problem* p) {
    return vsa2::bwd_workspace_bytes(p->dtype, p->head_dim, p->batch, p->heads_q, p->heads_kv,
                                     static_cast<int>(s.Nj));
}

#define VSA2_TRY_HIP(expr)                          \
    do {                                            \
        if ((expr) != hipSuccess) return VSA2_ERR_HIP; \
    } while (0)

// entries of the joint lists beyond the video ones: the text blocks of the
// video rows and the full text rows
int64_t joint_extra(const vsa2_problem* p, const shape& s) {
    return static_cast<int64_t>(p->batch) * p->heads_q * (s.N * s.M + s.M * s.Nj);
}

}  // namespace

extern "C" {

const char* vsa2_status_str(vsa2_status s) {
    switch (s) {
        case VSA2_OK: return "ok";
        case VSA2_ERR_NULL: return "null pointer";
        case VSA2_ERR_SHAPE: return "invalid or inconsistent shape";
        case VSA2_ERR_DTYPE: return "unsupported dtype";
        case VSA2_ERR_SELECT: return "invalid selection rule";
        case VSA2_ERR_CAPACITY: return "column capacity too small";
        case VSA2_ERR_ALIGN: return "pointer not 16-byte aligned";
        case VSA2_ERR_WORKSPACE: return "workspace missing or too small";
        case VSA2_ERR_HIP: return "HIP launch failed";
        case VSA2_ERR_UNSUPPORTED: return "shape outside the supported kernel configurations";
    }
    return "unknown status";
}

vsa2_status vsa2_pool(const vsa2_problem* p, int32_t heads, const void* x, int32_t Pt, int32_t Ph,
                      int32_t Pw, void* out, hipStream_t stream) {
    shape s;
    vsa2_status st = check_problem(p, &s);
    if (st != VSA2_OK) return st;
    if (!x || !out) return VSA2_ERR_NULL;
    if (heads < 1 || Pt < 1 || Ph < 1 || Pw < 1) return VSA2_ERR_SHAPE;
    if (p->Bt % Pt || p->Bh % Ph || p->Bw % Pw) return VSA2_ERR_SHAPE;
    if (p->head_dim % 8) return VSA2_ERR_UNSUPPORTED;
    if (!aligned16(x) || !aligned16(out)) return VSA2_ERR_ALIGN;
    VSA2_TRY_HIP(vsa2::launch_pool(p->dtype, x, out, static_cast<int64_t>(p->batch) * heads,
                                   static_cast<int>(s.N), s.Lj, p->head_dim, grid_of(p), Pt, Ph, Pw, stream));
    return VSA2_OK;
}

vsa2_status vsa2_route_capacity(const vsa2_problem* p, const vsa2_select* sel, int64_t* pairs) {
    shape s;
    vsa2_status st = check_problem(p, &s);
    if (st != VSA2_OK) return st;
    if ((st = check_select(sel)) != VSA2_OK) return st;
    if (!pairs) return VSA2_ERR_NULL;
    *pairs = s.rows_q * keep_per_row(sel, s.N);
    return VSA2_OK;
}

vsa2_status vsa2_route_workspace(const vsa2_problem* p, const vsa2_select* sel, size_t* bytes) {
    shape s;
    vsa2_status st = check_problem(p, &s);
    if (st != VSA2_OK) return st;
    if ((st = check_select(sel)) != VSA2_OK) return st;
    if (!bytes) return VSA2_ERR_NULL;
    *bytes = route_layout(p, s, sel).total;
    return VSA2_OK;
}

vsa2_status vsa2_route(const vsa2_problem* p, const vsa2_select* sel, const void* q_r, const void* k_r,
                       int32_t* row_ptr, int32_t* col_idx, int64_t col_cap, int32_t* kv_ptr,
                       int32_t* kv_idx, float* block_scores, void* ws, size_t ws_bytes,
                       hipStream_t stream) {
    shape s;
    vsa2_status st = check_problem(p, &s);
    if (st != VSA2_OK) return st;
    if ((st = check_select(sel)) != VSA2_OK) return st;
    if ((st = check_kernel_shape(p, s)) != VSA2_OK) return st;
    if (s.G != 1 && s.G != 2 && s.G != 4 && s.G != 8) return VSA2_ERR_UNSUPPORTED;
    if (s.N > 4096) return VSA2_ERR_UNSUPPORTED;
    if (!q_r || !k_r || !row_ptr || !col_idx) return VSA2_ERR_NULL;
    if ((kv_ptr == nullptr) != (kv_idx == nullptr)) return VSA2_ERR_NULL;
    if (!aligned16(q_r) || !aligned16(k_r)) return VSA2_ERR_ALIGN;
    const int64_t keep = keep_per_row(sel, s.N);
    if (col_cap < s.rows_q * keep) return VSA2_ERR_CAPACITY;
    const route_ws w = route_layout(p, s, sel);
    if (!ws || ws_bytes < w.total) return VSA2_ERR_WORKSPACE;
    if (reinterpret_cast<uintptr_t>(ws) % kAlign) return VSA2_ERR_ALIGN;
    char* base = static_cast<char*>(ws);
    float* lse2 = reinterpret_cast<float*>(base + w.lse2);
    float* scores = block_scores ? block_scores : reinterpret_cast<float*>(base + w.scores);
    int32_t* counts = reinterpret_cast<int32_t*>(base + w.counts);
    const int N = static_cast<int>(s.N);

    VSA2_TRY_HIP(vsa2::launch_route_passes(p->dtype, p->head_dim, static_cast<int>(s.G), q_r, k_r, lse2,
                                           scores, p->batch, p->heads_q, p->heads_kv, N, grid_of(p), p->Rt,
                                           p->Rh, p->Rw, stream));
    if (sel->mode == VSA2_SEL_SEQ_TOPK) {
        VSA2_TRY_HIP(vsa2::launch_select_seq(scores, static_cast<int64_t>(p->batch) * p->heads_q, N, sel->k,
                                             base + w.seq, counts, row_ptr, col_idx, col_cap, stream));
    } else {
        if (sel->mode == VSA2_SEL_TOPK) {
            VSA2_TRY_HIP(vsa2::launch_uniform_ptr(row_ptr, s.rows_q, static_cast<int>(keep), stream));
        } else {
            VSA2_TRY_HIP(vsa2::launch_select(0, scores, s.rows_q, N, sel->mode, sel->k, sel->mass, sel->cap,
                                             counts, nullptr, nullptr, col_cap, stream));
            VSA2_TRY_HIP(vsa2::launch_scan(counts, s.rows_q, row_ptr, stream));
        }
        VSA2_TRY_HIP(vsa2::launch_select(1, scores, s.rows_q, N, sel->mode, sel->k, sel->mass, sel->cap,
                                         counts, row_ptr, col_idx, col_cap, stream));
    }
    if (kv_ptr) {
        VSA2_TRY_HIP(vsa2::launch_csc(row_ptr, col_idx, p->batch, p->heads_q, p->heads_kv, N, col_cap,
                                      reinterpret_cast<uint32_t*>(base + w.mask),
                                      reinterpret_cast<int32_t*>(base + w.kv_counts), kv_ptr, kv_idx,
                                      stream));
    }
    return VSA2_OK;
}

vsa2_status vsa2_attn_workspace(const vsa2_problem* p, int32_t pass, size_t* bytes) {
    shape s;
    vsa2_status st = check_problem(p, &s);
    if (st != VSA2_OK) return st;
    if (!bytes) return VSA2_ERR_NULL;
    if (pass == 0) *bytes = fwd_ws_bytes(s, p);
    else if (pass == 1) *bytes = bwd_ws_bytes(s, p);
    else if (pass == 2) *bytes = align_up(8 * static_cast<size_t>(s.rows_q));   // coarse backward
    else return VSA2_ERR_SHAPE;
    return VSA2_OK;
}

vsa2_status vsa2_attn_fwd(const vsa2_problem* p, const void* q, const void* k, const void* v,
                          const int32_t* row_ptr, const int32_t* col_idx, int64_t col_cap, void* o,
                          float* lse, void* o_lo, void* ws, size_t ws_bytes, hipStream_t stream) {
    shape s;
    vsa2_status st = check_problem(p, &s);
    if (st != VSA2_OK) return st;
    if ((st = check_kernel_shape(p, s)) != VSA2_OK) return st;
    if (!q || !k || !v || !row_ptr || !o || !lse) return VSA2_ERR_NULL;
    if (!col_idx && col_cap > 0) return VSA2_ERR_NULL;
    if (col_cap < 0) return VSA2_ERR_CAPACITY;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o) || !aligned16(o_lo))
        return VSA2_ERR_ALIGN;
    if (!ws || ws_bytes < fwd_ws_bytes(s, p)) return VSA2_ERR_WORKSPACE;
    if (reinterpret_cast<uintptr_t>(ws) % kAlign) return VSA2_ERR_ALIGN;
    VSA2_TRY_HIP(vsa2::launch_attn_fwd(p->dtype, p->head_dim, q, k, v, row_ptr, col_idx, col_cap, o, lse,
                                       o_lo, ws, p->batch, p->heads_q, p->heads_kv, static_cast<int>(s.Nj),
                                       grid_of(p), stream));
    return VSA2_OK;
}

// ---------------------------------------------------------------------------
// vsa2_attn_fwd_noalloc: the forward with its workspace in a fixed device
// array of the library.  Each GPU holds its own copy of `scratch` until the
// process ends; its address on a device comes from hipGetSymbolAddress,
// taken once per device with that device current and kept here (in host
// code the array's name is not a device address, so it is never passed to
// a kernel or a copy).
// ---------------------------------------------------------------------------
namespace {

__device__ __align__(256) unsigned char scratch[VSA2_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The scratch array of the current device (set up on the first call there).
vsa2_status scratch_of_current_device(void** out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return VSA2_ERR_HIP;
    if (dev < 0 || dev >= kMaxDevices) return VSA2_ERR_UNSUPPORTED;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return VSA2_ERR_HIP;
        g_scratch_ptr[dev] = ptr;
    }
    *out = g_scratch_ptr[dev];
    return VSA2_OK;
}

}  // namespace

vsa2_status vsa2_attn_fwd_noalloc(const vsa2_problem* p, const void* q, const void* k, const void* v,
                                  const int32_t* row_ptr, const int32_t* col_idx, int64_t col_cap, void* o,
                                  float* lse, void* o_lo, hipStream_t stream) {
    shape s;
    vsa2_status st = check_problem(p, &s);
    if (st != VSA2_OK) return st;
    if ((st = check_kernel_shape(p, s)) != VSA2_OK) return st;
    if (!q || !k || !v || !row_ptr || !o || !lse) return VSA2_ERR_NULL;
    if (!col_idx && col_cap > 0) return VSA2_ERR_NULL;
    if (col_cap < 0) return VSA2_ERR_CAPACITY;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o) || !aligned16(o_lo))
        return VSA2_ERR_ALIGN;
    if (fwd_ws_bytes(s, p) > VSA2_NOALLOC_SCRATCH_BYTES) return VSA2_ERR_WORKSPACE;
    void* ws = nullptr;
    if ((st = scratch_of_current_device(&ws)) != VSA2_OK) return st;
    // every part of the workspace the forward reads is written earlier in the
    // same call (work order, block flags; their summary words are cleared by
    // a fill kernel), so the previous call's contents do not matter
    VSA2_TRY_HIP(vsa2::launch_attn_fwd(p->dtype, p->head_dim, q, k, v, row_ptr, col_idx, col_cap, o, lse,
                                       o_lo, ws, p->batch, p->heads_q, p->heads_kv, static_cast<int>(s.Nj),
                                       grid_of(p), stream));
    return VSA2_OK;
}

vsa2_status vsa2_attn_bwd(const vsa2_problem* p, const void* q, const void* k, const void* v, const void* o,
                          const float* lse, const void* o_lo, const void* dout, const int32_t* row_ptr,
                          const int32_t* col_idx, const int32_t* kv_ptr, const int32_t* kv_idx,
                          int64_t col_cap, void* dq, void* dk, void* dv, void* ws, size_t ws_bytes,
                          hipStream_t stream) {
    shape s;
    vsa2_status st = check_problem(p, &s);
    if (st != VSA2_OK) return st;
    if ((st = check_kernel_shape(p, s)) != VSA2_OK) return st;
    if (!q || !k || !v || !o || !lse || !o_lo || !dout || !row_ptr || !kv_ptr || !dq || !dk || !dv)
        return VSA2_ERR_NULL;
    if ((!col_idx || !kv_idx) && col_cap > 0) return VSA2_ERR_NULL;
    if (col_cap < 0) return VSA2_ERR_CAPACITY;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o) || !aligned16(dout) ||
        !aligned16(dq) || !aligned16(dk) || !aligned16(dv) || !aligned16(o_lo))
        return VSA2_ERR_ALIGN;
    const size_t need = bwd_ws_bytes(s, p);
    if (!ws || ws_bytes < need) return VSA2_ERR_WORKSPACE;
    if (reinterpret_cast<uintptr_t>(ws) % kAlign) return VSA2_ERR_ALIGN;
    VSA2_TRY_HIP(vsa2::launch_attn_bwd(p->dtype, p->head_dim, q, k, v, o, lse, o_lo, dout, row_ptr, col_idx,
                                       kv_ptr, kv_idx, col_cap, dq, dk, dv, ws,
                                       p->batch, p->heads_q, p->heads_kv, static_cast<int>(s.Nj), grid_of(p),
                                       stream));
    return VSA2_OK;
}

vsa2_status vsa2_attn_bwd_prep(const vsa2_problem* p, const void* q, const void* k, const void* v, const void* o,
                               const float* lse, const void* o_lo, const void* dout, void* ws, size_t ws_bytes,
                               hipStream_t stream) {
    shape s;
    vsa2_status st = check_problem(p, &s);
    if (st != VSA2_OK) return st;
    if ((st = check_kernel_shape(p, s)) != VSA2_OK) return st;
    if (!q || !k || !v || !o || !lse || !o_lo || !dout) return VSA2_ERR_NULL;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o) || !aligned16(dout) || !aligned16(o_lo))
        return VSA2_ERR_ALIGN;
    const size_t need = bwd_ws_bytes(s, p);
    if (!ws || ws_bytes < need) return VSA2_ERR_WORKSPACE;
    if (reinterpret_cast<uintptr_t>(ws) % kAlign) return VSA2_ERR_ALIGN;
    VSA2_TRY_HIP(vsa2::launch_attn_bwd_prep(p->dtype, p->head_dim, q, k, v, o, lse, o_lo, dout, ws, p->batch,
                                            p->heads_q, p->heads_kv, static_cast<int>(s.Nj), grid_of(p), stream));
    return VSA2_OK;
}

vsa2_status vsa2_attn_bwd_dkdv(const vsa2_problem* p, const void* q, const void* k, const void* v,
                               const void* dout, const int32_t* kv_ptr, const int32_t* kv_idx, int64_t col_cap,
                               void* dk, void* dv, void* ws, size_t ws_bytes, hipStream_t stream) {
    shape s;
    vsa2_status st = check_problem(p, &s);
    if (st != VSA2_OK) return st;
    if ((st = check_kernel_shape(p, s)) != VSA2_OK) return st;
    if (!q || !k || !v || !dout || !kv_ptr || !dk || !dv) return VSA2_ERR_NULL;
    if (!kv_idx && col_cap > 0) return VSA2_ERR_NULL;
    if (col_cap < 0) return VSA2_ERR_CAPACITY;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(dout) || !aligned16(dk) || !aligned16(dv))
        return VSA2_ERR_ALIGN;
    const size_t need = bwd_ws_bytes(s, p);
    if (!ws || ws_bytes < need) return VSA2_ERR_WORKSPACE;
    if (reinterpret_cast<uintptr_t>(ws) % kAlign) return VSA2_ERR_ALIGN;
    VSA2_TRY_HIP(vsa2::launch_attn_bwd_dkdv(p->dtype, p->head_dim, q, k, v, dout, kv_ptr, kv_idx, col_cap, dk, dv,
                                            ws, p->batch, p->heads_q, p->heads_kv, static_cast<int>(s.Nj),
                                            grid_of(p), stream));
    return VSA2_OK;
}

vsa2_status vsa2_attn_bwd_dq(const vsa2_problem* p, const void* q, const void* k, const void* v,
                             const void* dout, const int32_t* row_ptr, const int32_t* col_idx, int64_t col_cap,
                             void* dq, void* ws, size_t ws_bytes, hipStream_t stream) {
    shape s;
    vsa2_status st = check_problem(p, &s);
    if (st != VSA2_OK) return st;
    if ((st = check_kernel_shape(p, s)) != VSA2_OK) return st;
    if (!q || !k || !v || !dout || !row_ptr || !dq) return VSA2_ERR_NULL;
    if (!col_idx && col_cap > 0) return VSA2_ERR_NULL;
    if (col_cap < 0) return VSA2_ERR_CAPACITY;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(dout) || !aligned16(dq))
        return VSA2_ERR_ALIGN;
    const size_t need = bwd_ws_bytes(s, p);
    if (!ws || ws_bytes < need) return VSA2_ERR_WORKSPACE;
    if (reinterpret_cast<uintptr_t>(ws) % kAlign) return VSA2_ERR_ALIGN;
    VSA2_TRY_HIP(vsa2::launch_attn_bwd_dq(p->dtype, p->head_dim, q, k, v, dout, row_ptr, col_idx, col_cap, dq, ws,
                                          p->batch, p->heads_q, p->heads_kv, static_cast<int>(s.Nj), grid_of(p),
                                          stream));
    return VSA2_OK;
}

vsa2_status vsa2_coarse_fwd(const vsa2_problem* p, const void* q_c, const void* k_c, const void* v_c, void* o_c,
                            float* lse_c, hipStream_t stream) {
    shape s;
    vsa2_status st = check_problem(p, &s);
    if (st != VSA2_OK) return st;
    if ((st = check_kernel_shape(p, s)) != VSA2_OK) return st;
    if (!q_c || !k_c || !v_c || !o_c || !lse_c) return VSA2_ERR_NULL;
    if (!aligned16(q_c) || !aligned16(k_c) || !aligned16(v_c) || !aligned16(o_c)) return VSA2_ERR_ALIGN;
    if (p->batch * static_cast<int64_t>(p->heads_q) > 65535) return VSA2_ERR_UNSUPPORTED;
    VSA2_TRY_HIP(vsa2::launch_coarse_fwd(p->dtype, p->head_dim, q_c, k_c, v_c, o_c, lse_c, p->batch, p->heads_q,
                                         p->heads_kv, static_cast<int>(s.N), stream));
    return VSA2_OK;
}

vsa2_status vsa2_coarse_bwd(const vsa2_problem* p, const void* q_c, const void* k_c, const void* v_c,
                            const void* do_c, void* dq_c, void* dk_c, void* dv_c, void* ws, size_t ws_bytes,
                            hipStream_t stream) {
    shape s;
    vsa2_status st = check_problem(p, &s);
    if (st != VSA2_OK) return st;
    if ((st = check_kernel_shape(p, s)) != VSA2_OK) return st;
    if (!q_c || !k_c || !v_c || !do_c || !dq_c || !dk_c || !dv_c) return VSA2_ERR_NULL;
    if (!aligned16(q_c) || !aligned16(k_c) || !aligned16(v_c) || !aligned16(do_c) ||
        !aligned16(dq_c) || !aligned16(dk_c) || !aligned16(dv_c))
        return VSA2_ERR_ALIGN;
    if (!ws || ws_bytes < align_up(8 * static_cast<size_t>(s.rows_q))) return VSA2_ERR_WORKSPACE;
    if (reinterpret_cast<uintptr_t>(ws) % kAlign) return VSA2_ERR_ALIGN;
    if (p->batch * static_cast<int64_t>(p->heads_q) > 65535) return VSA2_ERR_UNSUPPORTED;
    VSA2_TRY_HIP(vsa2::launch_coarse_bwd(p->dtype, p->head_dim, q_c, k_c, v_c, do_c, dq_c, dk_c, dv_c, ws,
                                         p->batch, p->heads_q, p->heads_kv, static_cast<int>(s.N), stream));
    return VSA2_OK;
}

vsa2_status vsa2_gate_merge(const vsa2_problem* p, const float* gate, const void* o_c, const void* o_f, void* out,
                            hipStream_t stream) {
    shape s;
    vsa2_status st = check_problem(p, &s);
    if (st != VSA2_OK) return st;
    if ((st = check_kernel_shape(p, s)) != VSA2_OK) return st;
    if (!gate || !o_c || !o_f || !out) return VSA2_ERR_NULL;
    if (!aligned16(o_c) || !aligned16(o_f) || !aligned16(out)) return VSA2_ERR_ALIGN;
    VSA2_TRY_HIP(vsa2::launch_gate_merge(p->dtype, p->head_dim, gate, o_c, o_f, out,
                                         static_cast<int64_t>(p->batch) * p->heads_q * s.Lj, s.L, s.Lj,
                                         static_cast<int>(s.N), stream));
    return VSA2_OK;
}

vsa2_status vsa2_gate_merge_bwd(const vsa2_problem* p, const float* gate, const void* o_c, const void* dout,
                                void* do_c, float* dgate, hipStream_t stream) {
    shape s;
    vsa2_status st = check_problem(p, &s);
    if (st != VSA2_OK) return st;
    if ((st = check_kernel_shape(p, s)) != VSA2_OK) return st;
    if (!gate || !o_c || !dout || !do_c || !dgate) return VSA2_ERR_NULL;
    if (!aligned16(o_c) || !aligned16(dout) || !aligned16(do_c)) return VSA2_ERR_ALIGN;
    VSA2_TRY_HIP(vsa2::launch_gate_merge_bwd(p->dtype, p->head_dim, gate, o_c, dout, do_c, dgate, s.rows_q,
                                             static_cast<int>(s.N), static_cast<int>(s.M), grid_of(p), stream));
    return VSA2_OK;
}

vsa2_status vsa2_joint_capacity(const vsa2_problem* p, const vsa2_select* sel, int64_t* pairs) {
    shape s;
    vsa2_status st = check_problem(p, &s);
    if (st != VSA2_OK) return st;
    if ((st = check_select(sel)) != VSA2_OK) return st;
    if (!pairs) return VSA2_ERR_NULL;
    *pairs = s.rows_q * keep_per_row(sel, s.N) + joint_extra(p, s);
    return VSA2_OK;
}

vsa2_status vsa2_joint_workspace(const vsa2_problem* p, size_t* bytes) {
    shape s;
    vsa2_status st = check_problem(p, &s);
    if (st != VSA2_OK) return st;
    if (!bytes) return VSA2_ERR_NULL;
    *bytes = vsa2::joint_workspace_bytes(p->batch, p->heads_q, p->heads_kv, static_cast<int>(s.N),
                                         static_cast<int>(s.M));
    return VSA2_OK;
}

vsa2_status vsa2_joint_lists(const vsa2_problem* p, const int32_t* row_ptr, const int32_t* col_idx,
                             int64_t col_cap, int32_t* j_row_ptr, int32_t* j_col_idx, int64_t j_cap,
                             int32_t* j_kv_ptr, int32_t* j_kv_idx, void* ws, size_t ws_bytes,
                             hipStream_t stream) {
    shape s;
    vsa2_status st = check_problem(p, &s);
    if (st != VSA2_OK) return st;
    if (p->text_len < 1) return VSA2_ERR_SHAPE;
    if (!row_ptr || !j_row_ptr || !j_col_idx || !j_kv_ptr || !j_kv_idx) return VSA2_ERR_NULL;
    if (!col_idx && col_cap > 0) return VSA2_ERR_NULL;
    if (col_cap < 0) return VSA2_ERR_CAPACITY;
    const int64_t need = col_cap + joint_extra(p, s);
    if (j_cap < need || need > (int64_t(1) << 31) - 1) return VSA2_ERR_CAPACITY;
    const size_t wsb = vsa2::joint_workspace_bytes(p->batch, p->heads_q, p->heads_kv, static_cast<int>(s.N),
                                                   static_cast<int>(s.M));
    if (!ws || ws_bytes < wsb) return VSA2_ERR_WORKSPACE;
    if (reinterpret_cast<uintptr_t>(ws) % kAlign) return VSA2_ERR_ALIGN;
    VSA2_TRY_HIP(vsa2::launch_joint_lists(row_ptr, col_idx, col_cap, p->batch, p->heads_q, p->heads_kv,
                                          static_cast<int>(s.N), static_cast<int>(s.M), j_row_ptr, j_col_idx, j_cap,
                                          j_kv_ptr, j_kv_idx, ws, stream));
    return VSA2_OK;
}

vsa2_status vsa2_unpool_add(const vsa2_problem* p, int32_t heads, const void* dx_c, int32_t Pt, int32_t Ph,
                            int32_t Pw, void* dx, hipStream_t stream) {
    shape s;
    vsa2_status st = check_problem(p, &s);
    if (st != VSA2_OK) return st;
    if (!dx_c || !dx) return VSA2_ERR_NULL;
    if (heads < 1 || Pt < 1 || Ph < 1 || Pw < 1) return VSA2_ERR_SHAPE;
    if (p->Bt % Pt || p->Bh % Ph || p->Bw % Pw) return VSA2_ERR_SHAPE;
    if (p->head_dim != 64 && p->head_dim != 128) return VSA2_ERR_UNSUPPORTED;
    if (!aligned16(dx_c) || !aligned16(dx)) return VSA2_ERR_ALIGN;
    VSA2_TRY_HIP(vsa2::launch_unpool_add(p->dtype, p->head_dim, dx_c, dx,
                                         static_cast<int64_t>(p->batch) * heads * s.L, s.L, s.Lj,
                                         static_cast<int>(s.N), grid_of(p), Pt, Ph, Pw, stream));
    return VSA2_OK;
}

vsa2_status vsa2_mfma_peak_probe(int32_t iters, float* sink, int64_t* flops, hipStream_t stream) {
    if (!flops || (iters > 0 && !sink)) return VSA2_ERR_NULL;
    if (iters < 0) return VSA2_ERR_SHAPE;
    VSA2_TRY_HIP(vsa2::launch_mfma_peak(iters, sink, flops, stream));
    return VSA2_OK;
}

vsa2_status vsa2_dq_atomic_probe(const vsa2_problem* p, const int32_t* kv_ptr, const int32_t* kv_idx,
                                 int64_t col_cap, float* acc, hipStream_t stream) {
    shape s;
    vsa2_status st = check_problem(p, &s);
    if (st != VSA2_OK) return st;
    if ((st = check_kernel_shape(p, s)) != VSA2_OK) return st;
    if (!kv_ptr || !acc) return VSA2_ERR_NULL;
    if (!kv_idx && col_cap > 0) return VSA2_ERR_NULL;
    if (col_cap < 0) return VSA2_ERR_CAPACITY;
    if (!aligned16(acc)) return VSA2_ERR_ALIGN;
    VSA2_TRY_HIP(vsa2::launch_dq_atomic_probe(kv_ptr, kv_idx, col_cap, acc, p->batch, p->heads_q, p->heads_kv,
                                              static_cast<int>(s.Nj), p->head_dim, stream));
    return VSA2_OK;
}

}  // extern "C"
