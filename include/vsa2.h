/*
 * vsa2.h - C-ABI of the MI355X (gfx950) routed sparse-attention library.
 *
 * Implements the data-parallel hot path of VSA2 ("Improving Video Sparse
 * Attention with Fine-grained Router and Sparse Rebasing"):
 *
 *   vsa2_pool      MeanPool over spatio-temporal sub-cubes
 *                  (Sec. 2.2, Eq. router_start for the router's R-pooling;
 *                   Eq. compress for the B-pooling of the coarse branch)
 *   vsa2_route     the fine-grained router: pooled-query x pooled-key
 *                  softmax, GxG score pooling, per-query-block selection,
 *                  CSR block lists and their transpose
 *                  (Sec. 2.2, Eq. router_start .. Eq. router_end)
 *   vsa2_attn_fwd  block-sparse attention over the selected block pairs
 *                  (Sec. 2.1 masked attention; Sec. 2.2 Eq. block_sparse)
 *   vsa2_attn_bwd  its gradients dQ, dK, dV with the block mask held fixed
 *                  (Sec. 2.1: the routing decision carries no gradient)
 *
 * Conventions shared by every call
 *   Memory     Every tensor pointer is a DEVICE pointer owned by the caller.
 *              The library never allocates device memory; calls that need
 *              scratch space take a caller-owned workspace whose size is
 *              returned by the matching *_workspace query (except
 *              vsa2_attn_fwd_noalloc, which uses a fixed array of the
 *              library instead).
 *   Streams    Work is enqueued asynchronously on the caller's stream; no call
 *              synchronises the device or reads device memory on the host.
 *   Errors     Argument errors are detected on the host and returned before
 *              any device work is enqueued.  A failed launch returns
 *              VSA2_ERR_HIP.  Nothing is thrown across the ABI.
 *   Layout     Token tensors are contiguous [batch][heads][L][D] in cube-major
 *              token order (Sec. 2.2 "Permutation"): L = N*B, token
 *              l = n*B + beta, cube n = (nt*Nh + nh)*Nw + nw and in-cube
 *              offset beta = (bt*Bh + bh)*Bw + bw (w fastest at both levels).
 *              Pointers to tensors are 16-byte aligned.
 *   Heads      Query head h reads key/value head h / (Hq/Hkv) (Hq % Hkv == 0).
 *   Block ids  Query-block rows are numbered (b*Hq + h)*N + n; key-block rows
 *              (b*Hkv + h)*N + n.
 *   Dtypes     VSA2_F32 or VSA2_BF16 inputs; outputs in the input dtype,
 *              rounded to nearest even from fp32 accumulators.
 *   Threads    Calls are thread-safe; the library keeps no mutable state
 *              other than the per-GPU array of vsa2_attn_fwd_noalloc (whose
 *              overlapping calls on one GPU race, see there).
 *   Determinism  Every output is bitwise reproducible for equal inputs.
 *
 * Supported shapes (other values return VSA2_ERR_UNSUPPORTED):
 *   cube B = Bt*Bh*Bw = 64 tokens; head_dim D in {64, 128};
 *   router score-pooling G = (Bt/Rt)(Bh/Rh)(Bw/Rw) in {1, 2, 4, 8};
 *   N = L/B <= 4096 cubes for vsa2_route.
 *
 * Padded grids (Sec. 2.2, kernel implementation: each axis is padded up to
 * a multiple of the cube size and the padding is masked out).  T, H, W need
 * not be multiples of Bt, Bh, Bw: the grid holds Nt = ceil(T/Bt),
 * Nh = ceil(H/Bh), Nw = ceil(W/Bw) cubes, N = Nt*Nh*Nw, L = N*B, and token
 * (n, beta) is a padding token when nt*Bt + bt >= T, nh*Bh + bh >= H or
 * nw*Bw + bw >= W.  Padding tokens may hold any finite values; no output
 * depends on them.  Every call masks them:
 *   vsa2_pool / vsa2_unpool_add  average over (spread to) the real tokens of
 *       each sub-cube only; a sub-cube without one pools to 0;
 *   vsa2_route  pooled keys without a real token get no score mass, and the
 *       G x G pooling averages over the pooled queries that hold a real token
 *       (every row still sums to 1/G);
 *   vsa2_attn_fwd / _bwd  padding keys are masked out of every softmax;
 *       padding queries give O = 0, LSE = -inf, dQ = 0; padding keys get
 *       dK = dV = 0;
 *   vsa2_gate_merge_bwd  padding tokens are not outputs (dgate = 0, no
 *       contribution to dO_c_hat).
 * Every cube holds at least one real token.
 *
 * Text tokens (MMDiT joint attention: Eq. block_sparse extended with full
 * video-to-text and text-to-video blocks, Sec. 2.2).  With p->text_len =
 * Lt > 0, every token tensor of a (batch, head) holds the joint sequence:
 * the L = N*B video tokens (cube-major, as above), then M = ceil(Lt/B) text
 * blocks of B tokens whose first Lt tokens are real (the rest padding, masked
 * like grid padding).  Ljoint = (N + M)*B tokens per (batch, head); block
 * ids N .. N+M-1 are the text blocks.
 *   vsa2_pool, vsa2_unpool_add  read / update the video part only;
 *   vsa2_route, vsa2_coarse_*   work on pooled video tensors, unchanged;
 *   vsa2_joint_lists  expands the router's video lists to the joint lists:
 *       a video query block keeps its routed video blocks and gains every
 *       text block; a text query block takes every block;
 *   vsa2_attn_*  take joint tensors and joint lists (rows batch*Hq*(N+M));
 *   vsa2_gate_merge(_bwd)  apply the coarse branch to video tokens; text
 *       tokens keep O_f (out = o_f there) and get dgate = 0.
 */
#ifndef VSA2_H
#define VSA2_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    VSA2_OK = 0,
    VSA2_ERR_NULL = 1,         /* a required pointer is NULL                   */
    VSA2_ERR_SHAPE = 2,        /* inconsistent or non-divisible sizes          */
    VSA2_ERR_DTYPE = 3,        /* dtype is not VSA2_F32 / VSA2_BF16            */
    VSA2_ERR_SELECT = 4,       /* invalid selection rule                       */
    VSA2_ERR_CAPACITY = 5,     /* col_cap below what the selection can emit    */
    VSA2_ERR_ALIGN = 6,        /* a tensor pointer is not 16-byte aligned      */
    VSA2_ERR_WORKSPACE = 7,    /* workspace missing or smaller than required   */
    VSA2_ERR_HIP = 8,          /* a HIP launch failed                          */
    VSA2_ERR_UNSUPPORTED = 9   /* valid but outside the supported shapes       */
} vsa2_status;

typedef enum { VSA2_F32 = 0, VSA2_BF16 = 1 } vsa2_dtype;

/* Problem shape, in the paper's notation (Table 1): video grid T x H x W
 * after VAE compression, cube (Bt, Bh, Bw), router input pool (Rt, Rh, Rw). */
typedef struct {
    int32_t batch;
    int32_t heads_q;     /* Hq                                   */
    int32_t heads_kv;    /* Hkv, divides Hq                      */
    int32_t head_dim;    /* D                                    */
    int32_t T, H, W;
    int32_t Bt, Bh, Bw;
    int32_t Rt, Rh, Rw;  /* R_x divides B_x                      */
    int32_t dtype;       /* vsa2_dtype                           */
    int32_t text_len;    /* Lt >= 0 text tokens joined to the video (MMDiT);
                            0 = video only                          */
} vsa2_problem;

typedef enum {
    VSA2_SEL_TOPK = 0,   /* the k best key blocks of each query block         */
    VSA2_SEL_MASS = 1,   /* smallest best-first prefix whose score sum reaches
                            mass * (row total), at most cap blocks            */
    VSA2_SEL_SEQ_TOPK = 2 /* TopK_{N k} per (batch, head) (Sec. 2.2): the
                            N*k best (query block, key block) pairs of the
                            whole N x N map, ties to the lowest flat index
                            n_q*N + n_k; rows get different counts (0 to N) */
} vsa2_sel_mode;

/* Selection rule over the block scores P_r.  Order is (score desc, index
 * asc), decided on the fp32 scores: key-block index within a row for TOPK
 * and MASS, flat index over the sequence's map for SEQ_TOPK. */
typedef struct {
    int32_t mode;        /* vsa2_sel_mode                                    */
    int32_t k;           /* TOPK, SEQ_TOPK: 1 <= k; k >= N keeps every block */
    float mass;          /* MASS: 0 < mass <= 1                              */
    int32_t cap;         /* MASS: 1 <= cap                                   */
} vsa2_select;

/* Human-readable name of a status code (static string). */
const char* vsa2_status_str(vsa2_status s);

/*
 * vsa2_pool - MeanPool over (Pt, Ph, Pw) sub-cubes of every B-cube
 * (Sec. 2.2: Eq. router_start with P = R gives Q_r, K_r; Eq. compress with
 * P = B gives the coarse Q_c, K_c, V_c).
 *   x      [batch][heads][L][D], dtype p->dtype, cube-major ([Ljoint] rows
 *          per head with text tokens; only the video part is read).
 *   out    [batch][heads][N*Gp][D], Gp = (Bt/Pt)(Bh/Ph)(Bw/Pw); row n*Gp + g
 *          with g = (gt*Gh + gh)*Gw + gw.  Each value is the mean of the
 *          Pt*Ph*Pw tokens of its sub-cube (of its real tokens on a padded
 *          grid), accumulated in fp64 and rounded (nearest even) to the dtype.
 *   heads  number of heads of x (Hq for queries, Hkv for keys).
 * Errors: NULL pointers, P_x not dividing B_x, bad dtype/shape, misalignment.
 */
vsa2_status vsa2_pool(const vsa2_problem* p, int32_t heads, const void* x,
                      int32_t Pt, int32_t Ph, int32_t Pw, void* out, hipStream_t stream);

/* Largest number of (query block, key block) pairs the rule can select:
 * batch*Hq*N*min(k, N) for TOPK and SEQ_TOPK, batch*Hq*N*min(cap, N) for
 * MASS.  col_cap
 * of vsa2_route, and the CSC entry capacity, must be at least this. */
vsa2_status vsa2_route_capacity(const vsa2_problem* p, const vsa2_select* s, int64_t* pairs);

/* Bytes of workspace vsa2_route needs for this problem and rule. */
vsa2_status vsa2_route_workspace(const vsa2_problem* p, const vsa2_select* s, size_t* bytes);

/*
 * vsa2_route - the fine-grained router (Sec. 2.2, Eq. router_start ..
 * Eq. router_end) followed by selection and the sparse block lists.
 *   q_r    [batch][Hq][N*G][D]  pooled queries (vsa2_pool with P = R).
 *   k_r    [batch][Hkv][N*G][D] pooled keys.
 *   For pooled query i and every pooled key j of the matching KV head:
 *     s_ij = q_r[i].k_r[j] / sqrt(D), softmax over all N*G keys j, and
 *     P_r[n_q, n_k] = (1/G^2) * sum over the G x G pooled pairs of the two
 *     blocks (so every row of P_r sums to 1/G).  Two passes over the logits
 *     (row log-sum-exp, then softmax + pooling); P_hat is never stored.
 *   Selection by the rule *s: per query block n_q over P_r[n_q, :] (TOPK,
 *   MASS), or over each (batch, head)'s whole map (SEQ_TOPK).
 *   row_ptr [batch*Hq*N + 1]  CSR offsets (row_ptr[0] = 0).
 *   col_idx [col_cap]         selected key blocks, ascending within a row.
 *   kv_ptr  [batch*Hkv*N + 1] CSC offsets over key-block rows, or NULL.
 *   kv_idx  [col_cap]         for each key block, the query blocks that
 *                             selected it, value hq_local*N + n_q with
 *                             hq_local = h mod (Hq/Hkv), ordered ascending;
 *                             NULL together with kv_ptr to skip the CSC.
 *   block_scores  optional [batch][Hq][N][N] fp32 output of P_r; NULL keeps
 *                 the scores in the workspace only.
 *   ws, ws_bytes  workspace of at least vsa2_route_workspace bytes.
 * The number of selected pairs is row_ptr[batch*Hq*N] (device memory).
 * Errors: NULL pointers, bad rule (k < 1, mass outside (0,1], cap < 1),
 * col_cap below vsa2_route_capacity, small workspace, unsupported G or N.
 */
vsa2_status vsa2_route(const vsa2_problem* p, const vsa2_select* s,
                       const void* q_r, const void* k_r,
                       int32_t* row_ptr, int32_t* col_idx, int64_t col_cap,
                       int32_t* kv_ptr, int32_t* kv_idx,
                       float* block_scores, void* ws, size_t ws_bytes, hipStream_t stream);

/* Bytes of workspace vsa2_attn_fwd (pass 0: the work order, one int32 per
 * CSR row, and one byte per query and key block for the large-magnitude
 * flags), vsa2_attn_bwd (pass 1: two fp32 values per query token, its LSE
 * and its Delta, the work orders of the CSR and CSC rows, the flags and one
 * more byte per query block for the row flags, see vsa2_attn_bwd) or
 * vsa2_coarse_bwd (pass 2: one fp32 pair per coarse query) needs.  The
 * work order lists the rows of each XCD's range longest first (a stable
 * counting sort by length class), so the launch's last workgroups are
 * short ones; rows of equal length keep their order. */
vsa2_status vsa2_attn_workspace(const vsa2_problem* p, int32_t pass, size_t* bytes);

/*
 * vsa2_attn_fwd - block-sparse attention (Sec. 2.1 with a block mask M,
 * Eq. block_sparse): for query token l of block n_q, the softmax of
 * q_l.k_j / sqrt(D) over the keys j of the key blocks listed in CSR row
 * n_q, times V.
 *   q [batch][Hq][L][D], k, v [batch][Hkv][L][D]   (dtype p->dtype)
 *   row_ptr, col_idx   CSR as produced by vsa2_route; entries outside
 *                      [0, N) and offsets outside [0, col_cap] are skipped
 *                      (clamped), never dereferenced.
 *   With text tokens (p->text_len > 0) every [L] above is [Ljoint], every
 *   N is N + M and the lists are those of vsa2_joint_lists; the same holds
 *   for the backward calls below.
 *   o   [batch][Hq][L][D] output, dtype p->dtype.
 *   lse [batch][Hq][L] fp32 natural-log log-sum-exp of each query's scaled
 *       scores; a query block with no selected block gets o = 0, lse = -inf.
 *       O is the sum of p V over the sum of p as the products take them
 *       (rounded to the input dtype), a weighted mean with the weights the
 *       products used; lse uses the unrounded sum.
 *   o_lo  optional [batch][Hq][L][D] (dtype p->dtype): NULL for a forward
 *       that no backward follows (inference).  When given, the call writes
 *       the rounding remainder of O (o + o_lo ~ the fp32 result, about 16
 *       significant bits), which vsa2_attn_bwd needs for Delta, and on every
 *       block pair of a query block whose list touches a large-magnitude
 *       block (below; its own flag included) P enters the P.V product as two
 *       bf16 terms, so O itself carries about 16 bits in such a row (where
 *       one-term P on its small pairs would still reach Delta, weighted by
 *       how far each pair's dO . v lies from the row's mean).
 *   Large-magnitude blocks (bf16 problems): a 64-token block of Q, or of K
 *       and V together, holding a real-token value above 7 in magnitude.
 *       bf16 products round P and dS to 8 significant bits; when the tokens
 *       of a block share a large common component those rounding errors add
 *       up along it instead of cancelling, so the rows and block pairs that
 *       touch such a block take two-term (hi + lo) operands (the rules of
 *       each call are given with it) and all others one-term operands.  The
 *       flags are computed on the device in each call that uses them (no
 *       host synchronisation).
 *   ws, ws_bytes  workspace of vsa2_attn_workspace(p, 0) bytes, 256-byte
 *       aligned.
 * Errors: NULL pointers, shape/dtype, misalignment, small workspace.
 */
vsa2_status vsa2_attn_fwd(const vsa2_problem* p, const void* q, const void* k, const void* v,
                          const int32_t* row_ptr, const int32_t* col_idx, int64_t col_cap,
                          void* o, float* lse, void* o_lo, void* ws, size_t ws_bytes,
                          hipStream_t stream);

/*
 * vsa2_attn_fwd_noalloc - vsa2_attn_fwd for callers that cannot allocate
 * device memory (code under HIP graph capture, serving loops or harnesses
 * that forbid hipMalloc): the same computation and results, bit for bit,
 * with the call's workspace (work order and block flags) in a fixed array
 * of the library instead of a caller buffer.  The call allocates nothing.
 *   Arguments as for vsa2_attn_fwd, without ws / ws_bytes; the stream's
 *   device must be the current device.
 *   Limit: the array holds VSA2_NOALLOC_SCRATCH_BYTES (2 MiB) per GPU, for
 *   as long as the process runs; a problem whose forward workspace
 *   (vsa2_attn_workspace(p, 0)) is larger returns VSA2_ERR_WORKSPACE before
 *   any device work (about 6 bytes per query-block row: up to about
 *   349,000 rows batch * heads_q * blocks with heads_kv = heads_q).
 *   Every call on one GPU uses that GPU's one array: calls that overlap on
 *   one GPU (concurrent streams, or two graphs replayed at once) race and
 *   must be ordered by the caller.  Each call rewrites all of the array it
 *   reads, so what an earlier call left there does not matter.
 * Errors: as for vsa2_attn_fwd; VSA2_ERR_WORKSPACE for a problem beyond the
 *   limit; VSA2_ERR_HIP if the array's device address cannot be obtained.
 */
#define VSA2_NOALLOC_SCRATCH_BYTES ((size_t)2 << 20)
vsa2_status vsa2_attn_fwd_noalloc(const vsa2_problem* p, const void* q, const void* k, const void* v,
                                  const int32_t* row_ptr, const int32_t* col_idx, int64_t col_cap,
                                  void* o, float* lse, void* o_lo, hipStream_t stream);

/*
 * vsa2_attn_bwd - gradients of vsa2_attn_fwd with the block lists fixed
 * (no gradient reaches the router, Sec. 2.1).  With p the softmax row of
 * query l over its gathered keys:
 *   Delta_l = dO_l . O_l,  dS_lj = p_lj (dO_l . v_j - Delta_l),
 *   dQ_l = sum_j dS_lj k_j / sqrt(D),
 *   dK_j = sum_l dS_lj q_l / sqrt(D),  dV_j = sum_l p_lj dO_l,
 * where the sums over l run over every query (of every query head of the KV
 * group) whose block selected j's block.
 *   q, k, v, o, lse   as for vsa2_attn_fwd (o, lse from the forward call)
 *   o_lo  required: the forward's o_lo (Delta uses o + o_lo).  On block
 *         pairs that touch a large-magnitude block (see vsa2_attn_fwd) P
 *         enters the dV product as two bf16 terms; dS enters the dK and dQ
 *         products as two terms on every pair of a query block whose list
 *         touches a large-magnitude block (its own flag included) or one of
 *         whose queries (with attention mass) has |Delta| above 16: dS is
 *         then a small difference of large terms, which one-term rounding
 *         would not keep to the gradients' accuracy.
 *   dout  [batch][Hq][L][D]  dO
 *   row_ptr, col_idx  the CSR; kv_ptr, kv_idx its transpose (vsa2_route)
 *   dq [batch][Hq][L][D], dk, dv [batch][Hkv][L][D]  outputs, dtype p->dtype;
 *   key blocks no query selected get dk = dv = 0.
 * Errors: as for vsa2_attn_fwd; o_lo NULL is VSA2_ERR_NULL.
 */
vsa2_status vsa2_attn_bwd(const vsa2_problem* p, const void* q, const void* k, const void* v,
                          const void* o, const float* lse, const void* o_lo, const void* dout,
                          const int32_t* row_ptr, const int32_t* col_idx,
                          const int32_t* kv_ptr, const int32_t* kv_idx, int64_t col_cap,
                          void* dq, void* dk, void* dv, void* ws, size_t ws_bytes,
                          hipStream_t stream);

/*
 * The backward in three stages, for callers that schedule or time them one
 * by one.  vsa2_attn_bwd is exactly these three calls in this order on one
 * stream; the stages communicate through ws (vsa2_attn_workspace(p, 1)
 * bytes), which must not be reused in between.
 *
 * vsa2_attn_bwd_prep - per query token l: LSE_l and Delta_l = dO_l . O_l
 *   with O_l = o_l + o_lo_l, and (bf16) the large-magnitude flags of the
 *   blocks of q, k, v, stored in ws.
 *   q, k, v, o, lse, o_lo, dout  as for vsa2_attn_bwd (o_lo required).
 */
vsa2_status vsa2_attn_bwd_prep(const vsa2_problem* p, const void* q, const void* k, const void* v, const void* o,
                               const float* lse, const void* o_lo, const void* dout, void* ws, size_t ws_bytes,
                               hipStream_t stream);

/*
 * vsa2_attn_bwd_dkdv - dK and dV of vsa2_attn_bwd, one key block at a time
 *   over the query blocks of its transposed list (kv_ptr, kv_idx).
 *   ws           as written by vsa2_attn_bwd_prep (this stage also writes
 *                its work order and the query blocks' row flags there; the
 *                dQ stage derives its rows' flags from its own lists).
 *   dk, dv       [batch][Hkv][L][D] outputs, dtype p->dtype.
 */
vsa2_status vsa2_attn_bwd_dkdv(const vsa2_problem* p, const void* q, const void* k, const void* v,
                               const void* dout, const int32_t* kv_ptr, const int32_t* kv_idx, int64_t col_cap,
                               void* dk, void* dv, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * vsa2_attn_bwd_dq - dQ of vsa2_attn_bwd, one query block at a time over its
 *   CSR row (row_ptr, col_idx).  ws as for vsa2_attn_bwd_dkdv.
 *   dq  [batch][Hq][L][D] output, dtype p->dtype.
 */
vsa2_status vsa2_attn_bwd_dq(const vsa2_problem* p, const void* q, const void* k, const void* v,
                             const void* dout, const int32_t* row_ptr, const int32_t* col_idx, int64_t col_cap,
                             void* dq, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * Coarse branch and gated merge (Sec. 2.2, "Coarse Branch" and "Gated
 * Merge").  With [Q_c, K_c, V_c] = MeanPool_B([Q, K, V]) (vsa2_pool with
 * P = B, one row per cube):
 *   O_c_hat = Softmax(Q_c K_c^T / sqrt(D)) V_c       (dense over the N cubes)
 *   O = tanh(g) * Repeat_B(O_c_hat) + O_f            (O_f from vsa2_attn_fwd)
 * where g = X W_g holds one gate pre-activation per token and query head.
 * The gradients: vsa2_gate_merge_bwd gives dO_c_hat and dg (dO_f is dO
 * itself), vsa2_coarse_bwd gives dQ_c, dK_c, dV_c, and vsa2_unpool_add adds
 * the MeanPool adjoint of those onto the token gradients dQ, dK, dV.
 *
 * vsa2_coarse_fwd
 *   q_c [batch][Hq][N][D], k_c, v_c [batch][Hkv][N][D]  (dtype p->dtype)
 *   o_c [batch][Hq][N][D] output O_c_hat; lse_c [batch][Hq][N] fp32
 *   natural-log log-sum-exp of each coarse query's scaled scores.  Query head
 *   h reads KV head h / (Hq/Hkv).
 * Errors: NULL pointers, shape/dtype, misalignment, batch*Hq > 65535.
 */
vsa2_status vsa2_coarse_fwd(const vsa2_problem* p, const void* q_c, const void* k_c, const void* v_c, void* o_c,
                            float* lse_c, hipStream_t stream);

/*
 * vsa2_coarse_bwd - gradients of vsa2_coarse_fwd for do_c = dO_c_hat:
 *   dq_c [batch][Hq][N][D], dk_c, dv_c [batch][Hkv][N][D] outputs (dk_c and
 *   dv_c summed over the query heads of each KV group).  The softmax
 *   statistics are recomputed (one more pass over the N x N scores) with P
 *   and dS entering the products as two bf16 terms each: the cube means are
 *   dominated by their common component, which amplifies one-term rounding.
 *   ws, ws_bytes  vsa2_attn_workspace(p, 2) bytes, 256-byte aligned.
 */
vsa2_status vsa2_coarse_bwd(const vsa2_problem* p, const void* q_c, const void* k_c, const void* v_c,
                            const void* do_c, void* dq_c, void* dk_c, void* dv_c, void* ws, size_t ws_bytes,
                            hipStream_t stream);

/*
 * vsa2_gate_merge - out[l] = tanh(gate[l]) * o_c[cube of l] + o_f[l].
 *   gate [batch][Hq][L] fp32 pre-activations; o_c [batch][Hq][N][D];
 *   o_f, out [batch][Hq][L][D] (out may alias o_f).
 */
vsa2_status vsa2_gate_merge(const vsa2_problem* p, const float* gate, const void* o_c, const void* o_f, void* out,
                            hipStream_t stream);

/*
 * vsa2_gate_merge_bwd - for dout = dO:
 *   do_c [batch][Hq][N][D] = sum over the B tokens l of each cube of
 *        tanh(gate[l]) dout[l];
 *   dgate [batch][Hq][L] fp32 = (1 - tanh(gate[l])^2) (dout[l] . o_c[cube]).
 * On a padded grid the sum runs over real tokens and padding tokens get
 * dgate = 0.
 */
vsa2_status vsa2_gate_merge_bwd(const vsa2_problem* p, const float* gate, const void* o_c, const void* dout,
                                void* do_c, float* dgate, hipStream_t stream);

/*
 * Joint video + text block lists (p->text_len > 0).
 *
 * vsa2_joint_capacity: entries the joint CSR can hold at most for the
 *   router's rule: vsa2_route_capacity + batch*Hq*N*M (text blocks of the
 *   video rows) + batch*Hq*M*(N+M) (the text rows).
 * vsa2_joint_workspace: bytes of workspace vsa2_joint_lists needs.
 * vsa2_joint_lists: from the router's video lists (row_ptr [batch*Hq*N+1],
 *   col_idx [col_cap]) writes
 *     j_row_ptr [batch*Hq*(N+M) + 1], j_col_idx [j_cap]: joint query block
 *       (b*Hq + h)*(N+M) + n lists its video blocks (n < N: the routed ones
 *       in their order, entries outside [0, N) become -1 and are skipped by
 *       the attention) followed by N .. N+M-1; a text block n >= N lists
 *       0 .. N+M-1;
 *     j_kv_ptr [batch*Hkv*(N+M) + 1], j_kv_idx [j_cap]: its transpose, value
 *       hq_local*(N+M) + n_q ascending (the CSC of vsa2_route with N+M
 *       blocks).
 *   Index work only; the lists feed vsa2_attn_fwd / vsa2_attn_bwd with the
 *   same problem.
 * Errors: NULL pointers; text_len = 0 (VSA2_ERR_SHAPE); j_cap below
 *   col_cap + batch*Hq*(N*M + M*(N+M)) (VSA2_ERR_CAPACITY); workspace
 *   missing or too small.
 */
vsa2_status vsa2_joint_capacity(const vsa2_problem* p, const vsa2_select* s, int64_t* pairs);
vsa2_status vsa2_joint_workspace(const vsa2_problem* p, size_t* bytes);
vsa2_status vsa2_joint_lists(const vsa2_problem* p, const int32_t* row_ptr, const int32_t* col_idx,
                             int64_t col_cap, int32_t* j_row_ptr, int32_t* j_col_idx, int64_t j_cap,
                             int32_t* j_kv_ptr, int32_t* j_kv_idx, void* ws, size_t ws_bytes,
                             hipStream_t stream);

/*
 * vsa2_unpool_add - the MeanPool adjoint (gradient of vsa2_pool with the
 * same Pt, Ph, Pw): every token of sub-cube (n, g) gets dx_c[n*Gp + g] /
 * (Pt*Ph*Pw) added, in place (on a padded grid: every real token, divided
 * by the number of real tokens of the sub-cube; padding tokens are left
 * unchanged).
 *   dx_c [batch][heads][N*Gp][D]; dx [batch][heads][L][D] (updated).
 */
vsa2_status vsa2_unpool_add(const vsa2_problem* p, int32_t heads, const void* dx_c, int32_t Pt, int32_t Ph,
                            int32_t Pw, void* dx, hipStream_t stream);

/*
 * vsa2_mfma_peak_probe - a measurement aid, not part of the attention path:
 * the dense bf16 MFMA rate this GPU reaches, the measured counterpart of the
 * published peak the attention kernels are rated against.  Launches one
 * workgroup of 16 waves per CU; each wave runs `iters` rounds of 4
 * independent 32x32x16 bf16 MFMA chains on register operands.  The caller
 * times the launch (events on `stream`) and divides *flops by the time.
 *   iters  rounds (>= 0; 0 launches nothing and only reports *flops = 0).
 *   sink   device float, written only in a case no input reaches (it keeps
 *          the chains alive); may be NULL when iters = 0.
 *   flops  host int64: the work of the launch, CUs * 16 * 4 * iters * 32768.
 * Errors: NULL flops (or sink with iters > 0); iters < 0 (VSA2_ERR_SHAPE).
 */
vsa2_status vsa2_mfma_peak_probe(int32_t iters, float* sink, int64_t* flops, hipStream_t stream);

/*
 * vsa2_dq_atomic_probe - a measurement aid, not part of the attention path:
 * the atomic traffic a fused backward (dK, dV and dQ in one key-stationary
 * pass, the alternative to the two-kernel backward of vsa2_attn_bwd) would
 * spend on dQ alone.  For every entry of every key block's transposed list
 * (kv_ptr, kv_idx from vsa2_route) it adds 1.0 with an fp32 atomic to every
 * element of the listed query block's 64 x D tile of acc, and does nothing
 * else; the caller times the launch.
 *   acc  [batch][Hq][L][D] fp32 device buffer (accumulates entry counts).
 * Errors: NULL pointers, shape, negative col_cap, misaligned acc.
 */
vsa2_status vsa2_dq_atomic_probe(const vsa2_problem* p, const int32_t* kv_ptr, const int32_t* kv_idx,
                                 int64_t col_cap, float* acc, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* VSA2_H */
