/*
 * Plain CPU oracle for the VSA2 routed sparse-attention path.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, includes
 * or calls this file; only the test-suite, the smoke check and the CPU
 * baseline leg of the benchmark load it.  It shares no code, header, table or
 * helper with the HIP kernels.
 *
 * Paper: "Improving Video Sparse Attention with Fine-grained Router and Sparse
 * Rebasing" (VSA2).  Every function below follows one passage of its Method
 * section (Sec. 2) and is written for a reader checking it by eye:
 *   - every tensor value is widened to double on read, every sum is a plain
 *     loop in double, nothing is blocked, fused or reordered;
 *   - inputs arrive as float arrays holding the exact input values (a bf16
 *     value widens exactly into a float);
 *   - layout is cube-major [batch][head][L][D] with L = N * B tokens
 *     (Sec. 2.2 "Permutation"): token l = n*B + beta, n = (nt*Nh + nh)*Nw + nw,
 *     beta = (bt*Bh + bh)*Bw + bw (raster order, w fastest, at every level).
 *
 * Readings of points the paper leaves open:
 *   - pooled router inputs Q_r, K_r are rounded to the input dtype (RNE);
 *   - router softmax runs over all N*G pooled keys with scale 1/sqrt(D);
 *   - MeanPool_{GxG} is a true mean, so every P_r row sums to 1/G;
 *   - selection decides in fp32: scores are rounded to float, ordered by
 *     (score desc, block index asc);
 *   - a query block with no selected block gets O = 0, LSE = -inf, dQ = 0;
 *   - query head h reads KV head h / (Hq/Hkv).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ---------------------------------------------------------------------- */
/* Rounding of a double to the input dtype.                                */
/* ---------------------------------------------------------------------- */

/* Round-to-nearest-even of x to bfloat16 (8 significant bits, float's
 * exponent range), returned as the exactly representable float. */
static double round_to_bf16(double x)
{
    if (x == 0.0 || isnan(x) || isinf(x)) return x;
    double ax = fabs(x);
    double q;
    if (ax < ldexp(1.0, -126)) {
        /* bf16 subnormals are multiples of 2^-133 */
        q = nearbyint(x * ldexp(1.0, 133)) * ldexp(1.0, -133);
    } else {
        int e;
        double m = frexp(x, &e);           /* x = m * 2^e, 0.5 <= |m| < 1 */
        q = ldexp(nearbyint(ldexp(m, 8)), e - 8);  /* keep 8 bits, RNE */
    }
    if (fabs(q) > 3.3895313892515355e38) q = copysign(INFINITY, x);
    return q;
}

static float round_to_dtype(double x, int dtype_bf16)
{
    return dtype_bf16 ? (float)round_to_bf16(x) : (float)x;
}

void vo_round_bf16(const double* in, float* out, int64_t n)
{
    for (int64_t i = 0; i < n; ++i) out[i] = (float)round_to_bf16(in[i]);
}

/* ---------------------------------------------------------------------- */
/* Padded grids (Sec. 2.2 "Kernel Implementation": each of T, H, W is      */
/* padded up to a multiple of the cube size and padding is masked out).    */
/* geom = {T, H, W, Bt, Bh, Bw, Lt}: the real grid, the cube and the text  */
/* length.  The cube-major layout holds N = ceil(T/Bt) ceil(H/Bh)          */
/* ceil(W/Bw) video cubes of B tokens; token beta of cube n is real iff    */
/* its grid position lies inside the real grid.  With text tokens (MMDiT   */
/* joint attention, the extension of Eq. block_sparse in Sec. 2.2) the     */
/* sequence of a (batch, head) continues with ceil(Lt/B) text blocks of B  */
/* tokens, of which the first Lt are real.  geom == NULL: every token is   */
/* real.                                                                   */
/* ---------------------------------------------------------------------- */

static int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

static int vo_token_real(const int* geom, int64_t n, int beta)
{
    if (!geom) return 1;
    const int T = geom[0], H = geom[1], W = geom[2], Bt = geom[3], Bh = geom[4], Bw = geom[5];
    const int64_t Nh = ceil_div(H, Bh), Nw = ceil_div(W, Bw);
    const int64_t Nv = ceil_div(T, Bt) * Nh * Nw;
    if (n >= Nv)                        /* text block n - Nv */
        return (n - Nv) * (int64_t)(Bt * Bh * Bw) + beta < geom[6];
    const int64_t nt = n / (Nh * Nw), nh = (n / Nw) % Nh, nw = n % Nw;
    const int bt = beta / (Bh * Bw), bh = (beta / Bw) % Bh, bw = beta % Bw;
    return nt * Bt + bt < T && nh * Bh + bh < H && nw * Bw + bw < W;
}

/* Number of real tokens of sub-cube g (pool size Pt x Ph x Pw) of cube n. */
static int vo_subcube_real_count(const int* geom, int64_t n, int g, int Pt, int Ph, int Pw)
{
    const int Bh = geom[4], Bw = geom[5];
    const int Gh = Bh / Ph, Gw = Bw / Pw;
    const int gt = g / (Gh * Gw), gh = (g / Gw) % Gh, gw = g % Gw;
    int c = 0;
    for (int rt = 0; rt < Pt; ++rt)
        for (int rh = 0; rh < Ph; ++rh)
            for (int rw = 0; rw < Pw; ++rw)
                c += vo_token_real(geom, n, ((gt * Pt + rt) * Bh + gh * Ph + rh) * Bw + gw * Pw + rw);
    return c;
}

/* ---------------------------------------------------------------------- */
/* MeanPool over sub-cubes (Eq. router_start for P = R; Eq. compress for   */
/* P = B).                                                                 */
/* ---------------------------------------------------------------------- */

/* x: [nbh][N*B][D] cube-major.  out: [nbh][N*Gp][D] with Gp = B/P sub-cubes
 * per cube, ordered (n, g), g = (gt*Gh + gh)*Gw + gw.  Each output row is the
 * mean of the real tokens of its sub-cube (all P = Pt*Ph*Pw of them unless
 * the grid is padded), rounded to the dtype; a sub-cube with no real token
 * gives 0. */
void vo_pool(const float* x, int64_t nbh, int T, int H, int W,
             int Bt, int Bh, int Bw, int Pt, int Ph, int Pw, int D,
             int dtype_bf16, float* out)
{
    const int geom[7] = {T, H, W, Bt, Bh, Bw, 0};
    const int64_t N = ceil_div(T, Bt) * ceil_div(H, Bh) * ceil_div(W, Bw);
    const int B = Bt * Bh * Bw;
    const int Gt = Bt / Pt, Gh = Bh / Ph, Gw = Bw / Pw;
    const int G = Gt * Gh * Gw;
#pragma omp parallel for schedule(static)
    for (int64_t bh = 0; bh < nbh; ++bh) {
        for (int64_t n = 0; n < N; ++n) {
            for (int gt = 0; gt < Gt; ++gt)
            for (int gh = 0; gh < Gh; ++gh)
            for (int gw = 0; gw < Gw; ++gw) {
                const int g = (gt * Gh + gh) * Gw + gw;
                float* o = out + ((bh * N + n) * G + g) * (int64_t)D;
                for (int d = 0; d < D; ++d) {
                    double sum = 0.0;
                    int count = 0;
                    for (int rt = 0; rt < Pt; ++rt)
                    for (int rh = 0; rh < Ph; ++rh)
                    for (int rw = 0; rw < Pw; ++rw) {
                        const int bt = gt * Pt + rt, bhh = gh * Ph + rh, bw = gw * Pw + rw;
                        const int beta = (bt * Bh + bhh) * Bw + bw;
                        if (!vo_token_real(geom, n, beta)) continue;
                        sum += (double)x[((bh * N + n) * B + beta) * (int64_t)D + d];
                        ++count;
                    }
                    o[d] = count ? round_to_dtype(sum / (double)count, dtype_bf16) : 0.0f;
                }
            }
        }
    }
}

/* ---------------------------------------------------------------------- */
/* Router block scores (Eq. router_start .. Eq. router_end).               */
/* ---------------------------------------------------------------------- */

/* q_r: [nb][Hq][N*G][D], k_r: [nb][Hkv][N*G][D] (pooled, already rounded).
 * rows[i] = (b*Hq + h)*N + nq names one query block.  For each listed row:
 *   s[gq][j]  = Q_r[nq*G+gq] . K_r[j] / sqrt(D)       for all j < N*G,
 *   lse[gq]   = log sum_j exp(s[gq][j])                (max-shifted),
 *   P_hat     = exp(s - lse)                            (row softmax),
 *   P_r[nk]   = (1/G^2) sum_{gq,gk} P_hat[gq][nk*G+gk]  (MeanPool_{GxG}).
 * scores: [nrows][N]; lse_out: [nrows][G] or NULL. */
void vo_router_scores(const float* q_r, const float* k_r, int nb, int Hq, int Hkv,
                      int64_t N, int G, int D, const int64_t* rows, int64_t nrows,
                      double* scores, double* lse_out, const int* geom, int Rt, int Rh, int Rw)
{
    (void)nb;
    const int64_t NG = N * G;
    const int grp = Hq / Hkv;
    const double scale = 1.0 / sqrt((double)D);
#pragma omp parallel
    {
        double* s = (double*)malloc(sizeof(double) * (size_t)NG);
        uint8_t* real = (uint8_t*)malloc((size_t)NG);
        /* pooled keys (and queries) with no real token take no part */
        for (int64_t j = 0; j < NG; ++j)
            real[j] = geom ? vo_subcube_real_count(geom, j / G, (int)(j % G), Rt, Rh, Rw) > 0 : 1;
#pragma omp for schedule(dynamic, 1)
        for (int64_t r = 0; r < nrows; ++r) {
            const int64_t row = rows[r];
            const int64_t bh = row / N, nq = row % N;
            const int64_t b = bh / Hq, h = bh % Hq;
            const int64_t hkv = h / grp;
            const float* K = k_r + (b * Hkv + hkv) * NG * (int64_t)D;
            double* out = scores + r * N;
            for (int64_t nk = 0; nk < N; ++nk) out[nk] = 0.0;
            int gq_real = 0;
            for (int gq = 0; gq < G; ++gq) gq_real += real[nq * G + gq];
            for (int gq = 0; gq < G; ++gq) {
                const float* qi = q_r + ((bh * N + nq) * G + gq) * (int64_t)D;
                double m = -INFINITY;
                for (int64_t j = 0; j < NG; ++j) {
                    double dot = 0.0;
                    for (int d = 0; d < D; ++d) dot += (double)qi[d] * (double)K[j * D + d];
                    s[j] = real[j] ? dot * scale : -INFINITY;
                    if (s[j] > m) m = s[j];
                }
                double sum = 0.0;
                for (int64_t j = 0; j < NG; ++j) sum += exp(s[j] - m);
                const double lse = m + log(sum);
                if (lse_out) lse_out[r * G + gq] = lse;
                if (!real[nq * G + gq]) continue;
                /* MeanPool_{GxG} over the pooled queries that hold a real
                 * token (all G of them unless the grid is padded) */
                for (int64_t nk = 0; nk < N; ++nk)
                    for (int gk = 0; gk < G; ++gk)
                        out[nk] += exp(s[nk * G + gk] - lse) / ((double)G * (double)gq_real);
            }
        }
        free(real);
        free(s);
    }
}

/* ---------------------------------------------------------------------- */
/* Selection.                                                              */
/* ---------------------------------------------------------------------- */

typedef struct { float v; int32_t i; } vo_scored;

/* (score desc, index asc) */
static int cmp_desc(const void* a, const void* b)
{
    const vo_scored* x = (const vo_scored*)a;
    const vo_scored* y = (const vo_scored*)b;
    if (x->v > y->v) return -1;
    if (x->v < y->v) return 1;
    return (x->i > y->i) - (x->i < y->i);
}

static int cmp_int(const void* a, const void* b)
{
    const int32_t x = *(const int32_t*)a, y = *(const int32_t*)b;
    return (x > y) - (x < y);
}

/* Per-query-block selection over one row of N block scores.
 *   mode 0 (top-k):  the k best blocks (k > N keeps all N);
 *   mode 1 (mass):   the smallest prefix of the sorted row whose sum reaches
 *                    mass * (row total), capped at cap blocks.
 * Scores are rounded to float first: the decision is taken in fp32.
 * counts: [nrows]; idx: [nrows][N], selected blocks ascending, rest -1. */
void vo_select_rows(const double* scores, int64_t nrows, int N, int mode, int k,
                    double mass, int cap, int32_t* counts, int32_t* idx)
{
#pragma omp parallel
    {
        vo_scored* a = (vo_scored*)malloc(sizeof(vo_scored) * (size_t)N);
#pragma omp for schedule(dynamic, 16)
        for (int64_t r = 0; r < nrows; ++r) {
            for (int j = 0; j < N; ++j) { a[j].v = (float)scores[r * N + j]; a[j].i = j; }
            qsort(a, (size_t)N, sizeof(vo_scored), cmp_desc);
            int c;
            if (mode == 0) {
                c = k < N ? k : N;
            } else {
                double total = 0.0;
                for (int j = 0; j < N; ++j) total += (double)a[j].v;
                const double thr = mass * total;
                double cum = 0.0;
                c = N;
                for (int j = 0; j < N; ++j) {
                    cum += (double)a[j].v;
                    if (cum >= thr) { c = j + 1; break; }
                }
                if (c > cap) c = cap;
            }
            int32_t* out = idx + r * (int64_t)N;
            for (int j = 0; j < c; ++j) out[j] = a[j].i;
            qsort(out, (size_t)c, sizeof(int32_t), cmp_int);
            for (int j = c; j < N; ++j) out[j] = -1;
            counts[r] = c;
        }
        free(a);
    }
}

/* Sequence-level top-(N*k) over the flattened N x N score map of one
 * (batch, head) (the paper's TopK_{NK}): keeps the N*k best (query block,
 * key block) pairs, ties broken by flat index nq*N + nk.  scores: [nseq][N*N],
 * sel: [nseq][N*N] set to 1 for kept pairs, 0 otherwise. */
void vo_select_seq(const double* scores, int64_t nseq, int N, int k, uint8_t* sel)
{
    const int64_t NN = (int64_t)N * N;
    int64_t keep = (int64_t)N * k;
    if (keep > NN) keep = NN;
#pragma omp parallel
    {
        vo_scored* a = (vo_scored*)malloc(sizeof(vo_scored) * (size_t)NN);
#pragma omp for schedule(dynamic, 1)
        for (int64_t s = 0; s < nseq; ++s) {
            for (int64_t j = 0; j < NN; ++j) { a[j].v = (float)scores[s * NN + j]; a[j].i = (int32_t)j; }
            qsort(a, (size_t)NN, sizeof(vo_scored), cmp_desc);
            uint8_t* out = sel + s * NN;
            memset(out, 0, (size_t)NN);
            for (int64_t j = 0; j < keep; ++j) out[a[j].i] = 1;
        }
        free(a);
    }
}

/* ---------------------------------------------------------------------- */
/* Block-sparse attention forward (Sec. 2.1 masked attention; Eq.          */
/* block_sparse).                                                          */
/* ---------------------------------------------------------------------- */

/* One query token against the keys of its selected blocks.  Fills p[] (the
 * softmax row over the gathered keys, in CSR order), o[D] and returns the
 * natural-log LSE.  An empty selection gives o = 0 and -inf. */
static double token_forward(const float* qv, const float* K, const float* V, int D, int B,
                            const int32_t* sel, int nsel, double scale, double* p, double* o,
                            const int* geom)
{
    const int nkeys = nsel * B;
    for (int d = 0; d < D; ++d) o[d] = 0.0;
    if (nkeys == 0) return -INFINITY;
    double m = -INFINITY;
    for (int c = 0; c < nsel; ++c)
        for (int t = 0; t < B; ++t) {
            const int64_t j = (int64_t)sel[c] * B + t;
            if (!vo_token_real(geom, sel[c], t)) {   /* padding key: masked out */
                p[c * B + t] = -INFINITY;
                continue;
            }
            double dot = 0.0;
            for (int d = 0; d < D; ++d) dot += (double)qv[d] * (double)K[j * D + d];
            p[c * B + t] = dot * scale;
            if (p[c * B + t] > m) m = p[c * B + t];
        }
    if (m == -INFINITY) {                        /* only padding keys selected */
        for (int j = 0; j < nkeys; ++j) p[j] = 0.0;
        return -INFINITY;
    }
    double sum = 0.0;
    for (int j = 0; j < nkeys; ++j) { p[j] = exp(p[j] - m); sum += p[j]; }
    for (int j = 0; j < nkeys; ++j) p[j] /= sum;
    for (int c = 0; c < nsel; ++c)
        for (int t = 0; t < B; ++t) {
            const int64_t j = (int64_t)sel[c] * B + t;
            for (int d = 0; d < D; ++d) o[d] += p[c * B + t] * (double)V[j * D + d];
        }
    return m + log(sum);
}

/* q: [nb][Hq][L][D]; k, v: [nb][Hkv][L][D]; CSR row_ptr/col_idx over rows
 * (b*Hq + h)*N + n.  For each listed row, writes O: [nq][B][D] and
 * LSE: [nq][B] (natural log) of its B query tokens. */
void vo_attn_fwd(const float* q, const float* k, const float* v, int nb, int Hq, int Hkv,
                 int64_t L, int D, int B, const int32_t* row_ptr, const int32_t* col_idx,
                 const int64_t* qrows, int64_t nq, double* o, double* lse, const int* geom)
{
    (void)nb;
    const int64_t N = L / B;
    const int grp = Hq / Hkv;
    const double scale = 1.0 / sqrt((double)D);
#pragma omp parallel
    {
        double* p = (double*)malloc(sizeof(double) * (size_t)L);
#pragma omp for schedule(dynamic, 1)
        for (int64_t r = 0; r < nq; ++r) {
            const int64_t row = qrows[r];
            const int64_t bh = row / N, n = row % N;
            const int64_t b = bh / Hq, h = bh % Hq, hkv = h / grp;
            const float* K = k + (b * Hkv + hkv) * L * D;
            const float* V = v + (b * Hkv + hkv) * L * D;
            const int32_t* sel = col_idx + row_ptr[row];
            const int nsel = row_ptr[row + 1] - row_ptr[row];
            for (int t = 0; t < B; ++t) {
                const float* qv = q + (bh * L + n * B + t) * D;
                if (!vo_token_real(geom, n, t)) {       /* padding query: no output */
                    for (int d = 0; d < D; ++d) o[(r * B + t) * (int64_t)D + d] = 0.0;
                    lse[r * B + t] = -INFINITY;
                    continue;
                }
                lse[r * B + t] = token_forward(qv, K, V, D, B, sel, nsel, scale, p,
                                               o + (r * B + t) * (int64_t)D, geom);
            }
        }
        free(p);
    }
}

/* ---------------------------------------------------------------------- */
/* Block-sparse attention backward.  The mask is a constant: no gradient   */
/* reaches the router (Sec. 2.1, gradient-free routing).  With p the       */
/* softmax row of token l over its gathered keys j:                        */
/*   Delta_l = dO_l . O_l,  dP_j = dO_l . V_j,  dS_j = p_j (dP_j - Delta_l) */
/*   dQ_l = scale * sum_j dS_j K_j,  dK_j += scale * dS_j Q_l,             */
/*   dV_j += p_j dO_l  (summed over every query token that reads key j).   */
/* ---------------------------------------------------------------------- */

/* dQ for listed query blocks: qrows as in vo_attn_fwd, dq: [nq][B][D]. */
void vo_attn_bwd_dq(const float* q, const float* k, const float* v, const float* dout,
                    int nb, int Hq, int Hkv, int64_t L, int D, int B,
                    const int32_t* row_ptr, const int32_t* col_idx,
                    const int64_t* qrows, int64_t nq, double* dq, const int* geom)
{
    (void)nb;
    const int64_t N = L / B;
    const int grp = Hq / Hkv;
    const double scale = 1.0 / sqrt((double)D);
#pragma omp parallel
    {
        double* p = (double*)malloc(sizeof(double) * (size_t)L);
        double* o = (double*)malloc(sizeof(double) * (size_t)D);
#pragma omp for schedule(dynamic, 1)
        for (int64_t r = 0; r < nq; ++r) {
            const int64_t row = qrows[r];
            const int64_t bh = row / N, n = row % N;
            const int64_t b = bh / Hq, h = bh % Hq, hkv = h / grp;
            const float* K = k + (b * Hkv + hkv) * L * D;
            const float* V = v + (b * Hkv + hkv) * L * D;
            const int32_t* sel = col_idx + row_ptr[row];
            const int nsel = row_ptr[row + 1] - row_ptr[row];
            for (int t = 0; t < B; ++t) {
                const int64_t tok = bh * L + n * B + t;
                const float* qv = q + tok * D;
                const float* dov = dout + tok * D;
                double* g = dq + (r * B + t) * (int64_t)D;
                for (int d = 0; d < D; ++d) g[d] = 0.0;
                if (!vo_token_real(geom, n, t)) continue;   /* padding query: dQ = 0 */
                token_forward(qv, K, V, D, B, sel, nsel, scale, p, o, geom);
                double delta = 0.0;
                for (int d = 0; d < D; ++d) delta += (double)dov[d] * o[d];
                for (int c = 0; c < nsel; ++c)
                    for (int u = 0; u < B; ++u) {
                        const int64_t j = (int64_t)sel[c] * B + u;
                        double dp = 0.0;
                        for (int d = 0; d < D; ++d) dp += (double)dov[d] * (double)V[j * D + d];
                        const double ds = p[c * B + u] * (dp - delta);
                        for (int d = 0; d < D; ++d) g[d] += scale * ds * (double)K[j * D + d];
                    }
            }
        }
        free(p);
        free(o);
    }
}

/* dK and dV for listed key blocks: kvrows[i] = (b*Hkv + hkv)*N + nk.
 * Every query token of every query head of the KV head's group whose row
 * selects block nk contributes.  dk, dv: [nkv][B][D].
 * The (key block, selecting query block) pairs are enumerated first and their
 * contributions computed independently (in parallel), then summed per key
 * block in pair order, so the result does not depend on the thread count. */
void vo_attn_bwd_dkdv(const float* q, const float* k, const float* v, const float* dout,
                      int nb, int Hq, int Hkv, int64_t L, int D, int B,
                      const int32_t* row_ptr, const int32_t* col_idx,
                      const int64_t* kvrows, int64_t nkv, double* dk, double* dv, const int* geom)
{
    (void)nb;
    const int64_t N = L / B;
    const int grp = Hq / Hkv;
    const double scale = 1.0 / sqrt((double)D);
    const int64_t BD = (int64_t)B * D;

    /* 1. pairs (kv index r, query-block row, position of nk in that row) */
    int64_t npairs = 0, cap = 16;
    int64_t* pr = (int64_t*)malloc(sizeof(int64_t) * 3 * (size_t)cap);
    for (int64_t r = 0; r < nkv; ++r) {
        const int64_t krow = kvrows[r];
        const int64_t bkv = krow / N, nk = krow % N;
        const int64_t b = bkv / Hkv, hkv = bkv % Hkv;
        for (int hl = 0; hl < grp; ++hl) {
            const int64_t bh = b * Hq + hkv * grp + hl;
            for (int64_t n = 0; n < N; ++n) {
                const int64_t row = bh * N + n;
                for (int32_t e = row_ptr[row]; e < row_ptr[row + 1]; ++e) {
                    if (col_idx[e] != nk) continue;
                    if (npairs == cap) {
                        cap *= 2;
                        pr = (int64_t*)realloc(pr, sizeof(int64_t) * 3 * (size_t)cap);
                    }
                    pr[3 * npairs + 0] = r;
                    pr[3 * npairs + 1] = row;
                    pr[3 * npairs + 2] = e - row_ptr[row];
                    ++npairs;
                }
            }
        }
    }
    double* ck = (double*)calloc((size_t)(npairs > 0 ? npairs : 1) * (size_t)BD, sizeof(double));
    double* cv = (double*)calloc((size_t)(npairs > 0 ? npairs : 1) * (size_t)BD, sizeof(double));

    /* 2. contribution of each pair */
#pragma omp parallel
    {
        double* p = (double*)malloc(sizeof(double) * (size_t)L);
        double* o = (double*)malloc(sizeof(double) * (size_t)D);
#pragma omp for schedule(dynamic, 1)
        for (int64_t i = 0; i < npairs; ++i) {
            const int64_t r = pr[3 * i], row = pr[3 * i + 1];
            const int pos = (int)pr[3 * i + 2];
            const int64_t krow = kvrows[r];
            const int64_t bkv = krow / N, nk = krow % N;
            const float* K = k + bkv * L * D;
            const float* V = v + bkv * L * D;
            const int64_t bh = row / N, n = row % N;
            const int32_t* sel = col_idx + row_ptr[row];
            const int nsel = row_ptr[row + 1] - row_ptr[row];
            double* gk = ck + i * BD;
            double* gv = cv + i * BD;
            for (int t = 0; t < B; ++t) {
                const int64_t tok = bh * L + n * B + t;
                const float* qv = q + tok * D;
                const float* dov = dout + tok * D;
                if (!vo_token_real(geom, n, t)) continue;   /* padding query: no contribution */
                token_forward(qv, K, V, D, B, sel, nsel, scale, p, o, geom);
                double delta = 0.0;
                for (int d = 0; d < D; ++d) delta += (double)dov[d] * o[d];
                for (int u = 0; u < B; ++u) {
                    const int64_t j = nk * B + u;
                    const double pj = p[pos * B + u];
                    double dp = 0.0;
                    for (int d = 0; d < D; ++d) dp += (double)dov[d] * (double)V[j * D + d];
                    const double ds = pj * (dp - delta);
                    for (int d = 0; d < D; ++d) {
                        gv[u * D + d] += pj * (double)dov[d];
                        gk[u * D + d] += scale * ds * (double)qv[d];
                    }
                }
            }
        }
        free(p);
        free(o);
    }

    /* 3. sum per key block, in pair order */
    for (int64_t i = 0; i < nkv * BD; ++i) { dk[i] = 0.0; dv[i] = 0.0; }
    for (int64_t i = 0; i < npairs; ++i) {
        const int64_t r = pr[3 * i];
        for (int64_t x = 0; x < BD; ++x) {
            dk[r * BD + x] += ck[i * BD + x];
            dv[r * BD + x] += cv[i * BD + x];
        }
    }
    free(ck);
    free(cv);
    free(pr);
}

/* ---------------------------------------------------------------------- */
/* Coarse branch (Sec. 2.2 "Coarse Branch", Eq. compress and the two       */
/* equations after it): dense softmax attention among the N cube means of  */
/* a head, P_c = Softmax(Q_c K_c^T / sqrt(D)), O_c_hat = P_c V_c; Repeat_B */
/* then broadcasts row n to the B tokens of cube n (done by the merge).    */
/* ---------------------------------------------------------------------- */

/* qc: [nb][Hq][N][D]; kc, vc: [nb][Hkv][N][D] (MeanPool_B outputs, float).
 * oc: [nb][Hq][N][D], lse: [nb][Hq][N] natural-log log-sum-exp of each row's
 * scaled scores.  Query head h reads KV head h / (Hq/Hkv). */
void vo_coarse_fwd(const float* qc, const float* kc, const float* vc, int nb, int Hq, int Hkv,
                   int N, int D, double* oc, double* lse)
{
    const int grp = Hq / Hkv;
    const double scale = 1.0 / sqrt((double)D);
    const int64_t nrows = (int64_t)nb * Hq * N;
#pragma omp parallel
    {
        double* s = (double*)malloc(sizeof(double) * (size_t)N);
#pragma omp for schedule(static)
        for (int64_t row = 0; row < nrows; ++row) {
            const int64_t bh = row / N;
            const int64_t b = bh / Hq, h = bh % Hq;
            const int64_t kv = b * Hkv + h / grp;
            const float* qv = qc + row * D;
            double m = -INFINITY;
            for (int j = 0; j < N; ++j) {
                const float* kj = kc + (kv * N + j) * (int64_t)D;
                double dot = 0.0;
                for (int d = 0; d < D; ++d) dot += (double)qv[d] * (double)kj[d];
                s[j] = dot * scale;
                if (s[j] > m) m = s[j];
            }
            double sum = 0.0;
            for (int j = 0; j < N; ++j) { s[j] = exp(s[j] - m); sum += s[j]; }
            double* o = oc + row * D;
            for (int d = 0; d < D; ++d) o[d] = 0.0;
            for (int j = 0; j < N; ++j) {
                const double pj = s[j] / sum;
                const float* vj = vc + (kv * N + j) * (int64_t)D;
                for (int d = 0; d < D; ++d) o[d] += pj * (double)vj[d];
            }
            lse[row] = m + log(sum);
        }
        free(s);
    }
}

/* Gradients of vo_coarse_fwd for the output gradient doc ([nb][Hq][N][D]):
 * with p the softmax row of coarse query i,
 *   Delta_i = doc_i . oc_i,  dS_ij = p_ij (doc_i . vc_j - Delta_i),
 *   dqc_i = scale sum_j dS_ij kc_j,  dkc_j = scale sum_i dS_ij qc_i,
 *   dvc_j = sum_i p_ij doc_i,
 * the sums over i running over every query head of j's KV group.  One task
 * per (batch, KV head) owns its dkc / dvc rows. */
void vo_coarse_bwd(const float* qc, const float* kc, const float* vc, const float* doc, int nb,
                   int Hq, int Hkv, int N, int D, double* dqc, double* dkc, double* dvc)
{
    const int grp = Hq / Hkv;
    const double scale = 1.0 / sqrt((double)D);
    const int64_t nkv = (int64_t)nb * Hkv;
#pragma omp parallel
    {
        double* p = (double*)malloc(sizeof(double) * (size_t)N);
        double* o = (double*)malloc(sizeof(double) * (size_t)D);
#pragma omp for schedule(dynamic, 1)
        for (int64_t kv = 0; kv < nkv; ++kv) {
            const int64_t b = kv / Hkv, hkv = kv % Hkv;
            double* gk = dkc + kv * N * (int64_t)D;
            double* gv = dvc + kv * N * (int64_t)D;
            for (int64_t x = 0; x < (int64_t)N * D; ++x) { gk[x] = 0.0; gv[x] = 0.0; }
            for (int hl = 0; hl < grp; ++hl) {
                const int64_t bh = b * Hq + hkv * grp + hl;
                for (int i = 0; i < N; ++i) {
                    const int64_t row = bh * N + i;
                    const float* qv = qc + row * D;
                    const float* dov = doc + row * D;
                    double m = -INFINITY;
                    for (int j = 0; j < N; ++j) {
                        const float* kj = kc + (kv * N + j) * (int64_t)D;
                        double dot = 0.0;
                        for (int d = 0; d < D; ++d) dot += (double)qv[d] * (double)kj[d];
                        p[j] = dot * scale;
                        if (p[j] > m) m = p[j];
                    }
                    double sum = 0.0;
                    for (int j = 0; j < N; ++j) { p[j] = exp(p[j] - m); sum += p[j]; }
                    for (int j = 0; j < N; ++j) p[j] /= sum;
                    for (int d = 0; d < D; ++d) o[d] = 0.0;
                    for (int j = 0; j < N; ++j)
                        for (int d = 0; d < D; ++d) o[d] += p[j] * (double)vc[(kv * N + j) * (int64_t)D + d];
                    double delta = 0.0;
                    for (int d = 0; d < D; ++d) delta += (double)dov[d] * o[d];
                    double* gq = dqc + row * D;
                    for (int d = 0; d < D; ++d) gq[d] = 0.0;
                    for (int j = 0; j < N; ++j) {
                        const float* kj = kc + (kv * N + j) * (int64_t)D;
                        const float* vj = vc + (kv * N + j) * (int64_t)D;
                        double dp = 0.0;
                        for (int d = 0; d < D; ++d) dp += (double)dov[d] * (double)vj[d];
                        const double ds = p[j] * (dp - delta);
                        for (int d = 0; d < D; ++d) {
                            gq[d] += scale * ds * (double)kj[d];
                            gk[(int64_t)j * D + d] += scale * ds * (double)qv[d];
                            gv[(int64_t)j * D + d] += p[j] * (double)dov[d];
                        }
                    }
                }
            }
        }
        free(p);
        free(o);
    }
}

/* ---------------------------------------------------------------------- */
/* Gated merge (Sec. 2.2 "Gated Merge", Eq. gate_linear and the merge      */
/* after it): G = tanh(X W_g), one gate per token and head; O = G * O_c +  */
/* O_f with O_c = Repeat_B(O_c_hat).  g holds the pre-activations X W_g.   */
/* ---------------------------------------------------------------------- */

/* g: [nbh][L]; oc: [nbh][N][D]; of, out: [nbh][L][D]; token l is in cube l / B. */
void vo_gate_merge(const float* g, const float* oc, const float* of, int64_t nbh, int N, int B,
                   int D, double* out)
{
    const int64_t L = (int64_t)N * B;
#pragma omp parallel for schedule(static)
    for (int64_t bh = 0; bh < nbh; ++bh)
        for (int64_t l = 0; l < L; ++l) {
            const double gate = tanh((double)g[bh * L + l]);
            const float* c = oc + (bh * N + l / B) * (int64_t)D;
            const float* f = of + (bh * L + l) * (int64_t)D;
            double* o = out + (bh * L + l) * (int64_t)D;
            for (int d = 0; d < D; ++d) o[d] = gate * (double)c[d] + (double)f[d];
        }
}

/* Gradients of vo_gate_merge for dout ([nbh][L][D]):
 *   doc[n] = sum over the B tokens l of cube n of tanh(g_l) dout_l,
 *   dg_l = (1 - tanh(g_l)^2) (dout_l . oc[n(l)]);  d(O_f) = dout.
 * Padding tokens of a padded grid are not outputs: they add nothing and get
 * dg = 0. */
void vo_gate_merge_bwd(const float* g, const float* oc, const float* dout, int64_t nbh, int N,
                       int B, int D, double* doc, double* dg, const int* geom)
{
    const int64_t L = (int64_t)N * B;
#pragma omp parallel for schedule(static)
    for (int64_t bh = 0; bh < nbh; ++bh)
        for (int64_t n = 0; n < N; ++n) {
            double* dc = doc + (bh * N + n) * (int64_t)D;
            const float* c = oc + (bh * N + n) * (int64_t)D;
            for (int d = 0; d < D; ++d) dc[d] = 0.0;
            for (int t = 0; t < B; ++t) {
                const int64_t l = n * B + t;
                if (!vo_token_real(geom, n, t)) {       /* padding token: not an output */
                    dg[bh * L + l] = 0.0;
                    continue;
                }
                const double gate = tanh((double)g[bh * L + l]);
                const float* dl = dout + (bh * L + l) * (int64_t)D;
                double dot = 0.0;
                for (int d = 0; d < D; ++d) {
                    dc[d] += gate * (double)dl[d];
                    dot += (double)dl[d] * (double)c[d];
                }
                dg[bh * L + l] = (1.0 - gate * gate) * dot;
            }
        }
}

/* The adjoint of vo_pool (the gradient of MeanPool over (Pt, Ph, Pw)):
 * every real token of sub-cube (n, g) receives dxc[n*Gp + g] / (number of
 * real tokens of the sub-cube), added to dx; padding tokens receive nothing.
 * dxc: [nbh][N*Gp][D]; dx: [nbh][N*B][D]. */
void vo_unpool_add(const double* dxc, int64_t nbh, int T, int H, int W, int Bt, int Bh, int Bw,
                   int Pt, int Ph, int Pw, int D, double* dx)
{
    const int geom[7] = {T, H, W, Bt, Bh, Bw, 0};
    const int64_t N = ceil_div(T, Bt) * ceil_div(H, Bh) * ceil_div(W, Bw);
    const int B = Bt * Bh * Bw;
    const int Gt = Bt / Pt, Gh = Bh / Ph, Gw = Bw / Pw;
    const int G = Gt * Gh * Gw;
#pragma omp parallel for schedule(static)
    for (int64_t bh = 0; bh < nbh; ++bh)
        for (int64_t n = 0; n < N; ++n)
            for (int bt = 0; bt < Bt; ++bt)
            for (int bhh = 0; bhh < Bh; ++bhh)
            for (int bw = 0; bw < Bw; ++bw) {
                const int g = ((bt / Pt) * Gh + bhh / Ph) * Gw + bw / Pw;
                const int beta = (bt * Bh + bhh) * Bw + bw;
                if (!vo_token_real(geom, n, beta)) continue;
                const double cnt = (double)vo_subcube_real_count(geom, n, g, Pt, Ph, Pw);
                const double* src = dxc + ((bh * N + n) * G + g) * (int64_t)D;
                double* dst = dx + ((bh * N + n) * B + beta) * (int64_t)D;
                for (int d = 0; d < D; ++d) dst[d] += src[d] / cnt;
            }
}
