/*
 * Memory-safety driver for the CPU oracle (test infrastructure only).
 *
 * Calls every function of vsa2_oracle.c on small problems -- a divisible
 * grid, a padded grid, a padded grid with text tokens, bf16 and fp32
 * rounding, GQA, top-k / mass / per-sequence selection, block lists with
 * empty rows -- with every buffer malloc'ed at exactly the size the
 * function's contract gives, so that a build with AddressSanitizer and
 * UndefinedBehaviorSanitizer reports any read or write outside them.  It
 * prints one checksum line per call; the test compares the sanitized
 * build's lines with those of a plain build of the same sources.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

void vo_round_bf16(const double* in, float* out, int64_t n);
void vo_pool(const float* x, int64_t nbh, int T, int H, int W, int Bt, int Bh, int Bw, int Pt, int Ph, int Pw,
             int D, int dtype_bf16, float* out);
void vo_router_scores(const float* q_r, const float* k_r, int nb, int Hq, int Hkv, int64_t N, int G, int D,
                      const int64_t* rows, int64_t nrows, double* scores, double* lse_out, const int* geom, int Rt,
                      int Rh, int Rw);
void vo_select_rows(const double* scores, int64_t nrows, int N, int mode, int k, double mass, int cap,
                    int32_t* counts, int32_t* idx);
void vo_select_seq(const double* scores, int64_t nseq, int N, int k, uint8_t* sel);
void vo_attn_fwd(const float* q, const float* k, const float* v, int nb, int Hq, int Hkv, int64_t L, int D, int B,
                 const int32_t* row_ptr, const int32_t* col_idx, const int64_t* qrows, int64_t nq, double* o,
                 double* lse, const int* geom);
void vo_attn_bwd_dq(const float* q, const float* k, const float* v, const float* dout, int nb, int Hq, int Hkv,
                    int64_t L, int D, int B, const int32_t* row_ptr, const int32_t* col_idx, const int64_t* qrows,
                    int64_t nq, double* dq, const int* geom);
void vo_attn_bwd_dkdv(const float* q, const float* k, const float* v, const float* dout, int nb, int Hq, int Hkv,
                      int64_t L, int D, int B, const int32_t* row_ptr, const int32_t* col_idx,
                      const int64_t* kvrows, int64_t nkv, double* dk, double* dv, const int* geom);
void vo_coarse_fwd(const float* qc, const float* kc, const float* vc, int nb, int Hq, int Hkv, int N, int D,
                   double* oc, double* lse);
void vo_coarse_bwd(const float* qc, const float* kc, const float* vc, const float* doc, int nb, int Hq, int Hkv,
                   int N, int D, double* dqc, double* dkc, double* dvc);
void vo_gate_merge(const float* g, const float* oc, const float* of, int64_t nbh, int N, int B, int D, double* out);
void vo_gate_merge_bwd(const float* g, const float* oc, const float* dout, int64_t nbh, int N, int B, int D,
                       double* doc, double* dg, const int* geom);
void vo_unpool_add(const double* dxc, int64_t nbh, int T, int H, int W, int Bt, int Bh, int Bw, int Pt, int Ph,
                   int Pw, int D, double* dx);

static uint64_t rng_state = 0x9e3779b97f4a7c15ull;

/* splitmix64 step, mapped to [-1, 1) */
static double urand(void)
{
    uint64_t z = (rng_state += 0x9e3779b97f4a7c15ull);
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
    z ^= z >> 31;
    return (double)(z >> 11) / 4503599627370496.0 - 1.0;
}

static void* xmalloc(size_t n)
{
    void* p = malloc(n ? n : 1);
    if (!p) {
        fprintf(stderr, "out of memory\n");
        exit(2);
    }
    return p;
}

static float* rand_f32(int64_t n, double scale)
{
    float* a = (float*)xmalloc(sizeof(float) * (size_t)n);
    for (int64_t i = 0; i < n; ++i) a[i] = (float)(scale * urand());
    return a;
}

static double sum_f64(const double* a, int64_t n)
{
    double s = 0.0;
    for (int64_t i = 0; i < n; ++i)
        if (isfinite(a[i])) s += a[i];
    return s;
}

static double sum_f32(const float* a, int64_t n)
{
    double s = 0.0;
    for (int64_t i = 0; i < n; ++i) s += a[i];
    return s;
}

/* CSR over nrows rows of nblk blocks: row r holds about `fill` of them
 * (ascending), every seventh row none. */
static void make_lists(int64_t nrows, int nblk, double fill, int32_t** rp_out, int32_t** ci_out)
{
    int32_t* rp = (int32_t*)xmalloc(sizeof(int32_t) * (size_t)(nrows + 1));
    int32_t* tmp = (int32_t*)xmalloc(sizeof(int32_t) * (size_t)(nrows * nblk));
    int64_t nnz = 0;
    rp[0] = 0;
    for (int64_t r = 0; r < nrows; ++r) {
        if (r % 7 != 3)
            for (int c = 0; c < nblk; ++c)
                if (urand() * 0.5 + 0.5 < fill) tmp[nnz++] = c;
        rp[r + 1] = (int32_t)nnz;
    }
    int32_t* ci = (int32_t*)xmalloc(sizeof(int32_t) * (size_t)nnz);
    memcpy(ci, tmp, sizeof(int32_t) * (size_t)nnz);
    free(tmp);
    *rp_out = rp;
    *ci_out = ci;
}

struct problem {
    const char* name;
    int nb, Hq, Hkv, D, T, H, W, text_len, bf16;
};

static void run(const struct problem* pr)
{
    const int Bt = 4, Bh = 4, Bw = 4, B = 64, Rt = 2, Rh = 2, Rw = 2, G = 8;
    const int Nt = (pr->T + Bt - 1) / Bt, Nh = (pr->H + Bh - 1) / Bh, Nw = (pr->W + Bw - 1) / Bw;
    const int N = Nt * Nh * Nw;
    const int M = (pr->text_len + B - 1) / B;
    const int Nj = N + M;
    const int64_t L = (int64_t)N * B, Lj = (int64_t)Nj * B;
    const int D = pr->D, nb = pr->nb, Hq = pr->Hq, Hkv = pr->Hkv;
    const int geom[7] = {pr->T, pr->H, pr->W, Bt, Bh, Bw, pr->text_len};
    const int64_t nq_rows = (int64_t)nb * Hq * N, nkv_rows = (int64_t)nb * Hkv * N;

    /* rounding */
    {
        const int64_t n = 257;
        double* in = (double*)xmalloc(sizeof(double) * n);
        float* out = (float*)xmalloc(sizeof(float) * n);
        for (int64_t i = 0; i < n; ++i) in[i] = 40.0 * urand();
        vo_round_bf16(in, out, n);
        printf("%s round %.17g\n", pr->name, sum_f32(out, n));
        free(in);
        free(out);
    }

    /* pooling (video tokens) and the router */
    float* qv = rand_f32((int64_t)nb * Hq * L * D, 2.0);
    float* kv = rand_f32((int64_t)nb * Hkv * L * D, 2.0);
    float* q_r = (float*)xmalloc(sizeof(float) * (size_t)(nb * Hq * (int64_t)N * G * D));
    float* k_r = (float*)xmalloc(sizeof(float) * (size_t)(nb * Hkv * (int64_t)N * G * D));
    vo_pool(qv, (int64_t)nb * Hq, pr->T, pr->H, pr->W, Bt, Bh, Bw, Rt, Rh, Rw, D, pr->bf16, q_r);
    vo_pool(kv, (int64_t)nb * Hkv, pr->T, pr->H, pr->W, Bt, Bh, Bw, Rt, Rh, Rw, D, pr->bf16, k_r);
    printf("%s pool %.17g %.17g\n", pr->name, sum_f32(q_r, nb * Hq * (int64_t)N * G * D),
           sum_f32(k_r, nb * Hkv * (int64_t)N * G * D));
    int64_t* rows = (int64_t*)xmalloc(sizeof(int64_t) * (size_t)nq_rows);
    for (int64_t r = 0; r < nq_rows; ++r) rows[r] = r;
    double* scores = (double*)xmalloc(sizeof(double) * (size_t)(nq_rows * N));
    double* lse_r = (double*)xmalloc(sizeof(double) * (size_t)(nq_rows * G));
    vo_router_scores(q_r, k_r, nb, Hq, Hkv, N, G, D, rows, nq_rows, scores, lse_r, geom, Rt, Rh, Rw);
    printf("%s router %.17g %.17g\n", pr->name, sum_f64(scores, nq_rows * N), sum_f64(lse_r, nq_rows * G));

    /* selection: top-k, mass with cap, per-sequence */
    int32_t* counts = (int32_t*)xmalloc(sizeof(int32_t) * (size_t)nq_rows);
    int32_t* idx = (int32_t*)xmalloc(sizeof(int32_t) * (size_t)(nq_rows * N));
    for (int mode = 0; mode < 2; ++mode) {
        vo_select_rows(scores, nq_rows, N, mode, 3, 0.7, 4, counts, idx);
        int64_t tot = 0, isum = 0;
        for (int64_t r = 0; r < nq_rows; ++r) {
            tot += counts[r];
            for (int i = 0; i < counts[r]; ++i) isum += idx[r * N + i];
        }
        printf("%s select%d %lld %lld\n", pr->name, mode, (long long)tot, (long long)isum);
    }
    uint8_t* sel = (uint8_t*)xmalloc((size_t)(nb * Hq * (int64_t)N * N));
    vo_select_seq(scores, (int64_t)nb * Hq, N, 2, sel);
    int64_t nsel = 0;
    for (int64_t i = 0; i < (int64_t)nb * Hq * N * N; ++i) nsel += sel[i];
    printf("%s select_seq %lld\n", pr->name, (long long)nsel);

    /* attention over the joint sequence (video, then text blocks) */
    const int64_t nqj = (int64_t)nb * Hq * Nj, nkvj = (int64_t)nb * Hkv * Nj;
    float* q = rand_f32((int64_t)nb * Hq * Lj * D, 1.5);
    float* k = rand_f32((int64_t)nb * Hkv * Lj * D, 1.5);
    float* v = rand_f32((int64_t)nb * Hkv * Lj * D, 1.5);
    float* dout = rand_f32((int64_t)nb * Hq * Lj * D, 1.0);
    int32_t *rp, *ci;
    make_lists(nqj, Nj, 0.4, &rp, &ci);
    int64_t* qrows = (int64_t*)xmalloc(sizeof(int64_t) * (size_t)nqj);
    for (int64_t r = 0; r < nqj; ++r) qrows[r] = r;
    int64_t* kvrows = (int64_t*)xmalloc(sizeof(int64_t) * (size_t)nkvj);
    for (int64_t r = 0; r < nkvj; ++r) kvrows[r] = r;
    double* o = (double*)xmalloc(sizeof(double) * (size_t)(nqj * B * D));
    double* lse = (double*)xmalloc(sizeof(double) * (size_t)(nqj * B));
    double* dq = (double*)xmalloc(sizeof(double) * (size_t)(nqj * B * D));
    double* dk = (double*)xmalloc(sizeof(double) * (size_t)(nkvj * B * D));
    double* dv = (double*)xmalloc(sizeof(double) * (size_t)(nkvj * B * D));
    vo_attn_fwd(q, k, v, nb, Hq, Hkv, Lj, D, B, rp, ci, qrows, nqj, o, lse, geom);
    vo_attn_bwd_dq(q, k, v, dout, nb, Hq, Hkv, Lj, D, B, rp, ci, qrows, nqj, dq, geom);
    vo_attn_bwd_dkdv(q, k, v, dout, nb, Hq, Hkv, Lj, D, B, rp, ci, kvrows, nkvj, dk, dv, geom);
    printf("%s attn %.17g %.17g %.17g %.17g %.17g\n", pr->name, sum_f64(o, nqj * B * D), sum_f64(lse, nqj * B),
           sum_f64(dq, nqj * B * D), sum_f64(dk, nkvj * B * D), sum_f64(dv, nkvj * B * D));

    /* coarse branch (cube means), gated merge, MeanPool adjoint */
    float* qc = (float*)xmalloc(sizeof(float) * (size_t)(nq_rows * D));
    float* kc = (float*)xmalloc(sizeof(float) * (size_t)(nkv_rows * D));
    float* vc = (float*)xmalloc(sizeof(float) * (size_t)(nkv_rows * D));
    float* vvid = rand_f32((int64_t)nb * Hkv * L * D, 2.0);
    vo_pool(qv, (int64_t)nb * Hq, pr->T, pr->H, pr->W, Bt, Bh, Bw, Bt, Bh, Bw, D, pr->bf16, qc);
    vo_pool(kv, (int64_t)nb * Hkv, pr->T, pr->H, pr->W, Bt, Bh, Bw, Bt, Bh, Bw, D, pr->bf16, kc);
    vo_pool(vvid, (int64_t)nb * Hkv, pr->T, pr->H, pr->W, Bt, Bh, Bw, Bt, Bh, Bw, D, pr->bf16, vc);
    double* oc = (double*)xmalloc(sizeof(double) * (size_t)(nq_rows * D));
    double* lsec = (double*)xmalloc(sizeof(double) * (size_t)nq_rows);
    vo_coarse_fwd(qc, kc, vc, nb, Hq, Hkv, N, D, oc, lsec);
    float* doc_in = rand_f32(nq_rows * D, 1.0);
    double* dqc = (double*)xmalloc(sizeof(double) * (size_t)(nq_rows * D));
    double* dkc = (double*)xmalloc(sizeof(double) * (size_t)(nkv_rows * D));
    double* dvc = (double*)xmalloc(sizeof(double) * (size_t)(nkv_rows * D));
    vo_coarse_bwd(qc, kc, vc, doc_in, nb, Hq, Hkv, N, D, dqc, dkc, dvc);
    printf("%s coarse %.17g %.17g %.17g %.17g %.17g\n", pr->name, sum_f64(oc, nq_rows * D), sum_f64(lsec, nq_rows),
           sum_f64(dqc, nq_rows * D), sum_f64(dkc, nkv_rows * D), sum_f64(dvc, nkv_rows * D));
    const int64_t nbh = (int64_t)nb * Hq;
    float* g = rand_f32(nbh * L, 2.0);
    float* ocf = rand_f32(nbh * N * D, 1.0);
    float* of = rand_f32(nbh * L * D, 1.0);
    float* dov = rand_f32(nbh * L * D, 1.0);
    double* merged = (double*)xmalloc(sizeof(double) * (size_t)(nbh * L * D));
    vo_gate_merge(g, ocf, of, nbh, N, B, D, merged);
    double* doc = (double*)xmalloc(sizeof(double) * (size_t)(nbh * N * D));
    double* dg = (double*)xmalloc(sizeof(double) * (size_t)(nbh * L));
    vo_gate_merge_bwd(g, ocf, dov, nbh, N, B, D, doc, dg, geom);
    printf("%s merge %.17g %.17g %.17g\n", pr->name, sum_f64(merged, nbh * L * D), sum_f64(doc, nbh * N * D),
           sum_f64(dg, nbh * L));
    double* dxc = (double*)xmalloc(sizeof(double) * (size_t)(nbh * N * G * D));
    for (int64_t i = 0; i < nbh * N * G * D; ++i) dxc[i] = urand();
    double* dx = (double*)xmalloc(sizeof(double) * (size_t)(nbh * L * D));
    for (int64_t i = 0; i < nbh * L * D; ++i) dx[i] = urand();
    vo_unpool_add(dxc, nbh, pr->T, pr->H, pr->W, Bt, Bh, Bw, Rt, Rh, Rw, D, dx);
    printf("%s unpool %.17g\n", pr->name, sum_f64(dx, nbh * L * D));

    free(qv); free(kv); free(q_r); free(k_r); free(rows); free(scores); free(lse_r); free(counts); free(idx);
    free(sel); free(q); free(k); free(v); free(dout); free(rp); free(ci); free(qrows); free(kvrows); free(o);
    free(lse); free(dq); free(dk); free(dv); free(qc); free(kc); free(vc); free(vvid); free(oc); free(lsec);
    free(doc_in); free(dqc); free(dkc); free(dvc); free(g); free(ocf); free(of); free(dov); free(merged);
    free(doc); free(dg); free(dxc); free(dx);
}

int main(void)
{
    static const struct problem cases[] = {
        {"divisible-bf16-gqa", 1, 4, 2, 16, 8, 8, 8, 0, 1},
        {"padded-f32", 2, 2, 2, 8, 5, 6, 7, 0, 0},
        {"padded-text-bf16", 1, 2, 1, 8, 3, 5, 9, 70, 1},
    };
    for (size_t i = 0; i < sizeof(cases) / sizeof(cases[0]); ++i) run(&cases[i]);
    printf("done\n");
    return 0;
}
