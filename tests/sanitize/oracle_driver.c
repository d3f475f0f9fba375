/*
 * Host-code check of the input generator and the CPU oracle under
 * AddressSanitizer and UndefinedBehaviorSanitizer (built by
 * tests/test_sanitizers.py with -fsanitize=address,undefined and
 * -fno-sanitize-recover, without OpenMP).  Small graphs that reach every
 * generator and every oracle function, including empty rows, repeated
 * entries, a single row, requested-row subsets and bf16 inputs; only the
 * return codes are checked here (the values are pinned by the other tests).
 * Exit status 0 when every call returned what it should.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

void synth_normal(uint64_t seed, uint32_t stream, double std, int64_t n, float* out_f32, uint16_t* out_bf16);
void synth_uniform01(uint64_t seed, uint32_t stream, int64_t n, double* out);
int synth_distinct_sources(uint64_t seed, uint32_t stream, int64_t N, const int64_t* rowptr, int32_t* colidx,
                           int add_self);
int64_t synth_rmat(uint64_t seed, uint32_t stream, int scale, double a, double b, double c, int64_t target,
                   int64_t max_samples, int32_t* src, int32_t* dst);
void synth_csr_from_pairs(int64_t N, int64_t n, const int32_t* dst, const int32_t* src, int add_self,
                          int64_t* rowptr, int32_t* colidx);
void synth_sbm(uint64_t seed, uint32_t stream, int64_t N, int64_t bs, int64_t n_out, int64_t* rowptr,
               int32_t* colidx);

int gt_oracle_fwd(int dtype, const int64_t* rowptr, const int32_t* colidx, const void* Q, const void* K,
                  const void* V, int64_t N, int64_t E, int32_t H, int32_t D, float scale, const int64_t* rows,
                  int64_t nrows, double* out, double* absagg, double* lse);
int gt_oracle_bwd_dq(int dtype, const int64_t* rowptr, const int32_t* colidx, const void* Q, const void* K,
                     const void* V, const void* dO, int64_t N, int64_t E, int32_t H, int32_t D, float scale,
                     const int64_t* rows, int64_t nrows, double* dQ, double* sdQ);
int gt_oracle_bwd_dkv(int dtype, const int64_t* rowptr, const int32_t* colidx, const int64_t* rowptr_t,
                      const int32_t* colidx_t, const void* Q, const void* K, const void* V, const void* dO,
                      int64_t N, int64_t E, int32_t H, int32_t D, float scale, const int64_t* cols, int64_t ncols,
                      double* dK, double* dV, double* sdK, double* sdV);
int gt_oracle_gatv2_fwd(int dtype, const int64_t* rowptr, const int32_t* colidx, const void* Lf, const void* Rf,
                        const float* att, int64_t N, int64_t E, int32_t H, int32_t D, float slope,
                        const int64_t* rows, int64_t nrows, double* out, double* absagg, double* lse);
int gt_oracle_segment_reduce(int dtype, int op, const int64_t* rowptr, const int32_t* colidx, const void* X,
                             int64_t N, int64_t E, int32_t F, const int64_t* rows, int64_t nrows, float* out,
                             int32_t* arg);
int gt_oracle_dot_aggr(const int64_t* rowptr, const int32_t* colidx, const float* X, int64_t N, int64_t E,
                       int32_t F, const int64_t* rows, int64_t nrows, double* out, double* absout);

static int failures = 0;
#define EXPECT(cond)                                                   \
    do {                                                               \
        if (!(cond)) {                                                 \
            fprintf(stderr, "%s:%d: %s\n", __FILE__, __LINE__, #cond); \
            ++failures;                                                \
        }                                                              \
    } while (0)

/* transposed structure: row j lists every destination whose row holds j */
static void transpose(int64_t N, const int64_t* rp, const int32_t* ci, int64_t* rpt, int32_t* cit) {
    int64_t E = rp[N];
    memset(rpt, 0, (size_t)(N + 1) * sizeof(int64_t));
    for (int64_t e = 0; e < E; ++e) rpt[ci[e] + 1]++;
    for (int64_t i = 0; i < N; ++i) rpt[i + 1] += rpt[i];
    int64_t* fill = (int64_t*)malloc((size_t)(N > 0 ? N : 1) * sizeof(int64_t));
    for (int64_t i = 0; i < N; ++i) fill[i] = rpt[i];
    for (int64_t i = 0; i < N; ++i)
        for (int64_t e = rp[i]; e < rp[i + 1]; ++e) cit[fill[ci[e]]++] = (int32_t)i;
    free(fill);
}

/* every oracle function on one graph, fp32 and bf16, all rows and a subset */
static void run_all(int64_t N, const int64_t* rp, const int32_t* ci, int32_t H, int32_t D) {
    /* outputs sized for max(N, 3) rows: the subset calls ask for three */
    const int64_t E = rp[N], n = (N > 3 ? N : 3) * H * D;
    float* f = (float*)malloc((size_t)(4 * n + 1) * sizeof(float));
    uint16_t* b = (uint16_t*)malloc((size_t)(4 * n + 1) * sizeof(uint16_t));
    synth_normal(1, 2, 1.0, 4 * n, f, b);
    float* att = (float*)malloc((size_t)(H * D) * sizeof(float));
    synth_normal(1, 9, 0.2, H * D, att, NULL);
    double* o1 = (double*)malloc((size_t)(n + 1) * sizeof(double));
    double* o2 = (double*)malloc((size_t)(n + 1) * sizeof(double));
    double* o3 = (double*)malloc((size_t)(n + 1) * sizeof(double));
    double* o4 = (double*)malloc((size_t)(n + 1) * sizeof(double));
    double* l = (double*)malloc((size_t)((N > 3 ? N : 3) * H + 1) * sizeof(double));
    float* rf = (float*)malloc((size_t)(n + 1) * sizeof(float));
    int32_t* ra = (int32_t*)malloc((size_t)(n + 1) * sizeof(int32_t));
    int64_t* rpt = (int64_t*)malloc((size_t)(N + 1) * sizeof(int64_t));
    int32_t* cit = (int32_t*)malloc((size_t)(E + 1) * sizeof(int32_t));
    transpose(N, rp, ci, rpt, cit);
    const int64_t rows[3] = {N - 1, 0, N / 2};
    for (int dt = 0; dt < 2; ++dt) {
        const void* Q = dt ? (const void*)b : (const void*)f;
        const void* K = dt ? (const void*)(b + n) : (const void*)(f + n);
        const void* V = dt ? (const void*)(b + 2 * n) : (const void*)(f + 2 * n);
        const void* dO = dt ? (const void*)(b + 3 * n) : (const void*)(f + 3 * n);
        EXPECT(gt_oracle_fwd(dt, rp, ci, Q, K, V, N, E, H, D, 0.17f, NULL, N, o1, o2, l) == 0);
        EXPECT(gt_oracle_fwd(dt, rp, ci, Q, K, V, N, E, H, D, 0.17f, rows, 3, o1, NULL, NULL) == 0);
        EXPECT(gt_oracle_bwd_dq(dt, rp, ci, Q, K, V, dO, N, E, H, D, 0.17f, NULL, N, o1, o2) == 0);
        EXPECT(gt_oracle_bwd_dkv(dt, rp, ci, rpt, cit, Q, K, V, dO, N, E, H, D, 0.17f, rows, 3, o1, o2, o3, o4) == 0);
        EXPECT(gt_oracle_gatv2_fwd(dt, rp, ci, Q, K, att, N, E, H, D, 0.2f, NULL, N, o1, o2, l) == 0);
        for (int op = 0; op < 2; ++op) {
            EXPECT(gt_oracle_segment_reduce(dt, op, rp, ci, Q, N, E, H * D, NULL, N, rf, ra) == 0);
            EXPECT(gt_oracle_segment_reduce(dt, op, rp, ci, Q, N, E, H * D, rows, 3, rf, ra) == 0);
        }
    }
    EXPECT(gt_oracle_dot_aggr(rp, ci, f, N, E, H * D, NULL, N, o1, o2) == 0);
    /* invalid arguments are refused, not read */
    EXPECT(gt_oracle_fwd(2, rp, ci, f, f, f, N, E, H, D, 0.1f, NULL, N, o1, NULL, NULL) == 1);
    EXPECT(gt_oracle_fwd(0, rp, ci, f, f, f, N, E, 0, D, 0.1f, NULL, N, o1, NULL, NULL) == 1);
    const int64_t bad_row[1] = {N};
    EXPECT(gt_oracle_fwd(0, rp, ci, f, f, f, N, E, H, D, 0.1f, bad_row, 1, o1, NULL, NULL) == 2);
    free(f); free(b); free(att); free(o1); free(o2); free(o3); free(o4); free(l); free(rf); free(ra);
    free(rpt); free(cit);
}

int main(void) {
    /* uniform degrees with self-loops; some empty rows (no self-loop) */
    {
        const int64_t N = 97;
        int64_t* rp = (int64_t*)malloc((N + 1) * sizeof(int64_t));
        rp[0] = 0;
        for (int64_t i = 0; i < N; ++i) rp[i + 1] = rp[i] + (i % 7 == 3 ? 0 : 1 + (i * 13) % 11);
        int32_t* ci = (int32_t*)malloc((size_t)rp[N] * sizeof(int32_t));
        EXPECT(synth_distinct_sources(3, 1, N, rp, ci, 0) == 0);
        run_all(N, rp, ci, 2, 32);
        free(rp); free(ci);
    }
    /* R-MAT pairs into CSR with self-loops */
    {
        const int scale = 8;
        const int64_t N = 1 << scale, target = 5 * N;
        int32_t* src = (int32_t*)malloc((size_t)target * sizeof(int32_t));
        int32_t* dst = (int32_t*)malloc((size_t)target * sizeof(int32_t));
        EXPECT(synth_rmat(0, 1, scale, 0.57, 0.19, 0.19, target, 8 * target, src, dst) >= target);
        int64_t* rp = (int64_t*)malloc((N + 1) * sizeof(int64_t));
        int32_t* ci = (int32_t*)malloc((size_t)(target + N) * sizeof(int32_t));
        synth_csr_from_pairs(N, target, dst, src, 1, rp, ci);
        run_all(N, rp, ci, 1, 32);
        free(src); free(dst); free(rp); free(ci);
    }
    /* block model with a partial last block; repeated entries; a single row */
    {
        const int64_t N = 64 * 3 + 5;
        int64_t* rp = (int64_t*)malloc((N + 1) * sizeof(int64_t));
        synth_sbm(0, 1, N, 64, 4, rp, NULL);
        int32_t* ci = (int32_t*)malloc((size_t)rp[N] * sizeof(int32_t));
        synth_sbm(0, 1, N, 64, 4, rp, ci);
        ci[1] = ci[0];
        run_all(N, rp, ci, 4, 32);
        const int64_t rp1[2] = {0, 3};
        const int32_t ci1[3] = {0, 0, 0};
        run_all(1, rp1, ci1, 1, 32);
        free(rp); free(ci);
    }
    double u[5];
    synth_uniform01(0, 7, 5, u);
    EXPECT(u[0] > 0.0 && u[0] < 1.0);
    printf("oracle driver: %d failure(s)\n", failures);
    return failures ? 1 : 0;
}
