/*
 * A standalone C caller of the library on the GPU, with no Python and no
 * torch: it allocates device memory with the HIP runtime, calls the contract
 * entry points (gt_attn_fwd, gt_attn_fwd_bf16, gt_attn_fwd_noalloc) on the
 * null stream and compares every output element with the float64 oracle
 * (oracle/gt_oracle.c, linked as test infrastructure).
 *
 * Input: a ragged graph of 3000 rows with a 2500-entry hub (split into
 * chunks) and some empty rows, sources distinct per row, drawn from a
 * 64-bit xorshift with a fixed seed; N(0, 1)-like features from the same
 * generator.  Gate: max |x - r| / max(|r|, sum_e alpha_e |v_e|) over all
 * elements, 1e-5 for fp32 and 2e-2 for bf16 features.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "gt_attn.h"

int gt_oracle_fwd(int dtype, const int64_t* rowptr, const int32_t* colidx, const void* Q, const void* K,
                  const void* V, int64_t N, int64_t E, int32_t H, int32_t D, float scale, const int64_t* rows,
                  int64_t nrows, double* out, double* absagg, double* lse);

static uint64_t rng_state = 0x9E3779B97F4A7C15ull;
static uint64_t next_u64(void) {
    rng_state ^= rng_state << 13;
    rng_state ^= rng_state >> 7;
    rng_state ^= rng_state << 17;
    return rng_state;
}
static double next_unit(void) { return (double)(next_u64() >> 11) * (1.0 / 9007199254740992.0); }
/* sum of four uniforms, centred and scaled to unit variance */
static float next_normalish(void) {
    double s = next_unit() + next_unit() + next_unit() + next_unit() - 2.0;
    return (float)(s * 1.7320508075688772);
}

static uint16_t to_bf16(float x) {
    uint32_t u;
    memcpy(&u, &x, 4);
    return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}
static float from_bf16(uint16_t b) {
    uint32_t u = (uint32_t)b << 16;
    float x;
    memcpy(&x, &u, 4);
    return x;
}

#define HIP_OK(call)                                                             \
    do {                                                                         \
        hipError_t e_ = (call);                                                  \
        if (e_ != hipSuccess) {                                                  \
            fprintf(stderr, "%s failed: %s\n", #call, hipGetErrorString(e_));    \
            exit(2);                                                             \
        }                                                                        \
    } while (0)

static double gate(const float* x, const double* ref, const double* absagg, size_t n) {
    double worst = 0.0;
    for (size_t i = 0; i < n; ++i) {
        double d = fabs(ref[i]) > absagg[i] ? fabs(ref[i]) : absagg[i];
        if (d < 1e-30) d = 1e-30;
        const double e = fabs((double)x[i] - ref[i]) / d;
        if (!(e <= worst)) worst = e; /* NaN propagates */
    }
    return worst;
}

int main(void) {
    const int64_t N = 3000;
    int64_t* rowptr = malloc((N + 1) * sizeof(int64_t));
    int64_t* deg = malloc(N * sizeof(int64_t));
    rowptr[0] = 0;
    for (int64_t i = 0; i < N; ++i) {
        deg[i] = (next_u64() % 10 == 0) ? 0 : (int64_t)(next_u64() % 60);
        if (i == 7) deg[i] = 2500;
        rowptr[i + 1] = rowptr[i] + deg[i];
    }
    const int64_t E = rowptr[N];
    int32_t* colidx = malloc((E > 0 ? E : 1) * sizeof(int32_t));
    unsigned char* seen = calloc((size_t)N, 1);
    for (int64_t i = 0; i < N; ++i) {
        for (int64_t t = 0; t < deg[i]; ++t) {
            int32_t j;
            do j = (int32_t)(next_u64() % (uint64_t)N); while (seen[j]);
            seen[j] = 1;
            colidx[rowptr[i] + t] = j;
        }
        for (int64_t t = 0; t < deg[i]; ++t) seen[colidx[rowptr[i] + t]] = 0;
    }

    int bad = 0;
    const int32_t shapes[2][2] = {{4, 32}, {2, 64}};
    for (int dt = 0; dt < 2; ++dt) {
        const int32_t H = shapes[dt][0], D = shapes[dt][1];
        const size_t n = (size_t)N * H * D, eb = dt == 0 ? 4 : 2;
        const float scale = 1.0f / sqrtf((float)D);
        void* host[3];
        for (int a = 0; a < 3; ++a) {
            host[a] = malloc(n * eb);
            for (size_t k = 0; k < n; ++k) {
                const float v = next_normalish();
                if (dt == 0)
                    ((float*)host[a])[k] = v;
                else
                    ((uint16_t*)host[a])[k] = to_bf16(v);
            }
        }
        int64_t* d_rowptr;
        int32_t* d_colidx;
        void *d_q, *d_k, *d_v, *d_out;
        HIP_OK(hipMalloc((void**)&d_rowptr, (N + 1) * sizeof(int64_t)));
        HIP_OK(hipMalloc((void**)&d_colidx, (E > 0 ? E : 1) * sizeof(int32_t)));
        HIP_OK(hipMalloc(&d_q, n * eb));
        HIP_OK(hipMalloc(&d_k, n * eb));
        HIP_OK(hipMalloc(&d_v, n * eb));
        HIP_OK(hipMalloc(&d_out, n * eb));
        HIP_OK(hipMemcpy(d_rowptr, rowptr, (N + 1) * sizeof(int64_t), hipMemcpyHostToDevice));
        HIP_OK(hipMemcpy(d_colidx, colidx, E * sizeof(int32_t), hipMemcpyHostToDevice));
        HIP_OK(hipMemcpy(d_q, host[0], n * eb, hipMemcpyHostToDevice));
        HIP_OK(hipMemcpy(d_k, host[1], n * eb, hipMemcpyHostToDevice));
        HIP_OK(hipMemcpy(d_v, host[2], n * eb, hipMemcpyHostToDevice));

        double* ref = malloc(n * sizeof(double));
        double* absagg = malloc(n * sizeof(double));
        if (gt_oracle_fwd(dt, rowptr, colidx, host[0], host[1], host[2], N, E, H, D, scale, NULL, N, ref, absagg,
                          NULL) != 0) {
            fprintf(stderr, "oracle failed\n");
            return 3;
        }
        void* got = malloc(n * eb);
        float* gotf = malloc(n * sizeof(float));
        const double tol = dt == 0 ? 1e-5 : 2e-2;
        for (int entry = 0; entry < 2; ++entry) {
            HIP_OK(hipMemset(d_out, 0xFF, n * eb));
            gt_status s;
            if (entry == 0)
                s = dt == 0 ? gt_attn_fwd(d_rowptr, d_colidx, d_q, d_k, d_v, d_out, N, E, H, D, scale, NULL)
                            : gt_attn_fwd_bf16(d_rowptr, d_colidx, d_q, d_k, d_v, d_out, N, E, H, D, scale, NULL);
            else
                s = gt_attn_fwd_noalloc(dt == 0 ? GT_DTYPE_F32 : GT_DTYPE_BF16, d_rowptr, d_colidx, d_q, d_k, d_v,
                                        d_out, NULL, N, E, H, D, scale, NULL, NULL);
            if (s != GT_SUCCESS) {
                fprintf(stderr, "call failed: %s: %s\n", gt_status_string(s), gt_last_error_message());
                return 4;
            }
            HIP_OK(hipDeviceSynchronize());
            HIP_OK(hipMemcpy(got, d_out, n * eb, hipMemcpyDeviceToHost));
            for (size_t k = 0; k < n; ++k)
                gotf[k] = dt == 0 ? ((float*)got)[k] : from_bf16(((uint16_t*)got)[k]);
            const double g = gate(gotf, ref, absagg, n);
            printf("%s %s: N=%lld E=%lld H=%d D=%d gate error %.3g (tolerance %.0e)\n",
                   dt == 0 ? "fp32" : "bf16", entry == 0 ? (dt == 0 ? "gt_attn_fwd" : "gt_attn_fwd_bf16")
                                                         : "gt_attn_fwd_noalloc",
                   (long long)N, (long long)E, H, D, g, tol);
            if (!(g <= tol)) bad = 1;
        }
        free(got);
        free(gotf);
        free(ref);
        free(absagg);
        for (int a = 0; a < 3; ++a) free(host[a]);
        HIP_OK(hipFree(d_rowptr));
        HIP_OK(hipFree(d_colidx));
        HIP_OK(hipFree(d_q));
        HIP_OK(hipFree(d_k));
        HIP_OK(hipFree(d_v));
        HIP_OK(hipFree(d_out));
    }
    if (gt_workspace_release() != GT_SUCCESS) bad = 1;
    free(rowptr);
    free(deg);
    free(colidx);
    free(seen);
    if (!bad) printf("c_caller_gpu ok\n");
    return bad;
}
