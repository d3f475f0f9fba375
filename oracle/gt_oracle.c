/*
 * CPU oracle: graph-transformer attention over a CSR graph, in float64.
 *
 * TEST INFRASTRUCTURE.  Only the test suite, the smoke check and the CPU
 * baseline leg of the benchmark may load or call this code.  It shares no
 * code, header or constant with the GPU implementation and never calls it.
 *
 * Definition followed (paper, Section 2.2, attention-based family (iii), with
 * the graph-transformer logits e_ij = q_i . k_j / sqrt(D)):
 *
 *   for every destination row i and head h, over the CSR entries e of row i
 *   (source j_e = colidx[e]; every entry is one softmax term, so a repeated
 *   entry counts twice; no self-loop is added beyond what the CSR lists):
 *     s_e      = scale * sum_d Q[i,h,d] * K[j_e,h,d]
 *     alpha_e  = exp(s_e) / sum_e' exp(s_e')
 *     out[i,h,:]    = sum_e alpha_e * V[j_e,h,:]
 *     absagg[i,h,:] = sum_e alpha_e * |V[j_e,h,:]|   (scale of the rounding error)
 *     lse[i,h]      = log sum_e exp(s_e)              (statistic the paper stores
 *                                                      for the backward pass, App. D.2)
 *   A row with no entries gives out = absagg = 0 and lse = -inf.
 *
 * The softmax is evaluated as the plain two-pass form: pass 1 computes every
 * score and their maximum m, pass 2 sums exp(s_e - m).  Subtracting m leaves
 * alpha unchanged and keeps exp from overflowing.  The paper's kernels reach
 * the same values in one streaming pass (online softmax, App. D.2); this file
 * deliberately does not.
 *
 * Inputs are read exactly as stored: fp32 values are widened to double; bf16
 * values (uint16 bit patterns) are widened by placing them in the upper half
 * of an fp32 word.  `scale` is used as double(scale).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { ORACLE_F32 = 0, ORACLE_BF16 = 1 };

static double elem(const void* base, int dtype, int64_t k) {
    if (dtype == ORACLE_F32) return (double)((const float*)base)[k];
    uint32_t bits = (uint32_t)((const uint16_t*)base)[k] << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
}

int gt_oracle_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/*
 * Computes rows rows[0..nrows) (all rows 0..N-1 when rows == NULL, with
 * nrows == N).  Results for the r-th requested row go to out[r,h,d],
 * absagg[r,h,d] (both [nrows][H][D]) and lse[r,h] ([nrows][H]); absagg and
 * lse may be NULL.  Returns 0 on success, 1 for bad arguments, 2 if the CSR
 * structure of a requested row is invalid (no results are then promised).
 */
int gt_oracle_fwd(int dtype, const int64_t* rowptr, const int32_t* colidx, const void* Q,
                  const void* K, const void* V, int64_t N, int64_t E, int32_t H, int32_t D,
                  float scale, const int64_t* rows, int64_t nrows, double* out, double* absagg,
                  double* lse) {
    if ((dtype != ORACLE_F32 && dtype != ORACLE_BF16) || N < 0 || E < 0 || H < 1 || D < 1 ||
        nrows < 0 || !rowptr || (nrows > 0 && !out) || (E > 0 && !colidx) ||
        (N > 0 && (!Q || !K || !V)) || (!rows && nrows != N))
        return 1;
    if (rowptr[0] != 0 || rowptr[N] != E) return 2;
    int status = 0;
#pragma omp parallel for schedule(dynamic, 16) reduction(| : status)
    for (int64_t r = 0; r < nrows; ++r) {
        const int64_t i = rows ? rows[r] : r;
        if (i < 0 || i >= N) { status |= 2; continue; }
        const int64_t b = rowptr[i], e = rowptr[i + 1];
        if (b < 0 || e < b || e > E) { status |= 2; continue; }
        const int64_t deg = e - b;
        int bad_col = 0;
        for (int64_t t = 0; t < deg; ++t)
            if (colidx[b + t] < 0 || colidx[b + t] >= N) bad_col = 1;
        if (bad_col) { status |= 2; continue; }
        double* s = (double*)malloc((size_t)(deg > 0 ? deg : 1) * sizeof(double));
        for (int32_t h = 0; h < H; ++h) {
            double* o = out + (r * H + h) * (int64_t)D;
            double* a = absagg ? absagg + (r * H + h) * (int64_t)D : NULL;
            for (int32_t d = 0; d < D; ++d) {
                o[d] = 0.0;
                if (a) a[d] = 0.0;
            }
            if (deg == 0) {
                if (lse) lse[r * H + h] = -INFINITY;
                continue;
            }
            /* pass 1: scores and their maximum */
            double m = -INFINITY;
            for (int64_t t = 0; t < deg; ++t) {
                const int64_t j = colidx[b + t];
                double dot = 0.0;
                for (int32_t d = 0; d < D; ++d)
                    dot += elem(Q, dtype, (i * H + h) * (int64_t)D + d) *
                           elem(K, dtype, (j * H + h) * (int64_t)D + d);
                s[t] = (double)scale * dot;
                if (s[t] > m) m = s[t];
            }
            /* pass 2: normaliser and weighted sums of V */
            double Z = 0.0;
            for (int64_t t = 0; t < deg; ++t) {
                const int64_t j = colidx[b + t];
                const double w = exp(s[t] - m);
                Z += w;
                for (int32_t d = 0; d < D; ++d) {
                    const double v = elem(V, dtype, (j * H + h) * (int64_t)D + d);
                    o[d] += w * v;
                    if (a) a[d] += w * fabs(v);
                }
            }
            for (int32_t d = 0; d < D; ++d) {
                o[d] /= Z;
                if (a) a[d] /= Z;
            }
            if (lse) lse[r * H + h] = m + log(Z);
        }
        free(s);
    }
    return status ? 2 : 0;
}
