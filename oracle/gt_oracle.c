/*
 * CPU oracle: graph-transformer attention over a CSR graph, in float64 (this
 * header); its backward, the GATv2 forward and the segment min/max reduction
 * follow further down, each with its own definition.
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

/* Threads of later parallel regions (n >= 1); used to time single-threaded runs. */
void gt_oracle_set_threads(int n) {
#ifdef _OPENMP
    if (n >= 1) omp_set_num_threads(n);
#else
    (void)n;
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

/* ------------------------------------------------------------- backward
 *
 * Gradients of the same attention with respect to Q, K and V, for an upstream
 * gradient dO [N][H][D] (same dtype as the features), in float64.  Followed
 * from the paper's backward description (Appendix D.2, backward pass of the
 * graph transformer): with the row statistic L_i = ln sum_e exp(s_e) the
 * weights are recomputed as alpha_e = exp(s_e - L_i); with
 * Delta_i = <O_i, dO_i> (O the exact forward output) and, per entry
 * e = (i, j):
 *     dalpha_e = <dO_i, V_j>,   ds_e = alpha_e * (dalpha_e - Delta_i)
 *     dQ_i += scale * ds_e * K_j
 *     dK_j += scale * ds_e * Q_i
 *     dV_j += alpha_e * dO_i
 * (all per head).  Alongside each gradient the routines return the same sums
 * taken over absolute values of every factor (dalpha and Delta as sums of
 * |products|), the scale of the rounding error of any evaluation.
 */

/* Row statistics of row i, head h: L (lse), o[D] (output), as the forward. */
static void row_stats(int dtype, const int64_t* rowptr, const int32_t* colidx, const void* Q,
                      const void* K, const void* V, int32_t H, int32_t D, double scale, int64_t i,
                      int32_t h, double* L, double* o, double* s) {
    const int64_t b = rowptr[i], e = rowptr[i + 1], deg = e - b;
    for (int32_t d = 0; d < D; ++d) o[d] = 0.0;
    if (deg == 0) { *L = -INFINITY; return; }
    double m = -INFINITY;
    for (int64_t t = 0; t < deg; ++t) {
        const int64_t j = colidx[b + t];
        double dot = 0.0;
        for (int32_t d = 0; d < D; ++d)
            dot += elem(Q, dtype, (i * H + h) * (int64_t)D + d) * elem(K, dtype, (j * H + h) * (int64_t)D + d);
        s[t] = scale * dot;
        if (s[t] > m) m = s[t];
    }
    double Z = 0.0;
    for (int64_t t = 0; t < deg; ++t) {
        const int64_t j = colidx[b + t];
        const double w = exp(s[t] - m);
        Z += w;
        for (int32_t d = 0; d < D; ++d) o[d] += w * elem(V, dtype, (j * H + h) * (int64_t)D + d);
    }
    for (int32_t d = 0; d < D; ++d) o[d] /= Z;
    *L = m + log(Z);
}

static int64_t max_degree(const int64_t* rowptr, int64_t N) {
    int64_t mx = 0;
    for (int64_t i = 0; i < N; ++i)
        if (rowptr[i + 1] - rowptr[i] > mx) mx = rowptr[i + 1] - rowptr[i];
    return mx;
}

/* dQ (and its error scale sdQ) for rows rows[0..nrows) (all rows if NULL). */
int gt_oracle_bwd_dq(int dtype, const int64_t* rowptr, const int32_t* colidx, const void* Q,
                     const void* K, const void* V, const void* dO, int64_t N, int64_t E, int32_t H,
                     int32_t D, float scale, const int64_t* rows, int64_t nrows, double* dQ,
                     double* sdQ) {
    if ((dtype != ORACLE_F32 && dtype != ORACLE_BF16) || N < 0 || H < 1 || D < 1 || !rowptr ||
        (E > 0 && !colidx) || (N > 0 && (!Q || !K || !V || !dO)) || (nrows > 0 && (!dQ || !sdQ)) ||
        (!rows && nrows != N))
        return 1;
    if (rowptr[0] != 0 || rowptr[N] != E) return 2;
    const double sc = (double)scale;
    const int64_t maxdeg = max_degree(rowptr, N);
    int status = 0;
#pragma omp parallel for schedule(dynamic, 16) reduction(| : status)
    for (int64_t r = 0; r < nrows; ++r) {
        const int64_t i = rows ? rows[r] : r;
        if (i < 0 || i >= N) { status |= 2; continue; }
        double* s = (double*)malloc((size_t)(maxdeg > 0 ? maxdeg : 1) * sizeof(double));
        double* o = (double*)malloc((size_t)D * sizeof(double));
        const int64_t b = rowptr[i], deg = rowptr[i + 1] - b;
        for (int32_t h = 0; h < H; ++h) {
            double* g = dQ + (r * H + h) * (int64_t)D;
            double* sg = sdQ + (r * H + h) * (int64_t)D;
            for (int32_t d = 0; d < D; ++d) g[d] = sg[d] = 0.0;
            if (deg == 0) continue;
            double L;
            row_stats(dtype, rowptr, colidx, Q, K, V, H, D, sc, i, h, &L, o, s);
            double delta = 0.0, delta_abs = 0.0;
            for (int32_t d = 0; d < D; ++d) {
                const double go = elem(dO, dtype, (i * H + h) * (int64_t)D + d);
                delta += o[d] * go;
                delta_abs += fabs(o[d] * go);
            }
            for (int64_t t = 0; t < deg; ++t) {
                const int64_t j = colidx[b + t];
                const double alpha = exp(s[t] - L);
                double da = 0.0, da_abs = 0.0;
                for (int32_t d = 0; d < D; ++d) {
                    const double p = elem(dO, dtype, (i * H + h) * (int64_t)D + d) *
                                     elem(V, dtype, (j * H + h) * (int64_t)D + d);
                    da += p;
                    da_abs += fabs(p);
                }
                const double ds = alpha * (da - delta);
                const double ds_abs = alpha * (da_abs + delta_abs);
                for (int32_t d = 0; d < D; ++d) {
                    const double kv = elem(K, dtype, (j * H + h) * (int64_t)D + d);
                    g[d] += sc * ds * kv;
                    sg[d] += fabs(sc) * ds_abs * fabs(kv);
                }
            }
        }
        free(o);
        free(s);
    }
    return status ? 2 : 0;
}

/*
 * dK, dV (and error scales) for source ids cols[0..ncols) (all if NULL),
 * using the transposed structure rowptr_t/colidx_t: colidx_t lists, for
 * source j, every destination row i whose CSR row holds j (once per entry).
 */
int gt_oracle_bwd_dkv(int dtype, const int64_t* rowptr, const int32_t* colidx,
                      const int64_t* rowptr_t, const int32_t* colidx_t, const void* Q, const void* K,
                      const void* V, const void* dO, int64_t N, int64_t E, int32_t H, int32_t D,
                      float scale, const int64_t* cols, int64_t ncols, double* dK, double* dV,
                      double* sdK, double* sdV) {
    if ((dtype != ORACLE_F32 && dtype != ORACLE_BF16) || N < 0 || H < 1 || D < 1 || !rowptr ||
        !rowptr_t || (E > 0 && (!colidx || !colidx_t)) || (N > 0 && (!Q || !K || !V || !dO)) ||
        (ncols > 0 && (!dK || !dV || !sdK || !sdV)) || (!cols && ncols != N))
        return 1;
    if (rowptr[0] != 0 || rowptr[N] != E || rowptr_t[0] != 0 || rowptr_t[N] != E) return 2;
    const double sc = (double)scale;
    /* statistics (L, o, Delta) of every destination row that points at a requested source */
    char* need = (char*)calloc((size_t)(N > 0 ? N : 1), 1);
    for (int64_t c = 0; c < ncols; ++c) {
        const int64_t j = cols ? cols[c] : c;
        if (j < 0 || j >= N) { free(need); return 2; }
        for (int64_t t = rowptr_t[j]; t < rowptr_t[j + 1]; ++t) {
            if (colidx_t[t] < 0 || colidx_t[t] >= N) { free(need); return 2; }
            need[colidx_t[t]] = 1;
        }
    }
    int64_t* slot = (int64_t*)malloc((size_t)(N > 0 ? N : 1) * sizeof(int64_t));
    int64_t n_need = 0;
    for (int64_t i = 0; i < N; ++i) slot[i] = need[i] ? n_need++ : -1;
    int64_t* which = (int64_t*)malloc((size_t)(n_need > 0 ? n_need : 1) * sizeof(int64_t));
    for (int64_t i = 0; i < N; ++i)
        if (need[i]) which[slot[i]] = i;
    double* Ls = (double*)malloc((size_t)(n_need > 0 ? n_need : 1) * H * sizeof(double));
    double* Dl = (double*)malloc((size_t)(n_need > 0 ? n_need : 1) * H * sizeof(double));
    double* Da = (double*)malloc((size_t)(n_need > 0 ? n_need : 1) * H * sizeof(double));
    const int64_t maxdeg = max_degree(rowptr, N);
#pragma omp parallel for schedule(dynamic, 16)
    for (int64_t u = 0; u < n_need; ++u) {
        const int64_t i = which[u];
        double* s = (double*)malloc((size_t)(maxdeg > 0 ? maxdeg : 1) * sizeof(double));
        double* o = (double*)malloc((size_t)D * sizeof(double));
        for (int32_t h = 0; h < H; ++h) {
            row_stats(dtype, rowptr, colidx, Q, K, V, H, D, sc, i, h, &Ls[u * H + h], o, s);
            double delta = 0.0, delta_abs = 0.0;
            for (int32_t d = 0; d < D; ++d) {
                const double go = elem(dO, dtype, (i * H + h) * (int64_t)D + d);
                delta += o[d] * go;
                delta_abs += fabs(o[d] * go);
            }
            Dl[u * H + h] = delta;
            Da[u * H + h] = delta_abs;
        }
        free(o);
        free(s);
    }
#pragma omp parallel for schedule(dynamic, 16)
    for (int64_t c = 0; c < ncols; ++c) {
        const int64_t j = cols ? cols[c] : c;
        for (int32_t h = 0; h < H; ++h) {
            double* gk = dK + (c * H + h) * (int64_t)D;
            double* gv = dV + (c * H + h) * (int64_t)D;
            double* sk = sdK + (c * H + h) * (int64_t)D;
            double* sv = sdV + (c * H + h) * (int64_t)D;
            for (int32_t d = 0; d < D; ++d) gk[d] = gv[d] = sk[d] = sv[d] = 0.0;
            for (int64_t t = rowptr_t[j]; t < rowptr_t[j + 1]; ++t) {
                const int64_t i = colidx_t[t], u = slot[i];
                double dot = 0.0, da = 0.0, da_abs = 0.0;
                for (int32_t d = 0; d < D; ++d) {
                    dot += elem(Q, dtype, (i * H + h) * (int64_t)D + d) * elem(K, dtype, (j * H + h) * (int64_t)D + d);
                    const double p = elem(dO, dtype, (i * H + h) * (int64_t)D + d) *
                                     elem(V, dtype, (j * H + h) * (int64_t)D + d);
                    da += p;
                    da_abs += fabs(p);
                }
                const double alpha = exp(sc * dot - Ls[u * H + h]);
                const double ds = alpha * (da - Dl[u * H + h]);
                const double ds_abs = alpha * (da_abs + Da[u * H + h]);
                for (int32_t d = 0; d < D; ++d) {
                    const double qv = elem(Q, dtype, (i * H + h) * (int64_t)D + d);
                    const double go = elem(dO, dtype, (i * H + h) * (int64_t)D + d);
                    gk[d] += sc * ds * qv;
                    sk[d] += fabs(sc) * ds_abs * fabs(qv);
                    gv[d] += alpha * go;
                    sv[d] += alpha * fabs(go);
                }
            }
        }
    }
    free(Da);
    free(Dl);
    free(Ls);
    free(which);
    free(slot);
    free(need);
    return 0;
}

/* ------------------------------------------------------------- GATv2
 *
 * Forward of the GATv2 attention (paper, Section 2.2, attention family (iii):
 * e_ij = a^T LeakyReLU(W_l h_i + W_r h_j), values v_j = W_r h_j; Appendix D.2,
 * "Fused forward in CSR (GATv2)").  With the projected features given,
 * Lf = W_l h and Rf = W_r h as [N][H][D], and the attention vector att
 * [H][D] (float32), per row i and head h over the CSR entries e of row i:
 *     s_e = sum_d att[h,d] * LeakyReLU(Lf[i,h,d] + Rf[j_e,h,d])
 *     out[i,h,:] = sum_e softmax_e(s) * Rf[j_e,h,:]
 * with LeakyReLU(x) = x for x > 0, slope * x otherwise.  Same two-pass
 * softmax, outputs (out, absagg, lse) and conventions as gt_oracle_fwd.
 */
int gt_oracle_gatv2_fwd(int dtype, const int64_t* rowptr, const int32_t* colidx, const void* Lf,
                        const void* Rf, const float* att, int64_t N, int64_t E, int32_t H,
                        int32_t D, float slope, const int64_t* rows, int64_t nrows, double* out,
                        double* absagg, double* lse) {
    if ((dtype != ORACLE_F32 && dtype != ORACLE_BF16) || N < 0 || E < 0 || H < 1 || D < 1 ||
        nrows < 0 || !rowptr || !att || (nrows > 0 && !out) || (E > 0 && !colidx) ||
        (N > 0 && (!Lf || !Rf)) || (!rows && nrows != N))
        return 1;
    if (rowptr[0] != 0 || rowptr[N] != E) return 2;
    const double sl = (double)slope;
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
            double m = -INFINITY;
            for (int64_t t = 0; t < deg; ++t) {
                const int64_t j = colidx[b + t];
                double acc = 0.0;
                for (int32_t d = 0; d < D; ++d) {
                    const double x = elem(Lf, dtype, (i * H + h) * (int64_t)D + d) +
                                     elem(Rf, dtype, (j * H + h) * (int64_t)D + d);
                    acc += (double)att[h * D + d] * (x > 0.0 ? x : sl * x);
                }
                s[t] = acc;
                if (s[t] > m) m = s[t];
            }
            double Z = 0.0;
            for (int64_t t = 0; t < deg; ++t) {
                const int64_t j = colidx[b + t];
                const double w = exp(s[t] - m);
                Z += w;
                for (int32_t d = 0; d < D; ++d) {
                    const double v = elem(Rf, dtype, (j * H + h) * (int64_t)D + d);
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

/*
 * Reduction family (paper Section 2.2, family (ii): h_i <- REDUCE over the
 * sources j of row i of h_j, REDUCE = min or max; Appendix, degree-aware
 * reduction-based aggregation: per feature, the reduced value and the source
 * node that attains it, kept for the backward scatter).
 *
 *   out[i,f] = the value X[j_e,f] selected over the CSR entries e of row i
 *   arg[i,f] = the source j_e it was taken from
 *
 * Order (Appendix, order-preserving packing): a value is compared through the
 * 32-bit key formed from its fp32 bit pattern -- all bits inverted when the
 * sign bit is set, the sign bit set otherwise -- as an unsigned integer; that
 * key is then paired with the source index and pairs compare
 * lexicographically.  So every non-NaN value is ordered as the reals, -0 lies
 * below +0, and among equal values the smallest source index wins.
 *   op 0 (min): the entry with the smallest (key, source) pair;
 *   op 1 (max): the entry with the largest key, ties to the smallest source.
 * A row with no entries gives out = 0 and arg = -1.  Values are selected,
 * never computed, so out holds an input value exactly (as fp32; bf16 inputs
 * are widened exactly).
 */
static uint32_t order_key(float x) {
    uint32_t b;
    memcpy(&b, &x, sizeof b);
    return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

int gt_oracle_segment_reduce(int dtype, int op, const int64_t* rowptr, const int32_t* colidx,
                             const void* X, int64_t N, int64_t E, int32_t F,
                             const int64_t* rows, int64_t nrows, float* out, int32_t* arg) {
    if ((dtype != ORACLE_F32 && dtype != ORACLE_BF16) || (op != 0 && op != 1) || N < 0 ||
        E < 0 || F < 1 || nrows < 0 || !rowptr || (nrows > 0 && (!out || !arg)) ||
        (E > 0 && !colidx) || (N > 0 && !X) || (!rows && nrows != N))
        return 1;
    if (rowptr[0] != 0 || rowptr[N] != E) return 2;
    int status = 0;
#pragma omp parallel for schedule(dynamic, 16) reduction(| : status)
    for (int64_t r = 0; r < nrows; ++r) {
        const int64_t i = rows ? rows[r] : r;
        if (i < 0 || i >= N) { status |= 2; continue; }
        const int64_t b = rowptr[i], e = rowptr[i + 1];
        if (b < 0 || e < b || e > E) { status |= 2; continue; }
        int bad_col = 0;
        for (int64_t t = b; t < e; ++t)
            if (colidx[t] < 0 || colidx[t] >= N) bad_col = 1;
        if (bad_col) { status |= 2; continue; }
        for (int32_t f = 0; f < F; ++f) {
            int have = 0;
            float best = 0.0f;
            uint32_t best_key = 0;
            int32_t best_j = -1;
            for (int64_t t = b; t < e; ++t) {
                const int32_t j = colidx[t];
                const float x = (float)elem(X, dtype, (int64_t)j * F + f);
                const uint32_t k = order_key(x);
                int better;
                if (!have)
                    better = 1;
                else if (op == 0)
                    better = k < best_key || (k == best_key && j < best_j);
                else
                    better = k > best_key || (k == best_key && j < best_j);
                if (better) {
                    have = 1;
                    best = x;
                    best_key = k;
                    best_j = j;
                }
            }
            out[r * F + f] = have ? best : 0.0f;
            arg[r * F + f] = have ? best_j : -1;
        }
    }
    return status ? 2 : 0;
}

/*
 * Locality microbenchmark of the reordering study (paper, graph reordering
 * paragraph of Section 4 and its appendix figure: a "dot-aggr" kernel with
 * identical arithmetic under two mappings).  Reading: for every row i,
 *
 *   s[i] = sum over the CSR entries e of row i of sum_f X[i,f] * X[j_e,f]
 *
 * (a repeated entry counts twice; an empty row gives 0), fp32 X.  absout[i]
 * = the same sum of |X[i,f] * X[j_e,f]|, the scale of any floating-point
 * evaluation's rounding error.
 */
int gt_oracle_dot_aggr(const int64_t* rowptr, const int32_t* colidx, const float* X, int64_t N,
                       int64_t E, int32_t F, const int64_t* rows, int64_t nrows, double* out,
                       double* absout) {
    if (N < 0 || E < 0 || F < 1 || nrows < 0 || !rowptr || (nrows > 0 && !out) ||
        (E > 0 && !colidx) || (N > 0 && !X) || (!rows && nrows != N))
        return 1;
    if (rowptr[0] != 0 || rowptr[N] != E) return 2;
    int status = 0;
#pragma omp parallel for schedule(dynamic, 16) reduction(| : status)
    for (int64_t r = 0; r < nrows; ++r) {
        const int64_t i = rows ? rows[r] : r;
        if (i < 0 || i >= N) { status |= 2; continue; }
        const int64_t b = rowptr[i], e = rowptr[i + 1];
        if (b < 0 || e < b || e > E) { status |= 2; continue; }
        double s = 0.0, a = 0.0;
        for (int64_t t = b; t < e; ++t) {
            const int64_t j = colidx[t];
            if (j < 0 || j >= N) { status |= 2; break; }
            for (int32_t f = 0; f < F; ++f) {
                const double p = (double)X[i * F + f] * (double)X[j * F + f];
                s += p;
                a += fabs(p);
            }
        }
        out[r] = s;
        if (absout) absout[r] = a;
    }
    return status ? 2 : 0;
}
