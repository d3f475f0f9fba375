/*
 * Seeded synthetic inputs for the CSR graph-attention workloads.
 *
 * This file generates inputs only: graphs in CSR form (destination rows,
 * source columns) and Gaussian feature tensors.  It contains none of the
 * attention arithmetic.  Both the CPU oracle and the GPU path consume what
 * it produces; neither is linked into it.
 *
 * Every random value is a pure function of (seed, stream, counter) through
 * Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as
 * easy as 1, 2, 3", SC 2011), so results do not depend on the number of
 * OpenMP threads.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <math.h>

/* ---------------------------------------------------------------- Philox */

static inline void philox_round(uint32_t c[4], const uint32_t k[2]) {
    const uint64_t p0 = (uint64_t)0xD2511F53u * c[0];
    const uint64_t p1 = (uint64_t)0xCD9E8D57u * c[2];
    const uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
    const uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
    const uint32_t n0 = hi1 ^ c[1] ^ k[0];
    const uint32_t n2 = hi0 ^ c[3] ^ k[1];
    c[0] = n0; c[1] = lo1; c[2] = n2; c[3] = lo0;
}

void synth_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]) {
    uint32_t c[4] = {ctr[0], ctr[1], ctr[2], ctr[3]};
    uint32_t k[2] = {key[0], key[1]};
    philox_round(c, k);
    for (int r = 1; r < 10; ++r) {
        k[0] += 0x9E3779B9u;
        k[1] += 0xBB67AE85u;
        philox_round(c, k);
    }
    memcpy(out, c, sizeof c);
}

/* One Philox block addressed by (seed, stream, a, b). */
static inline void draw4(uint64_t seed, uint32_t stream, uint64_t a, uint32_t b, uint32_t out[4]) {
    const uint32_t ctr[4] = {(uint32_t)a, (uint32_t)(a >> 32), b, stream};
    const uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    synth_philox4x32_10(ctr, key, out);
}

/* u in the open interval (0, 1) from 32 random bits. */
static inline double u01(uint32_t x) { return ((double)x + 0.5) * (1.0 / 4294967296.0); }

/* Uniform integer in [0, bound) from 64 random bits (multiply-high). */
static inline uint64_t below(uint32_t lo, uint32_t hi, uint64_t bound) {
    const uint64_t x = ((uint64_t)hi << 32) | lo;
    return (uint64_t)(((unsigned __int128)x * bound) >> 64);
}

/* Round-to-nearest-even fp32 -> bf16 bit pattern (finite inputs). */
static inline uint16_t to_bf16(float f) {
    uint32_t u;
    memcpy(&u, &f, 4);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

/* ------------------------------------------------------------- features */

/*
 * n normals with standard deviation `std`, Box-Muller on Philox output.
 * Element e comes from block e/4 of (seed, stream); writes fp32 into out_f32
 * or bf16 (RNE of the fp32 value) into out_bf16, whichever is non-null.
 */
void synth_normal(uint64_t seed, uint32_t stream, double std, int64_t n,
                  float* out_f32, uint16_t* out_bf16) {
    const int64_t nblk = (n + 3) / 4;
#pragma omp parallel for schedule(static)
    for (int64_t b = 0; b < nblk; ++b) {
        uint32_t r[4];
        draw4(seed, stream, (uint64_t)b, 0u, r);
        float z[4];
        for (int p = 0; p < 2; ++p) {
            const double rad = sqrt(-2.0 * log(u01(r[2 * p])));
            const double ang = 6.283185307179586 * u01(r[2 * p + 1]);
            z[2 * p] = (float)(std * rad * cos(ang));
            z[2 * p + 1] = (float)(std * rad * sin(ang));
        }
        for (int t = 0; t < 4; ++t) {
            const int64_t e = 4 * b + t;
            if (e >= n) break;
            if (out_f32) out_f32[e] = z[t];
            if (out_bf16) out_bf16[e] = to_bf16(z[t]);
        }
    }
}

/* n uniforms in (0, 1); element e from block e of (seed, stream). */
void synth_uniform01(uint64_t seed, uint32_t stream, int64_t n, double* out) {
#pragma omp parallel for schedule(static)
    for (int64_t e = 0; e < n; ++e) {
        uint32_t r[4];
        draw4(seed, stream, (uint64_t)e, 1u, r);
        out[e] = u01(r[0]);
    }
}

/* ----------------------------------------------------------------- graphs */

static int cmp_i32(const void* a, const void* b) {
    const int32_t x = *(const int32_t*)a, y = *(const int32_t*)b;
    return (x > y) - (x < y);
}

/*
 * For each row i, fill colidx[rowptr[i] .. rowptr[i+1]) with distinct source
 * ids.  With add_self, the row holds i itself plus (len-1) distinct sources
 * drawn uniformly from [0,N) without i; otherwise len distinct sources drawn
 * uniformly from [0,N) without i.  Draw k of row i uses block (i, k).  Rows
 * are sorted ascending.  Returns 0, or -1 if a row asks for more distinct
 * sources than exist.
 */
int synth_distinct_sources(uint64_t seed, uint32_t stream, int64_t N, const int64_t* rowptr,
                           int32_t* colidx, int add_self) {
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 256) reduction(| : bad)
    for (int64_t i = 0; i < N; ++i) {
        int32_t* row = colidx + rowptr[i];
        int64_t len = rowptr[i + 1] - rowptr[i];
        int64_t want = len - (add_self && len > 0 ? 1 : 0);
        if (want > N - 1) { bad = 1; continue; }
        int64_t have = 0;
        if (add_self && len > 0) row[have++] = (int32_t)i;
        /* open-addressing set of accepted ids for rows beyond a small size */
        int64_t cap = 0;
        int32_t* set = NULL;
        if (want > 32) {
            cap = 1;
            while (cap < 4 * want) cap <<= 1;
            set = (int32_t*)malloc((size_t)cap * sizeof(int32_t));
            for (int64_t s = 0; s < cap; ++s) set[s] = -1;
        }
        uint64_t k = 0;
        int64_t got = 0;
        while (got < want) {
            uint32_t r[4];
            draw4(seed, stream, (uint64_t)i, (uint32_t)k, r);
            ++k;
            for (int p = 0; p < 2 && got < want; ++p) {
                uint64_t v = below(r[2 * p], r[2 * p + 1], (uint64_t)(N - 1));
                if ((int64_t)v >= i) ++v; /* skip i itself */
                int dup = 0;
                if (set) {
                    uint64_t h = (v * 0x9E3779B97F4A7C15ull) >> 20;
                    for (;;) {
                        int64_t s = (int64_t)(h & (uint64_t)(cap - 1));
                        if (set[s] < 0) { set[s] = (int32_t)v; break; }
                        if (set[s] == (int32_t)v) { dup = 1; break; }
                        ++h;
                    }
                } else {
                    for (int64_t t = (add_self && len > 0) ? 1 : 0; t < have; ++t)
                        if (row[t] == (int32_t)v) { dup = 1; break; }
                }
                if (!dup) { row[have++] = (int32_t)v; ++got; }
            }
        }
        free(set);
        qsort(row, (size_t)len, sizeof(int32_t), cmp_i32);
    }
    return bad ? -1 : 0;
}

/*
 * R-MAT sampling (Chakrabarti, Zhan, Faloutsos, SDM 2004).  Sample s descends
 * `scale` levels; at each level the quadrant (src bit, dst bit) is
 * (0,0) w.p. a, (0,1) w.p. b, (1,0) w.p. c, (1,1) otherwise.  Samples are
 * taken in order; self pairs and repeats of an earlier pair are dropped, and
 * sampling stops once `target` distinct pairs are kept.  Writes src/dst
 * (capacity target) and returns the number of samples consumed, or -1 if
 * max_samples did not suffice.
 */
int64_t synth_rmat(uint64_t seed, uint32_t stream, int scale, double a, double b, double c,
                   int64_t target, int64_t max_samples, int32_t* src, int32_t* dst) {
    const int64_t batch = 1 << 22;
    uint64_t* keys = (uint64_t*)malloc((size_t)batch * sizeof(uint64_t));
    int64_t cap = 1;
    while (cap < 2 * target) cap <<= 1;
    uint64_t* set = (uint64_t*)malloc((size_t)cap * sizeof(uint64_t));
    const uint64_t EMPTY = ~0ull;
    for (int64_t s = 0; s < cap; ++s) set[s] = EMPTY;
    const double ab = a + b, abc = a + b + c;
    int64_t kept = 0, used = 0;
    for (int64_t base = 0; kept < target && base < max_samples; base += batch) {
        const int64_t nb = (base + batch <= max_samples) ? batch : (max_samples - base);
#pragma omp parallel for schedule(static)
        for (int64_t t = 0; t < nb; ++t) {
            uint64_t su = 0, dv = 0;
            uint32_t r[4];
            for (int lvl = 0; lvl < scale; ++lvl) {
                if ((lvl & 3) == 0) draw4(seed, stream, (uint64_t)(base + t), (uint32_t)(lvl >> 2), r);
                const double u = u01(r[lvl & 3]);
                const uint64_t sb = (u >= ab) ? 1u : 0u;
                const uint64_t db = ((u >= a && u < ab) || u >= abc) ? 1u : 0u;
                su = (su << 1) | sb;
                dv = (dv << 1) | db;
            }
            keys[t] = (su << 32) | dv;
        }
        for (int64_t t = 0; t < nb && kept < target; ++t) {
            ++used;
            const uint64_t key = keys[t];
            if ((key >> 32) == (key & 0xFFFFFFFFull)) continue;
            uint64_t h = (key * 0x9E3779B97F4A7C15ull) >> 17;
            for (;;) {
                const int64_t s = (int64_t)(h & (uint64_t)(cap - 1));
                if (set[s] == EMPTY) {
                    set[s] = key;
                    src[kept] = (int32_t)(key >> 32);
                    dst[kept] = (int32_t)(key & 0xFFFFFFFFull);
                    ++kept;
                    break;
                }
                if (set[s] == key) break;
                ++h;
            }
        }
    }
    free(set);
    free(keys);
    return kept == target ? used : -1;
}

/*
 * CSR from (dst, src) pairs: row = dst.  With add_self every row also gets
 * its self-loop (callers guarantee no self pair is present).  rowptr has N+1
 * entries; colidx has n + (add_self ? N : 0).  Rows are sorted ascending.
 */
void synth_csr_from_pairs(int64_t N, int64_t n, const int32_t* dst, const int32_t* src,
                          int add_self, int64_t* rowptr, int32_t* colidx) {
    for (int64_t i = 0; i <= N; ++i) rowptr[i] = 0;
    for (int64_t e = 0; e < n; ++e) rowptr[dst[e] + 1]++;
    if (add_self)
        for (int64_t i = 0; i < N; ++i) rowptr[i + 1]++;
    for (int64_t i = 0; i < N; ++i) rowptr[i + 1] += rowptr[i];
    int64_t* fill = (int64_t*)malloc((size_t)N * sizeof(int64_t));
    for (int64_t i = 0; i < N; ++i) fill[i] = rowptr[i];
    if (add_self)
        for (int64_t i = 0; i < N; ++i) colidx[fill[i]++] = (int32_t)i;
    for (int64_t e = 0; e < n; ++e) colidx[fill[dst[e]]++] = src[e];
    free(fill);
#pragma omp parallel for schedule(dynamic, 1024)
    for (int64_t i = 0; i < N; ++i)
        qsort(colidx + rowptr[i], (size_t)(rowptr[i + 1] - rowptr[i]), sizeof(int32_t), cmp_i32);
}

/*
 * Stochastic block model with contiguous blocks of `bs` ids.  Row i gets:
 * its self-loop; every other id j of its block independently with
 * probability 1/2 (one Philox bit per (i, j)); and `n_out` distinct sources
 * drawn uniformly from outside its block.  Pass colidx = NULL to only fill
 * rowptr (N+1 entries); call again with colidx to fill the rows (sorted).
 */
void synth_sbm(uint64_t seed, uint32_t stream, int64_t N, int64_t bs, int64_t n_out,
               int64_t* rowptr, int32_t* colidx) {
    if (!colidx) {
        rowptr[0] = 0;
#pragma omp parallel for schedule(static)
        for (int64_t i = 0; i < N; ++i) {
            const int64_t b0 = (i / bs) * bs;
            int64_t deg = 1 + n_out;
            for (int64_t w = 0; w < (bs + 127) / 128; ++w) {
                uint32_t r[4];
                draw4(seed, stream, (uint64_t)i, (uint32_t)w, r);
                for (int64_t t = 0; t < 128 && w * 128 + t < bs; ++t) {
                    const int64_t j = b0 + w * 128 + t;
                    if (j == i || j >= N) continue;
                    deg += (r[t >> 5] >> (t & 31)) & 1u;
                }
            }
            rowptr[i + 1] = deg;
        }
        for (int64_t i = 0; i < N; ++i) rowptr[i + 1] += rowptr[i];
        return;
    }
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < N; ++i) {
        int32_t* row = colidx + rowptr[i];
        int64_t have = 0;
        const int64_t b0 = (i / bs) * bs;
        const int64_t b1 = (b0 + bs < N) ? b0 + bs : N;
        row[have++] = (int32_t)i;
        for (int64_t w = 0; w < (bs + 127) / 128; ++w) {
            uint32_t r[4];
            draw4(seed, stream, (uint64_t)i, (uint32_t)w, r);
            for (int64_t t = 0; t < 128 && w * 128 + t < bs; ++t) {
                const int64_t j = b0 + w * 128 + t;
                if (j == i || j >= N) continue;
                if ((r[t >> 5] >> (t & 31)) & 1u) row[have++] = (int32_t)j;
            }
        }
        const int64_t outside = N - (b1 - b0);
        const int64_t first_out = have;
        uint32_t k = 0;
        while (have < first_out + n_out) {
            uint32_t r[4];
            draw4(seed, stream ^ 0x80000000u, (uint64_t)i, k++, r);
            for (int p = 0; p < 2 && have < first_out + n_out; ++p) {
                int64_t v = (int64_t)below(r[2 * p], r[2 * p + 1], (uint64_t)outside);
                if (v >= b0) v += (b1 - b0);
                int dup = 0;
                for (int64_t t = first_out; t < have; ++t)
                    if (row[t] == (int32_t)v) { dup = 1; break; }
                if (!dup) row[have++] = (int32_t)v;
            }
        }
        qsort(row, (size_t)have, sizeof(int32_t), cmp_i32);
    }
}
