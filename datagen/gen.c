/*
 * Seeded synthetic workload generator (host C, OpenMP).
 *
 * This module only draws random inputs; it holds none of the method's
 * arithmetic.  The GPU path and the CPU oracle both consume its output.
 *
 * Every random number comes from Philox4x32-10 (Salmon, Moraes, Dror, Shaw,
 * "Parallel random numbers: as easy as 1, 2, 3", SC'11), keyed by
 * (seed, stream) with the counter holding the row (or feature) index and a
 * block index, so a row's draws do not depend on how rows are split across
 * threads.  Distributions:
 *   - normal: Box-Muller (cosine branch only);
 *   - Zipf(alpha) over ranks 1..d: inverse CDF by binary search over an fp64
 *     table; rank k maps to feature id k-1 (hot ids are small);
 *   - Poisson(mu): Hormann's transformed rejection with squeeze (PTRS,
 *     Insurance: Mathematics and Economics 12, 1993), for mu >= 10;
 *   - feature ids within a row are drawn without replacement (a redraw on a
 *     duplicate) and stored sorted ascending.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <omp.h>

/* ---------------- Philox4x32-10 ---------------- */
typedef struct { uint32_t v[4]; } u32x4;

static inline void mulhilo32(uint32_t a, uint32_t b, uint32_t *hi, uint32_t *lo) {
    uint64_t p = (uint64_t)a * (uint64_t)b;
    *hi = (uint32_t)(p >> 32);
    *lo = (uint32_t)p;
}

u32x4 gen_philox4x32_10(u32x4 ctr, uint32_t k0, uint32_t k1) {
    const uint32_t M0 = 0xD2511F53u, M1 = 0xCD9E8D57u;
    const uint32_t W0 = 0x9E3779B9u, W1 = 0xBB67AE85u;
    for (int r = 0; r < 10; ++r) {
        uint32_t hi0, lo0, hi1, lo1;
        mulhilo32(M0, ctr.v[0], &hi0, &lo0);
        mulhilo32(M1, ctr.v[2], &hi1, &lo1);
        u32x4 o;
        o.v[0] = hi1 ^ ctr.v[1] ^ k0;
        o.v[1] = lo1;
        o.v[2] = hi0 ^ ctr.v[3] ^ k1;
        o.v[3] = lo0;
        ctr = o;
        k0 += W0;
        k1 += W1;
    }
    return ctr;
}

/* exported for the known-answer test */
void gen_philox_block(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]) {
    u32x4 c = {{ctr[0], ctr[1], ctr[2], ctr[3]}};
    u32x4 r = gen_philox4x32_10(c, key[0], key[1]);
    memcpy(out, r.v, sizeof r.v);
}

typedef struct {
    uint32_t k0, k1;
    uint32_t c0, c1, blk;
    uint32_t buf[4];
    int idx;
} rng_t;

enum {
    ST_NNZ = 1, ST_COL = 2, ST_VAL = 3, ST_WSTAR = 4, ST_LABEL = 5,
    ST_USER = 6, ST_ITEM = 7, ST_USTAR = 8, ST_VSTAR = 9, ST_NOISE = 10,
    ST_U0 = 11, ST_V0 = 12, ST_DENSE = 13
};

static inline void rng_init(rng_t *r, uint64_t seed, uint32_t stream, uint64_t index) {
    r->k0 = (uint32_t)seed;
    r->k1 = (uint32_t)(seed >> 32) ^ (stream * 0x85EBCA6Bu);
    r->c0 = (uint32_t)index;
    r->c1 = (uint32_t)(index >> 32);
    r->blk = 0;
    r->idx = 4;
}

static inline uint32_t rng_u32(rng_t *r) {
    if (r->idx == 4) {
        u32x4 c = {{r->c0, r->c1, r->blk, 0u}};
        u32x4 o = gen_philox4x32_10(c, r->k0, r->k1);
        memcpy(r->buf, o.v, sizeof o.v);
        r->blk++;
        r->idx = 0;
    }
    return r->buf[r->idx++];
}

/* uniform double in the open interval (0,1), 53 random bits */
static inline double rng_unif(rng_t *r) {
    uint32_t a = rng_u32(r) >> 5, b = rng_u32(r) >> 6;
    uint64_t x = ((uint64_t)a << 26) | b;
    return ((double)x + 0.5) * (1.0 / 9007199254740992.0);
}

static inline double rng_normal(rng_t *r) {
    double u1 = rng_unif(r), u2 = rng_unif(r);
    return sqrt(-2.0 * log(u1)) * cos(6.283185307179586476925 * u2);
}

static int64_t rng_poisson_ptrs(rng_t *r, double mu) {
    double slam = sqrt(mu), loglam = log(mu);
    double b = 0.931 + 2.53 * slam;
    double a = -0.059 + 0.02483 * b;
    double invalpha = 1.1239 + 1.1328 / (b - 3.4);
    double vr = 0.9277 - 3.6224 / (b - 2.0);
    for (;;) {
        double U = rng_unif(r) - 0.5;
        double V = rng_unif(r);
        double us = 0.5 - fabs(U);
        int64_t k = (int64_t)floor((2.0 * a / us + b) * U + mu + 0.43);
        if (us >= 0.07 && V <= vr) return k;
        if (k < 0 || (us < 0.013 && V > us)) continue;
        if (log(V) + log(invalpha) - log(a / (us * us) + b) <=
            -mu + (double)k * loglam - lgamma((double)k + 1.0))
            return k;
    }
}

/* ---------------- Zipf inverse CDF ---------------- */
double *gen_zipf_cdf(int64_t d, double alpha) {
    double *cdf = (double *)malloc((size_t)d * sizeof(double));
    if (!cdf) return NULL;
    double s = 0.0;
    for (int64_t k = 0; k < d; ++k) {
        s += pow((double)(k + 1), -alpha);
        cdf[k] = s;
    }
    for (int64_t k = 0; k < d; ++k) cdf[k] /= s;
    cdf[d - 1] = 1.0;
    return cdf;
}

void gen_free(void *p) { free(p); }

static inline int64_t zipf_draw(rng_t *r, const double *cdf, int64_t d) {
    double u = rng_unif(r);
    int64_t lo = 0, hi = d - 1;
    while (lo < hi) {
        int64_t mid = lo + ((hi - lo) >> 1);
        if (cdf[mid] >= u) hi = mid; else lo = mid + 1;
    }
    return lo;
}

/* ---------------- sparse (CSR) workloads ---------------- */
typedef struct {
    int64_t n, d;
    int32_t nnz_kind;   /* 0 fixed nnz_a, 1 uniform int [a,b], 2 Poisson(mean) clipped to [a,b] */
    int32_t id_kind;    /* 0 Zipf(alpha), 1 uniform */
    int64_t nnz_a, nnz_b;
    double nnz_mean;
    double alpha;
    int32_t val_kind;   /* 0 N(0,1), 1 random sign * exp(N(0, val_s)), 2 all ones */
    int32_t label_kind; /* 0 sign(x.w*) with flips (prob label_p), 1 x.w* + N(0, label_p) */
    double val_s;
    double label_p;
    uint64_t seed;
} gen_params;

static int64_t row_nnz(const gen_params *p, int64_t i) {
    rng_t r;
    rng_init(&r, p->seed, ST_NNZ, (uint64_t)i);
    int64_t m;
    switch (p->nnz_kind) {
    case 0: m = p->nnz_a; break;
    case 1: m = p->nnz_a + (int64_t)floor(rng_unif(&r) * (double)(p->nnz_b - p->nnz_a + 1)); break;
    default:
        m = rng_poisson_ptrs(&r, p->nnz_mean);
        if (m < p->nnz_a) m = p->nnz_a;
        if (m > p->nnz_b) m = p->nnz_b;
        break;
    }
    if (m > p->d) m = p->d;
    return m;
}

/* Pass 1: row_ptr[0..n]; returns nnz (or -1 on bad parameters). */
int64_t gen_row_ptr(const gen_params *p, int64_t *row_ptr, int nthreads) {
    if (p->n < 0 || p->d <= 0) return -1;
    if (nthreads > 0) omp_set_num_threads(nthreads);
    row_ptr[0] = 0;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < p->n; ++i) row_ptr[i + 1] = row_nnz(p, i);
    for (int64_t i = 0; i < p->n; ++i) row_ptr[i + 1] += row_ptr[i];
    return row_ptr[p->n];
}

static void sort_i32(int32_t *a, int64_t m) {
    for (int64_t i = 1; i < m; ++i) {
        int32_t x = a[i];
        int64_t j = i - 1;
        while (j >= 0 && a[j] > x) { a[j + 1] = a[j]; --j; }
        a[j + 1] = x;
    }
}

static int cmp_i32(const void *a, const void *b) {
    int32_t x = *(const int32_t *)a, y = *(const int32_t *)b;
    return (x > y) - (x < y);
}

/* Planted weights w*[f] ~ N(0,1), keyed by feature. */
void gen_wstar(uint64_t seed, int64_t d, double *wstar, int nthreads) {
    if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for schedule(static)
    for (int64_t f = 0; f < d; ++f) {
        rng_t r;
        rng_init(&r, seed, ST_WSTAR, (uint64_t)f);
        wstar[f] = rng_normal(&r);
    }
}

/* Pass 2: columns (sorted, unique per row), values (if val != NULL) and labels. */
int gen_fill(const gen_params *p, const int64_t *row_ptr, int32_t *col, float *val, float *y,
             int nthreads) {
    double *cdf = NULL;
    if (p->id_kind == 0) {
        cdf = gen_zipf_cdf(p->d, p->alpha);
        if (!cdf) return -1;
    }
    double *wstar = (double *)malloc((size_t)p->d * sizeof(double));
    if (!wstar) { free(cdf); return -1; }
    gen_wstar(p->seed, p->d, wstar, nthreads);
    if (nthreads > 0) omp_set_num_threads(nthreads);
    int err = 0;
#pragma omp parallel
    {
        int64_t cap = 1024;
        int32_t *table = (int32_t *)malloc((size_t)cap * 2 * sizeof(int32_t));
        if (!table) err = 1;
#pragma omp for schedule(dynamic, 1024)
        for (int64_t i = 0; i < p->n; ++i) {
            if (!table) continue;
            int64_t b = row_ptr[i], m = row_ptr[i + 1] - b;
            int32_t *c = col + b;
            /* hash set of ids already in the row (open addressing, power of two) */
            int64_t hs = 16;
            while (hs < 2 * m) hs <<= 1;
            if (hs > cap * 2) {
                free(table);
                cap = hs;
                table = (int32_t *)malloc((size_t)cap * 2 * sizeof(int32_t));
                if (!table) { err = 1; continue; }
            }
            for (int64_t h = 0; h < hs; ++h) table[h] = -1;
            rng_t r;
            rng_init(&r, p->seed, ST_COL, (uint64_t)i);
            int64_t got = 0;
            while (got < m) {
                int64_t f = (p->id_kind == 0) ? zipf_draw(&r, cdf, p->d)
                                              : (int64_t)floor(rng_unif(&r) * (double)p->d);
                if (f >= p->d) f = p->d - 1;
                uint64_t h = ((uint64_t)f * 0x9E3779B97F4A7C15ull) >> 20;
                int dup = 0;
                for (;;) {
                    h &= (uint64_t)(hs - 1);
                    if (table[h] < 0) { table[h] = (int32_t)f; break; }
                    if (table[h] == (int32_t)f) { dup = 1; break; }
                    ++h;
                }
                if (!dup) c[got++] = (int32_t)f;
            }
            if (m <= 64) sort_i32(c, m); else qsort(c, (size_t)m, sizeof(int32_t), cmp_i32);
            rng_t rv;
            rng_init(&rv, p->seed, ST_VAL, (uint64_t)i);
            double dot = 0.0;
            for (int64_t k = 0; k < m; ++k) {
                float v;
                switch (p->val_kind) {
                case 0: v = (float)rng_normal(&rv); break;
                case 1: {
                    double mag = exp(p->val_s * rng_normal(&rv));
                    double sgn = (rng_u32(&rv) & 1u) ? -1.0 : 1.0;
                    v = (float)(sgn * mag);
                    break;
                }
                default: v = 1.0f; break;
                }
                if (val) val[b + k] = v;
                dot += (double)v * wstar[c[k]];
            }
            rng_t rl;
            rng_init(&rl, p->seed, ST_LABEL, (uint64_t)i);
            if (p->label_kind == 0) {
                float s = (dot >= 0.0) ? 1.0f : -1.0f;
                if (rng_unif(&rl) < p->label_p) s = -s;
                y[i] = s;
            } else {
                y[i] = (float)(dot + p->label_p * rng_normal(&rl));
            }
        }
        free(table);
    }
    free(wstar);
    free(cdf);
    return err ? -1 : 0;
}

/* ---------------- matrix completion ---------------- */
/* ratings r = <u*_u, v*_i> + N(0, noise_sd); u*, v*, U0, V0 entries ~ N(0, factor_sd) */
int gen_mf(uint64_t seed, int64_t n_ratings, int64_t n_users, int64_t n_items, double alpha_u,
           double alpha_i, int32_t rank, double factor_sd, double noise_sd, int32_t *user,
           int32_t *item, float *rating, float *U0, float *V0, int nthreads) {
    double *cu = gen_zipf_cdf(n_users, alpha_u);
    double *ci = gen_zipf_cdf(n_items, alpha_i);
    double *us = (double *)malloc((size_t)n_users * rank * sizeof(double));
    double *vs = (double *)malloc((size_t)n_items * rank * sizeof(double));
    if (!cu || !ci || !us || !vs) { free(cu); free(ci); free(us); free(vs); return -1; }
    if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for schedule(static)
    for (int64_t u = 0; u < n_users; ++u) {
        rng_t r, r0;
        rng_init(&r, seed, ST_USTAR, (uint64_t)u);
        rng_init(&r0, seed, ST_U0, (uint64_t)u);
        for (int32_t k = 0; k < rank; ++k) {
            us[u * rank + k] = factor_sd * rng_normal(&r);
            U0[u * rank + k] = (float)(factor_sd * rng_normal(&r0));
        }
    }
#pragma omp parallel for schedule(static)
    for (int64_t it = 0; it < n_items; ++it) {
        rng_t r, r0;
        rng_init(&r, seed, ST_VSTAR, (uint64_t)it);
        rng_init(&r0, seed, ST_V0, (uint64_t)it);
        for (int32_t k = 0; k < rank; ++k) {
            vs[it * rank + k] = factor_sd * rng_normal(&r);
            V0[it * rank + k] = (float)(factor_sd * rng_normal(&r0));
        }
    }
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n_ratings; ++i) {
        rng_t ru, ri, rn;
        rng_init(&ru, seed, ST_USER, (uint64_t)i);
        rng_init(&ri, seed, ST_ITEM, (uint64_t)i);
        rng_init(&rn, seed, ST_NOISE, (uint64_t)i);
        int64_t u = zipf_draw(&ru, cu, n_users), it = zipf_draw(&ri, ci, n_items);
        double dot = 0.0;
        for (int32_t k = 0; k < rank; ++k) dot += us[u * rank + k] * vs[it * rank + k];
        user[i] = (int32_t)u;
        item[i] = (int32_t)it;
        rating[i] = (float)(dot + noise_sd * rng_normal(&rn));
    }
    free(cu); free(ci); free(us); free(vs);
    return 0;
}

/* ---------------- dense examples ---------------- */
/* X (n x d, row stride ldx) with N(0,1) entries, drawn row by row; labels
 * from the hidden model w* (gen_wstar) through dot = <X_i, w*> / sqrt(d):
 * label_kind 0: sign(dot), flipped with probability label_p;
 * label_kind 1: dot + label_p * N(0,1). */
int gen_dense(uint64_t seed, int64_t n, int64_t d, int64_t ldx, int32_t label_kind,
              double label_p, float *X, float *y, int nthreads) {
    double *wstar = (double *)malloc((size_t)(d > 0 ? d : 1) * sizeof(double));
    if (!wstar) return -1;
    gen_wstar(seed, d, wstar, nthreads);
    const double scale = d > 0 ? 1.0 / sqrt((double)d) : 0.0;
    if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for schedule(dynamic, 16)
    for (int64_t i = 0; i < n; ++i) {
        rng_t r;
        rng_init(&r, seed, ST_DENSE, (uint64_t)i);
        float *x = X + i * ldx;
        double dot = 0.0;
        for (int64_t j = 0; j < d; ++j) {
            x[j] = (float)rng_normal(&r);
            dot += (double)x[j] * wstar[j];
        }
        dot *= scale;
        rng_t rl;
        rng_init(&rl, seed, ST_LABEL, (uint64_t)i);
        if (label_kind == 0) {
            float sg = (dot >= 0.0) ? 1.0f : -1.0f;
            if (rng_unif(&rl) < label_p) sg = -sg;
            y[i] = sg;
        } else {
            y[i] = (float)(dot + label_p * rng_normal(&rl));
        }
    }
    free(wstar);
    return 0;
}

/* uniform draws in (0,1) for tests of the distribution code */
void gen_uniform(uint64_t seed, uint32_t stream, int64_t count, double *out) {
    rng_t r;
    rng_init(&r, seed, stream, 0);
    for (int64_t i = 0; i < count; ++i) out[i] = rng_unif(&r);
}

void gen_zipf_sample(uint64_t seed, int64_t d, double alpha, int64_t count, int64_t *out) {
    double *cdf = gen_zipf_cdf(d, alpha);
    rng_t r;
    rng_init(&r, seed, 99, 0);
    for (int64_t i = 0; i < count; ++i) out[i] = zipf_draw(&r, cdf, d);
    free(cdf);
}

void gen_poisson_sample(uint64_t seed, double mu, int64_t count, int64_t *out) {
    rng_t r;
    rng_init(&r, seed, 98, 0);
    for (int64_t i = 0; i < count; ++i) out[i] = rng_poisson_ptrs(&r, mu);
}
