/*
 * CPU oracle for sequentially-correct sparse SGD.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the
 * benchmark's CPU-baseline leg may load this library.  It shares no code,
 * header or constant table with the GPU library; it is a plain, slow,
 * single-threaded restatement of what the paper defines:
 *
 *   - Sequential computation (Algorithm 1, Definition 4): iterations run one
 *     after another; in each, every parameter the iteration touches is read,
 *     the update is computed, then the parameters are written.  With SGD one
 *     iteration is one training example (Sec. 6.3), and the gradient step is
 *     the scalar form of the gradient-descent update of Sec. 2.
 *   - Conflict levels: the read and write constraints (Sec. 4.4, Theorem 2)
 *     order only accesses to the same parameter partition.  With one feature
 *     per partition, example i must follow the most recent earlier example
 *     that touched any of its features.  level(i) = 1 + max level over those
 *     examples (0 when there is none); examples of equal level touch disjoint
 *     features and may run concurrently.
 *
 * Floating point is IEEE binary32, round to nearest, no flush to zero; fused
 * multiply-add appears only where fmaf() is written (build with
 * -ffp-contract=off).  Two summation orders exist for the dot product:
 *   natural: z = fmaf(w[c_k], x_k, z) for k = 0..m-1;
 *   matched: 64 partial sums, entry k goes to partial k mod 64, then a
 *            butterfly: for off = 1,2,4,8,16,32 every partial l becomes
 *            p[l] + p[l xor off]; z is the common final value.
 * The logistic function is 1/(1 + expf(-z)) in natural mode and, in matched
 * mode, orc_sigmoid below: the same with orc_exp (Cody-Waite range reduction
 * and the degree-7 Taylor polynomial of e^r, its coefficient pairs combined
 * by Horner's rule in r^2)
 * and the exponent argument capped at 87.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

enum { ORC_NATURAL = 0, ORC_MATCHED = 1 };
enum { ORC_LOGISTIC = 0, ORC_SQUARED = 1 };

/* ------------------------------------------------------------------------ */
/* exp(x) = 2^k * e^r with k = rint(x log2 e), r = x - k ln 2 (ln 2 split in
 * two floats so r carries the low bits), e^r by its Taylor series to r^7:
 * pairs c_j + c_{j+1} r, combined by Horner's rule in r^2
 * (p01 + r^2 (p23 + r^2 (p45 + r^2 p67))). */
float orc_exp(float x) {
    if (x != x) return x;
    if (x > 89.0f) return INFINITY;
    if (x < -104.0f) return 0.0f;
    const float log2e = 0x1.715476p+0f;
    const float ln2_hi = 0x1.62e430p-1f;
    const float ln2_lo = -0x1.05c610p-29f;
    float k = rintf(x * log2e);
    float r = fmaf(-k, ln2_hi, x);
    r = fmaf(-k, ln2_lo, r);
    /* c_j = 1/j! rounded to binary32 */
    const float c0 = 1.0f, c1 = 1.0f, c2 = 0.5f, c3 = 0x1.555556p-3f;
    const float c4 = 0x1.555556p-5f, c5 = 0x1.111112p-7f, c6 = 0x1.6c16c2p-10f,
                c7 = 0x1.a01a02p-13f;
    float r2 = r * r;
    float p01 = fmaf(c1, r, c0), p23 = fmaf(c3, r, c2);
    float p45 = fmaf(c5, r, c4), p67 = fmaf(c7, r, c6);
    float q = fmaf(fmaf(fmaf(p67, r2, p45), r2, p23), r2, p01);
    int ki = (int)k;
    float two_k;
    if (ki > 127) {
        /* q * 2^127 is exact; the second product overflows or not by itself */
        uint32_t b127 = (uint32_t)(127 + 127) << 23, b1 = (uint32_t)(ki - 127 + 127) << 23;
        float s127, s1;
        memcpy(&s127, &b127, 4);
        memcpy(&s1, &b1, 4);
        return (q * s127) * s1;
    }
    if (ki < -126) {
        /* q * 2^(k+126) is exact and normal; one rounding into the subnormals */
        uint32_t ba = (uint32_t)(ki + 126 + 127) << 23, bb = (uint32_t)(-126 + 127) << 23;
        float sa, sb;
        memcpy(&sa, &ba, 4);
        memcpy(&sb, &bb, 4);
        return (q * sa) * sb;
    }
    uint32_t bk = (uint32_t)(ki + 127) << 23;
    memcpy(&two_k, &bk, 4);
    return q * two_k;
}

/* ------------------------------------------------------------------------ */
/* Conflict levels                                                          */

static int rows_share_feature(const int64_t *row_ptr, const int32_t *col, int64_t a, int64_t b) {
    /* columns of a row are sorted ascending: merge */
    int64_t p = row_ptr[a], pe = row_ptr[a + 1], q = row_ptr[b], qe = row_ptr[b + 1];
    while (p < pe && q < qe) {
        if (col[p] == col[q]) return 1;
        if (col[p] < col[q]) ++p; else ++q;
    }
    return 0;
}

/* Brute force from the definition: level(i) = 1 + max{ level(j) : j < i, S(j) and S(i)
 * intersect }, max of the empty set = 0.  O(n^2 m); tiny inputs only. */
int32_t orc_levels_brute(int64_t n, const int64_t *row_ptr, const int32_t *col, int32_t *level) {
    int32_t L = 0;
    for (int64_t i = 0; i < n; ++i) {
        int32_t lv = 1;
        for (int64_t j = 0; j < i; ++j)
            if (level[j] + 1 > lv && rows_share_feature(row_ptr, col, j, i)) lv = level[j] + 1;
        level[i] = lv;
        if (lv > L) L = lv;
    }
    return L;
}

/* One pass in example order.  last[f] = level of the latest example so far
 * that touched feature f (0 if none).  Returns L = max level, -1 on failure. */
int32_t orc_levels_seq(int64_t n, int64_t d, const int64_t *row_ptr, const int32_t *col,
                       int32_t *level) {
    int32_t *last = (int32_t *)calloc((size_t)(d > 0 ? d : 1), sizeof(int32_t));
    if (!last) return -1;
    int32_t L = 0;
    for (int64_t i = 0; i < n; ++i) {
        int32_t lv = 0;
        for (int64_t p = row_ptr[i]; p < row_ptr[i + 1]; ++p)
            if (last[col[p]] > lv) lv = last[col[p]];
        lv += 1;
        for (int64_t p = row_ptr[i]; p < row_ptr[i + 1]; ++p) last[col[p]] = lv;
        level[i] = lv;
        if (lv > L) L = lv;
    }
    free(last);
    return L;
}

/* Examples grouped by level, ascending index inside a level.
 * level_ptr[l] = number of examples with level <= l, l = 0..L. */
int orc_bucket(int64_t n, const int32_t *level, int32_t L, int32_t *perm, int64_t *level_ptr) {
    memset(level_ptr, 0, (size_t)(L + 1) * sizeof(int64_t));
    for (int64_t i = 0; i < n; ++i) {
        if (level[i] < 1 || level[i] > L) return -1;
        level_ptr[level[i]] += 1;
    }
    for (int32_t l = 1; l <= L; ++l) level_ptr[l] += level_ptr[l - 1];
    int64_t *next = (int64_t *)malloc((size_t)(L + 1) * sizeof(int64_t));
    if (!next) return -1;
    for (int32_t l = 1; l <= L; ++l) next[l] = level_ptr[l - 1];
    for (int64_t i = 0; i < n; ++i) perm[next[level[i]]++] = (int32_t)i;
    free(next);
    return 0;
}

/* For every stored entry (CSR order): the latest earlier example that touched
 * the same feature, or -1. */
int orc_prev_writer(int64_t n, int64_t d, const int64_t *row_ptr, const int32_t *col,
                    int32_t *prev_row) {
    int32_t *last = (int32_t *)malloc((size_t)(d > 0 ? d : 1) * sizeof(int32_t));
    if (!last) return -1;
    for (int64_t f = 0; f < d; ++f) last[f] = -1;
    for (int64_t i = 0; i < n; ++i) {
        for (int64_t p = row_ptr[i]; p < row_ptr[i + 1]; ++p) prev_row[p] = last[col[p]];
        for (int64_t p = row_ptr[i]; p < row_ptr[i + 1]; ++p) last[col[p]] = (int32_t)i;
    }
    free(last);
    return 0;
}

/* Per-feature occurrence lists (CSC): col_ptr[d+1], rows ascending per feature. */
int orc_transpose(int64_t n, int64_t d, const int64_t *row_ptr, const int32_t *col,
                  int64_t *col_ptr, int32_t *csc_row) {
    memset(col_ptr, 0, (size_t)(d + 1) * sizeof(int64_t));
    int64_t nnz = row_ptr[n];
    for (int64_t p = 0; p < nnz; ++p) col_ptr[col[p] + 1] += 1;
    for (int64_t f = 0; f < d; ++f) col_ptr[f + 1] += col_ptr[f];
    int64_t *next = (int64_t *)malloc((size_t)(d > 0 ? d : 1) * sizeof(int64_t));
    if (!next) return -1;
    memcpy(next, col_ptr, (size_t)d * sizeof(int64_t));
    for (int64_t i = 0; i < n; ++i)
        for (int64_t p = row_ptr[i]; p < row_ptr[i + 1]; ++p) csc_row[next[col[p]]++] = (int32_t)i;
    free(next);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Sequential SGD                                                           */

static float dot_natural(const float *w, const int32_t *c, const float *v, int64_t m) {
    float z = 0.0f;
    for (int64_t k = 0; k < m; ++k) z = fmaf(w[c[k]], v ? v[k] : 1.0f, z);
    return z;
}

static float butterfly64(float *acc, int width) {
    float nxt[64];
    for (int off = 1; off < width; off *= 2) {
        for (int l = 0; l < width; ++l) nxt[l] = acc[l] + acc[l ^ off];
        memcpy(acc, nxt, (size_t)width * sizeof(float));
    }
    return acc[0];
}

/* The logistic function in matched mode: 1 / (1 + exp(x)) with x = -z
 * capped at 87 (NaN stays NaN).  Below the cap this is the logistic function
 * itself, with orc_exp and one correctly rounded division; for z < -87 it is
 * 1/(1 + e^87) ~ 1.6e-38 instead of a smaller value, so that 1 + e stays
 * below 2^126 and the quotient is a normal number. */
float orc_sigmoid(float z) {
    float x = -z;
    if (x > 87.0f) x = 87.0f;
    return 1.0f / (1.0f + orc_exp(x));
}

static float dot_matched(const float *w, const int32_t *c, const float *v, int64_t m) {
    float acc[64];
    for (int l = 0; l < 64; ++l) acc[l] = 0.0f;
    for (int64_t k = 0; k < m; ++k) acc[k & 63] = fmaf(w[c[k]], v ? v[k] : 1.0f, acc[k & 63]);
    return butterfly64(acc, 64);
}

/* One SGD step per example, examples taken in the given order (NULL: index
 * order 0..n-1, which is Algorithm 1).  Per example i with entries (c_k, x_k):
 *   z = <w, x_i>;  logistic: g = sigma(z) - [y_i > 0];  squared: g = z - y_i
 *   s = lr * g;    w[c_k] <- fmaf(-s, x_k, w[c_k])  (all reads before any write). */
void orc_sgd_apply(int64_t count, const int32_t *order, const int64_t *row_ptr,
                   const int32_t *col, const float *val, const float *y, float *w, float lr,
                   int32_t loss, int32_t mode) {
    for (int64_t t = 0; t < count; ++t) {
        int64_t i = order ? order[t] : t;
        int64_t b = row_ptr[i], m = row_ptr[i + 1] - b;
        const int32_t *c = col + b;
        const float *v = val ? val + b : NULL;
        float z = (mode == ORC_MATCHED) ? dot_matched(w, c, v, m) : dot_natural(w, c, v, m);
        float g;
        if (loss == ORC_LOGISTIC) {
            float sig = (mode == ORC_MATCHED) ? orc_sigmoid(z) : 1.0f / (1.0f + expf(-z));
            g = sig - ((y[i] > 0.0f) ? 1.0f : 0.0f);
        } else {
            g = z - y[i];
        }
        float s = lr * g;
        /* the new values depend only on values read before any write: the
         * columns of a row are distinct, so writing in place is the same */
        for (int64_t k = 0; k < m; ++k) w[c[k]] = fmaf(-s, v ? v[k] : 1.0f, w[c[k]]);
    }
}

/* Matrix completion, one rating per iteration:
 *   e = r - <U_u, V_i>
 *   U_u <- U_u + lr (e V_i - reg U_u),  V_i <- V_i + lr (e U_u - reg V_i)
 * with both right-hand sides using the values read before the step (the L2
 * regulariser of Eq. 2 applied to the two touched rows). */
void orc_mf_apply(int64_t count, const int32_t *order, const int32_t *user, const int32_t *item,
                  const float *rating, float *U, float *V, int32_t rank, float lr, float reg,
                  int32_t mode) {
    float acc[64];
    for (int64_t t = 0; t < count; ++t) {
        int64_t i = order ? order[t] : t;
        float *u = U + (int64_t)user[i] * rank;
        float *v = V + (int64_t)item[i] * rank;
        float dot;
        if (mode == ORC_MATCHED) {
            for (int l = 0; l < rank; ++l) acc[l] = fmaf(u[l], v[l], 0.0f);
            dot = butterfly64(acc, rank);
        } else {
            dot = 0.0f;
            for (int l = 0; l < rank; ++l) dot = fmaf(u[l], v[l], dot);
        }
        float e = rating[i] - dot;
        for (int l = 0; l < rank; ++l) {
            float ul = u[l], vl = v[l];
            float a = e * vl, b = reg * ul;
            float a2 = e * ul, b2 = reg * vl;
            u[l] = fmaf(lr, a - b, ul);
            v[l] = fmaf(lr, a2 - b2, vl);
        }
    }
}

/* ------------------------------------------------------------------------ */
/* Mini-batch gradient descent (Sec. 6.3: gradient descent with a batch of a
 * fixed number of examples per iteration).  Batch b is examples
 * [b*B, min((b+1)*B, n)); its parameter set is the union of its examples'
 * features.  Within an iteration every read precedes every write
 * (Definition 3), so all examples of a batch see the weights as they were
 * when the batch started.  The step is the gradient step of Sec. 2 on the
 * batch's part of h, i.e. the sum of its examples' losses:
 *   w_f <- w_f - lr * sum_{i in b} g_i x_if,
 * evaluated as s_i = lr * g_i, then for each example in index order and each
 * of its entries w[c] = fmaf(-s_i, x, w[c]).  With B = 1 this is the SGD step
 * above, bit for bit. */

static int batches_share_feature(const int64_t *row_ptr, const int32_t *col, int64_t n,
                                 int64_t B, int64_t a, int64_t b) {
    int64_t ae = (a + 1) * B < n ? (a + 1) * B : n, be = (b + 1) * B < n ? (b + 1) * B : n;
    for (int64_t i = a * B; i < ae; ++i)
        for (int64_t j = b * B; j < be; ++j)
            if (rows_share_feature(row_ptr, col, i, j)) return 1;
    return 0;
}

/* From the definition: level(b) = 1 + max{ level(a) : a < b, batches a and b
 * share a feature }, max of the empty set = 0.  Tiny inputs only. */
int32_t orc_batch_levels_brute(int64_t n, const int64_t *row_ptr, const int32_t *col, int64_t B,
                               int32_t *level) {
    int64_t nb = (n + B - 1) / B;
    int32_t L = 0;
    for (int64_t b = 0; b < nb; ++b) {
        int32_t lv = 1;
        for (int64_t a = 0; a < b; ++a)
            if (level[a] + 1 > lv && batches_share_feature(row_ptr, col, n, B, a, b)) lv = level[a] + 1;
        level[b] = lv;
        if (lv > L) L = lv;
    }
    return L;
}

/* One pass in batch order with last[f] = level of the latest batch that
 * touched f.  Returns L, -1 on failure. */
int32_t orc_batch_levels_seq(int64_t n, int64_t d, const int64_t *row_ptr, const int32_t *col,
                             int64_t B, int32_t *level) {
    int32_t *last = (int32_t *)calloc((size_t)(d > 0 ? d : 1), sizeof(int32_t));
    if (!last) return -1;
    int64_t nb = (n + B - 1) / B;
    int32_t L = 0;
    for (int64_t b = 0; b < nb; ++b) {
        int64_t p0 = row_ptr[b * B], p1 = row_ptr[(b + 1) * B < n ? (b + 1) * B : n];
        int32_t lv = 0;
        for (int64_t p = p0; p < p1; ++p)
            if (last[col[p]] > lv) lv = last[col[p]];
        lv += 1;
        for (int64_t p = p0; p < p1; ++p) last[col[p]] = lv;
        level[b] = lv;
        if (lv > L) L = lv;
    }
    free(last);
    return L;
}

static int cmp_i32(const void *a, const void *b) {
    int32_t x = *(const int32_t *)a, y = *(const int32_t *)b;
    return (x > y) - (x < y);
}

/* Per batch, the union of its features in ascending order, and for each
 * union feature the batch's entries on it in example order:
 *   batch b's union entries are u in [bptr[b], bptr[b+1]), ucol[u] = feature,
 *   occurrences occ[uptr[u] .. uptr[u+1]) are CSR entry indices.
 * bptr [nb+1], ucol [nnz], uptr [nnz+1], occ [nnz].  Per batch: the distinct
 * features, sorted; then a counting sort of the batch's entries by feature,
 * which keeps each feature's entries in CSR (= example) order.
 * Returns the union size U, -1 on failure. */
int64_t orc_batch_union(int64_t n, int64_t d, const int64_t *row_ptr, const int32_t *col,
                        int64_t B, int64_t *bptr, int32_t *ucol, int64_t *uptr, int32_t *occ) {
    int64_t *next = (int64_t *)malloc((size_t)(d > 0 ? d : 1) * sizeof(int64_t));
    if (!next) return -1;
    for (int64_t f = 0; f < d; ++f) next[f] = -1;
    int64_t nb = (n + B - 1) / B, U = 0;
    for (int64_t b = 0; b < nb; ++b) {
        int64_t p0 = row_ptr[b * B], p1 = row_ptr[(b + 1) * B < n ? (b + 1) * B : n];
        bptr[b] = U;
        /* distinct features of the batch (next[f] = 0 marks "seen") */
        int64_t u0 = U;
        for (int64_t p = p0; p < p1; ++p)
            if (next[col[p]] < 0) {
                next[col[p]] = 0;
                ucol[U++] = col[p];
            }
        qsort(ucol + u0, (size_t)(U - u0), sizeof(int32_t), cmp_i32);
        /* occurrence counts, then each feature's first slot */
        for (int64_t p = p0; p < p1; ++p) next[col[p]] += 1;
        int64_t pos = p0;
        for (int64_t u = u0; u < U; ++u) {
            int64_t c = next[ucol[u]];
            uptr[u] = pos;
            next[ucol[u]] = pos;
            pos += c;
        }
        for (int64_t p = p0; p < p1; ++p) occ[next[col[p]]++] = (int32_t)p;
        for (int64_t u = u0; u < U; ++u) next[ucol[u]] = -1;
    }
    bptr[nb] = U;
    uptr[U] = row_ptr[n];
    free(next);
    return U;
}

/* One epoch of mini-batch gradient descent, batches taken in the given order
 * (NULL: 0..nb-1, the sequential computation).  Returns 0, -1 on failure. */
int orc_batch_apply(int64_t n, int64_t count, const int32_t *order, const int64_t *row_ptr,
                    const int32_t *col, const float *val, const float *y, float *w, float lr,
                    int32_t loss, int32_t mode, int64_t B) {
    float *s = (float *)malloc((size_t)(B > 0 ? B : 1) * sizeof(float));
    if (!s) return -1;
    for (int64_t t = 0; t < count; ++t) {
        int64_t b = order ? order[t] : t;
        int64_t i0 = b * B, i1 = (b + 1) * B < n ? (b + 1) * B : n;
        /* reads: every example of the batch against the batch-start weights */
        for (int64_t i = i0; i < i1; ++i) {
            int64_t p = row_ptr[i], m = row_ptr[i + 1] - p;
            const float *v = val ? val + p : NULL;
            float z = (mode == ORC_MATCHED) ? dot_matched(w, col + p, v, m)
                                            : dot_natural(w, col + p, v, m);
            float g;
            if (loss == ORC_LOGISTIC) {
                float sig = (mode == ORC_MATCHED) ? orc_sigmoid(z) : 1.0f / (1.0f + expf(-z));
                g = sig - ((y[i] > 0.0f) ? 1.0f : 0.0f);
            } else {
                g = z - y[i];
            }
            s[i - i0] = lr * g;
        }
        /* writes: each feature's contributions in example order */
        for (int64_t i = i0; i < i1; ++i)
            for (int64_t p = row_ptr[i]; p < row_ptr[i + 1]; ++p)
                w[col[p]] = fmaf(-s[i - i0], val ? val[p] : 1.0f, w[col[p]]);
    }
    free(s);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Bounded delay (Sec. 7): an iteration may read a partition once the write
 * of iteration alpha - 1 - delta to it is done (Asynchronous Read
 * Constraint); it need not wait for the writes of the delta iterations before
 * it.  The deterministic execution taken here reads as early as that allows:
 * example alpha computes z against the weights as they were after examples
 * 0 .. alpha - delta - 1, and every example's update is applied in example
 * order to each of its features, w_f = fmaf(-s, x, w_f), so no update is
 * lost.  delay = 0 is the sequential computation; delay >= n - 1 computes
 * every z at the initial weights. */

/* Literal form, tiny inputs: W[a] is the whole weight vector after examples
 * 0 .. a-1 (W[0] = w0); z_a uses W[max(0, a - delay)].  Needs
 * (n + 1) * d floats.  w receives W[n].  Returns 0, -1 on failure. */
int orc_stale_snapshot(int64_t n, int64_t d, const int64_t *row_ptr, const int32_t *col,
                       const float *val, const float *y, float *w, float lr, int32_t loss,
                       int32_t mode, int64_t delay) {
    float *W = (float *)malloc((size_t)(n + 1) * (size_t)(d > 0 ? d : 1) * sizeof(float));
    if (!W) return -1;
    memcpy(W, w, (size_t)d * sizeof(float));
    for (int64_t a = 0; a < n; ++a) {
        const float *R = W + (size_t)(a - delay > 0 ? a - delay : 0) * (size_t)d;
        float *cur = W + (size_t)a * (size_t)d, *nxt = W + (size_t)(a + 1) * (size_t)d;
        int64_t p = row_ptr[a], m = row_ptr[a + 1] - p;
        const float *v = val ? val + p : NULL;
        float z = (mode == ORC_MATCHED) ? dot_matched(R, col + p, v, m) : dot_natural(R, col + p, v, m);
        float g;
        if (loss == ORC_LOGISTIC) {
            float sig = (mode == ORC_MATCHED) ? orc_sigmoid(z) : 1.0f / (1.0f + expf(-z));
            g = sig - ((y[a] > 0.0f) ? 1.0f : 0.0f);
        } else {
            g = z - y[a];
        }
        float s = lr * g;
        memcpy(nxt, cur, (size_t)d * sizeof(float));
        for (int64_t k = 0; k < m; ++k) nxt[col[p + k]] = fmaf(-s, v ? v[k] : 1.0f, cur[col[p + k]]);
    }
    memcpy(w, W + (size_t)n * (size_t)d, (size_t)d * sizeof(float));
    free(W);
    return 0;
}

/* The same with one written value per stored entry: V[q] is the value entry q
 * wrote.  Entry q of example a reads the value of the latest earlier entry on
 * its feature whose example is below a - delay (found by walking the
 * previous-entry links back), w0 if there is none; it writes
 * fmaf(-s, x_q, value of its previous entry, or w0).  w receives each
 * feature's last written value.  Returns 0, -1 on failure. */
int orc_stale_apply(int64_t n, int64_t d, const int64_t *row_ptr, const int32_t *col,
                    const float *val, const float *y, float *w, float lr, int32_t loss,
                    int32_t mode, int64_t delay) {
    int64_t nnz = row_ptr[n];
    int64_t *prev = (int64_t *)malloc((size_t)(nnz > 0 ? nnz : 1) * sizeof(int64_t));
    int64_t *last = (int64_t *)malloc((size_t)(d > 0 ? d : 1) * sizeof(int64_t));
    float *V = (float *)malloc((size_t)(nnz > 0 ? nnz : 1) * sizeof(float));
    float *rv = (float *)malloc((size_t)(nnz > 0 ? nnz : 1) * sizeof(float));
    if (!prev || !last || !V || !rv) {
        free(prev); free(last); free(V); free(rv);
        return -1;
    }
    for (int64_t f = 0; f < d; ++f) last[f] = -1;
    for (int64_t q = 0; q < nnz; ++q) {
        prev[q] = last[col[q]];
        last[col[q]] = q;
    }
    for (int64_t a = 0; a < n; ++a) {
        int64_t p = row_ptr[a], m = row_ptr[a + 1] - p;
        /* entries of examples a - delay .. a - 1 start at row_ptr[a - delay] */
        int64_t lim = a - delay > 0 ? row_ptr[a - delay] : INT64_MAX;
        for (int64_t k = 0; k < m; ++k) {
            int64_t q = prev[p + k];
            if (lim == INT64_MAX) q = -1;
            while (q >= 0 && q >= lim) q = prev[q];
            rv[k] = q >= 0 ? V[q] : w[col[p + k]];
        }
        /* the reads gathered, the dot product as for a weight vector */
        float z = 0.0f;
        if (mode == ORC_MATCHED) {
            float acc[64];
            for (int l = 0; l < 64; ++l) acc[l] = 0.0f;
            for (int64_t k = 0; k < m; ++k)
                acc[k & 63] = fmaf(rv[k], val ? val[p + k] : 1.0f, acc[k & 63]);
            z = butterfly64(acc, 64);
        } else {
            for (int64_t k = 0; k < m; ++k) z = fmaf(rv[k], val ? val[p + k] : 1.0f, z);
        }
        float g;
        if (loss == ORC_LOGISTIC) {
            float sig = (mode == ORC_MATCHED) ? orc_sigmoid(z) : 1.0f / (1.0f + expf(-z));
            g = sig - ((y[a] > 0.0f) ? 1.0f : 0.0f);
        } else {
            g = z - y[a];
        }
        float s = lr * g;
        for (int64_t k = 0; k < m; ++k) {
            int64_t q = prev[p + k];
            float cur = q >= 0 ? V[q] : w[col[p + k]];
            V[p + k] = fmaf(-s, val ? val[p + k] : 1.0f, cur);
        }
    }
    for (int64_t f = 0; f < d; ++f)
        if (last[f] >= 0) w[f] = V[last[f]];
    free(prev); free(last); free(V); free(rv);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Dense full-batch gradient descent: the update of Sec. 2 with every
 * example in every iteration (the dense linear-regression workloads of
 * Sec. 6.1-6.2).  X is n x d, row-major with row stride ldx.  One iteration,
 * all reads from the weights before it (the scalar form of Sec. 2):
 *   z_i = <X_i, w>;  s_i = lr * g(z_i, y_i);  G_j = sum_i s_i X_ij;
 *   w_j <- w_j - G_j.
 * natural: z_i = fmaf(X_ij, w_j, z) over j = 0..d-1 from 0, and
 *          G_j = fmaf(s_i, X_ij, G) over i = 0..n-1 from 0.
 * matched: rows in blocks of row_block, columns in blocks of col_block.
 *   The partial dot of a column block has 64 partial sums; column k of the
 *   block (k from 0) goes into sum (k / 4) mod 64, in increasing k, then the
 *   butterfly; z_i adds the blocks' partials in block order, starting from
 *   block 0's.  A row block is cut into chunks of row_chunk rows; a chunk's
 *   partial of G_j is fmaf over its rows in order from 0, the row block's
 *   partial adds its chunks' partials in order (starting from the first's),
 *   and G_j adds the row blocks' partials in block order (starting from
 *   block 0's).
 * Returns 0, -1 on failure (bad blocking or no memory). */
static float residual(float z, float y, int32_t loss, int32_t mode) {
    if (loss == ORC_LOGISTIC) {
        float sig = (mode == ORC_MATCHED) ? orc_sigmoid(z) : 1.0f / (1.0f + expf(-z));
        return sig - ((y > 0.0f) ? 1.0f : 0.0f);
    }
    return z - y;
}

int orc_dense_gd(int64_t n, int64_t d, const float *X, int64_t ldx, const float *y, float *w,
                 float lr, int32_t loss, int32_t mode, int64_t iters, int64_t row_block,
                 int64_t col_block, int64_t row_chunk) {
    if (mode == ORC_MATCHED && (row_block < 1 || col_block < 1 || row_chunk < 1)) return -1;
    float *s = (float *)malloc((size_t)(n > 0 ? n : 1) * sizeof(float));
    float *G = (float *)malloc((size_t)(d > 0 ? d : 1) * sizeof(float));
    if (!s || !G) {
        free(s); free(G);
        return -1;
    }
    for (int64_t t = 0; t < iters; ++t) {
        for (int64_t i = 0; i < n; ++i) {
            const float *x = X + i * ldx;
            float z = 0.0f;
            if (mode == ORC_MATCHED) {
                for (int64_t c0 = 0; c0 < d; c0 += col_block) {
                    int64_t c1 = c0 + col_block < d ? c0 + col_block : d;
                    float acc[64];
                    for (int l = 0; l < 64; ++l) acc[l] = 0.0f;
                    for (int64_t k = 0; k < c1 - c0; ++k)
                        acc[(k >> 2) & 63] = fmaf(x[c0 + k], w[c0 + k], acc[(k >> 2) & 63]);
                    float part = butterfly64(acc, 64);
                    z = (c0 == 0) ? part : z + part;
                }
            } else {
                for (int64_t j = 0; j < d; ++j) z = fmaf(x[j], w[j], z);
            }
            s[i] = lr * residual(z, y[i], loss, mode);
        }
        for (int64_t j = 0; j < d; ++j) {
            float g = 0.0f;
            if (mode == ORC_MATCHED) {
                for (int64_t r0 = 0; r0 < n; r0 += row_block) {
                    int64_t r1 = r0 + row_block < n ? r0 + row_block : n;
                    float part = 0.0f;
                    for (int64_t h0 = r0; h0 < r1; h0 += row_chunk) {
                        int64_t h1 = h0 + row_chunk < r1 ? h0 + row_chunk : r1;
                        float chunk = 0.0f;
                        for (int64_t i = h0; i < h1; ++i) chunk = fmaf(s[i], X[i * ldx + j], chunk);
                        part = (h0 == r0) ? chunk : part + chunk;
                    }
                    g = (r0 == 0) ? part : g + part;
                }
            } else {
                for (int64_t i = 0; i < n; ++i) g = fmaf(s[i], X[i * ldx + j], g);
            }
            G[j] = g;
        }
        for (int64_t j = 0; j < d; ++j) w[j] = w[j] - G[j];
    }
    free(s); free(G);
    return 0;
}
