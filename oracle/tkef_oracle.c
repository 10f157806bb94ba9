/*
 * CPU oracle for exact top-k sparsification with error feedback and the
 * sparse aggregate + SGD update (test infrastructure only).
 *
 * This file is the plain, slow, obviously correct statement of what the GPU
 * library computes. Only the test suite, the smoke check and the CPU-baseline
 * leg of the benchmark use it; the product path never links or calls it. It
 * shares no code, header, table or constant with the GPU library.
 *
 * Precision: the paper represents every gradient element as a 32-bit float
 * (Sec. 3.2, All-Gather cost; Sec. 5.3 breakdown in FP32), so every
 * arithmetic step here is a single IEEE-754 binary32 operation with
 * round-to-nearest-even, exactly as written (x86-64 SSE arithmetic,
 * FLT_EVAL_METHOD == 0, compiled with -ffp-contract=off, no fast-math).
 *
 * Definitions followed:
 *  - TopK operator (Sec. 3.1, TopK definition): keep the elements whose
 *    magnitude reaches the k-th largest magnitude, zero the others. Read as
 *    "exactly k elements": order all positions by |x| descending and, among
 *    equal magnitudes, by position ascending; the first k are selected.
 *  - Sparse format (Sec. 3.2): k values and their k indices; k = rho * d,
 *    rounded up in double precision and clamped to [1, d].
 *  - The selected values are the entries of x itself, sign included
 *    (Alg. 1, the final gather of x at the selected indices).
 *  - Error feedback (not described in the paper; the residual memory of
 *    TopK-SGD): x = g + r; the residual keeps x where not selected and +0.0
 *    where selected.
 *  - Accumulation of the gathered sparse lists (Alg. 2, accumulate loop over
 *    p = 1..m into a zeroed dense vector) in worker order, then the SGD
 *    update of Eq. (1), w <- w - lr * sum_p g^p, optionally with weight decay
 *    and momentum (PyTorch SGD semantics, dampening 0, no Nesterov).
 */
#define _GNU_SOURCE
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_OK 0
#define ORC_EINVAL 1
#define ORC_ENAN 2
#define ORC_ENOMEM 3
#define ORC_ERANGE 4

int oracle_version(void) { return 1; }

/* k = ceil(rho * d) in double, clamped to [1, d]; 0 for d == 0; -1 for a
 * density outside (0, 1]. */
int64_t oracle_k_from_rho(int64_t d, double rho) {
    if (!(rho > 0.0 && rho <= 1.0) || d < 0) return -1;
    if (d == 0) return 0;
    double kd = ceil(rho * (double)d);
    int64_t k = (int64_t)kd;
    if (k < 1) k = 1;
    if (k > d) k = d;
    return k;
}

/* Residual add: x[i] = g[i] + r[i], one binary32 addition per element. */
void oracle_ef_add(const float *g, const float *r, float *x, int64_t n) {
    for (int64_t i = 0; i < n; ++i) x[i] = g[i] + r[i];
}

/* ---- exact top-k by full comparison sort -------------------------------- */

static int by_mag_desc_then_index(const void *pa, const void *pb, void *ctx) {
    const float *x = (const float *)ctx;
    int64_t a = *(const int64_t *)pa, b = *(const int64_t *)pb;
    float ma = fabsf(x[a]), mb = fabsf(x[b]);
    if (ma > mb) return -1;
    if (ma < mb) return 1;
    return (a < b) ? -1 : (a > b) ? 1 : 0;
}

static int by_index(const void *pa, const void *pb) {
    int64_t a = *(const int64_t *)pa, b = *(const int64_t *)pb;
    return (a < b) ? -1 : (a > b) ? 1 : 0;
}

/* Select the k positions of x (length n) that come first in the order
 * (|x| descending, index ascending) and write them in ascending order to
 * sel[0..k). NaN is rejected because it has no place in that order. */
int oracle_topk_select(const float *x, int64_t n, int64_t k, int64_t *sel) {
    if (n < 0 || k < 0 || k > n) return ORC_EINVAL;
    for (int64_t i = 0; i < n; ++i)
        if (isnan(x[i])) return ORC_ENAN;
    if (k == 0) return ORC_OK;
    int64_t *order = (int64_t *)malloc((size_t)n * sizeof(int64_t));
    if (!order) return ORC_ENOMEM;
    for (int64_t i = 0; i < n; ++i) order[i] = i;
    qsort_r(order, (size_t)n, sizeof(int64_t), by_mag_desc_then_index, (void *)x);
    memcpy(sel, order, (size_t)k * sizeof(int64_t));
    free(order);
    qsort(sel, (size_t)k, sizeof(int64_t), by_index);
    return ORC_OK;
}

/* One selection group: x = g + r; select k; emit (idx + index_base, x[idx]);
 * r_out = x with +0.0 at the selected positions. r_out may alias r. */
int oracle_sparsify(const float *g, const float *r, int64_t n, int64_t k,
                    int64_t index_base, int32_t *idx_out, float *val_out,
                    float *r_out) {
    if (n < 0 || k < 0 || k > n) return ORC_EINVAL;
    if (index_base < 0 || index_base + n > 2147483647LL) return ORC_ERANGE;
    float *x = (float *)malloc((size_t)(n > 0 ? n : 1) * sizeof(float));
    int64_t *sel = (int64_t *)malloc((size_t)(k > 0 ? k : 1) * sizeof(int64_t));
    if (!x || !sel) { free(x); free(sel); return ORC_ENOMEM; }
    oracle_ef_add(g, r, x, n);
    int rc = oracle_topk_select(x, n, k, sel);
    if (rc != ORC_OK) { free(x); free(sel); return rc; }
    for (int64_t j = 0; j < k; ++j) {
        idx_out[j] = (int32_t)(sel[j] + index_base);
        val_out[j] = x[sel[j]];
    }
    for (int64_t i = 0; i < n; ++i) r_out[i] = x[i];
    for (int64_t j = 0; j < k; ++j) r_out[sel[j]] = +0.0f;
    free(x);
    free(sel);
    return ORC_OK;
}

/* Rank of position i in the order (|x| descending, index ascending):
 * #{j : |x_j| > |x_i|} + #{j < i : |x_j| == |x_i|}. Position i is selected by
 * a top-k of x exactly when its rank is below k. */
int64_t oracle_rank(const float *x, int64_t n, int64_t i) {
    if (i < 0 || i >= n) return -1;
    float m = fabsf(x[i]);
    int64_t above = 0;
    for (int64_t j = 0; j < n; ++j) {
        float mj = fabsf(x[j]);
        if (mj > m || (mj == m && j < i)) ++above;
    }
    return above;
}

/* ---- aggregate + update -------------------------------------------------- */

/* Sparse lists in the gathered layout: worker p's entries are
 * idx[p*stride + j], val[p*stride + j] for j < nnz[p].
 * Step 1 (Alg. 2): G = 0; for p = 0..P-1 in order, for j in list order:
 *   G[idx] = G[idx] + val.
 * Step 2 (Eq. 1 and its momentum / weight-decay variant):
 *   mu == 0 and wd == 0: for every position that some list names,
 *       w = w - lr * G            (other positions untouched)
 *   otherwise, for every position:
 *       D = G + wd * w
 *       if mu != 0: b = mu * b + D; U = b   else U = D
 *       w = w - lr * U
 * Each operation above is one binary32 operation (no fused multiply-add). */
int oracle_update(float *w, float *b, int64_t d, int32_t P,
                  const int32_t *idx, const float *val, int64_t stride,
                  const int64_t *nnz, float lr, float mu, float wd) {
    if (d < 0 || P < 0 || stride < 0) return ORC_EINVAL;
    if (mu != 0.0f && b == NULL) return ORC_EINVAL;
    for (int32_t p = 0; p < P; ++p) {
        if (nnz[p] < 0 || nnz[p] > stride) return ORC_EINVAL;
        for (int64_t j = 0; j < nnz[p]; ++j) {
            int32_t i = idx[(int64_t)p * stride + j];
            if (i < 0 || (int64_t)i >= d) return ORC_ERANGE;
        }
    }
    float *G = (float *)calloc((size_t)(d > 0 ? d : 1), sizeof(float));
    unsigned char *touched = (unsigned char *)calloc((size_t)(d > 0 ? d : 1), 1);
    if (!G || !touched) { free(G); free(touched); return ORC_ENOMEM; }
    for (int32_t p = 0; p < P; ++p) {
        for (int64_t j = 0; j < nnz[p]; ++j) {
            int32_t i = idx[(int64_t)p * stride + j];
            G[i] = G[i] + val[(int64_t)p * stride + j];
            touched[i] = 1;
        }
    }
    if (mu == 0.0f && wd == 0.0f) {
        for (int64_t i = 0; i < d; ++i) {
            if (!touched[i]) continue;
            float step = lr * G[i];
            w[i] = w[i] - step;
        }
    } else {
        for (int64_t i = 0; i < d; ++i) {
            float decay = wd * w[i];
            float D = G[i] + decay;
            float U = D;
            if (mu != 0.0f) {
                float keep = mu * b[i];
                b[i] = keep + D;
                U = b[i];
            }
            float step = lr * U;
            w[i] = w[i] - step;
        }
    }
    free(G);
    free(touched);
    return ORC_OK;
}

/* Aggregation alone (Alg. 2, which returns the accumulated vector: g~ = 0,
 * then for p = 1..m in order: g~[iota_p] += kappa_p), written densely:
 * out[i] = the binary32 sum, in worker order, of the values that the lists
 * give position i; 0 where no list names i. */
int oracle_aggregate(float *out, int64_t d, int32_t P, const int32_t *idx,
                     const float *val, int64_t stride, const int64_t *nnz) {
    if (d < 0 || P < 0 || stride < 0) return ORC_EINVAL;
    for (int32_t q = 0; q < P; ++q) {
        if (nnz[q] < 0 || nnz[q] > stride) return ORC_EINVAL;
        for (int64_t j = 0; j < nnz[q]; ++j) {
            int32_t i = idx[(int64_t)q * stride + j];
            if (i < 0 || (int64_t)i >= d) return ORC_ERANGE;
        }
    }
    for (int64_t i = 0; i < d; ++i) out[i] = 0.0f;
    for (int32_t q = 0; q < P; ++q) {
        const int32_t *iq = idx + (int64_t)q * stride;
        const float *vq = val + (int64_t)q * stride;
        for (int64_t j = 0; j < nnz[q]; ++j) out[iq[j]] += vq[j];
    }
    return ORC_OK;
}
