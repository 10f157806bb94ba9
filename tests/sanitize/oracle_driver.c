/*
 * Driver of the C oracle (oracle/tkef_oracle.c) for AddressSanitizer /
 * UndefinedBehaviorSanitizer builds. It runs the oracle's functions over
 * small seeded inputs (ties, signed zeros, infinities, subnormals, every k
 * from 0 to n, empty inputs, repeated indices, error paths) and checks the
 * results against the rank definition (a position is selected exactly when
 * its rank is below k) and a few identities. Exit status: the number of
 * failed checks.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

/* the oracle's entry points (it has no header: nothing is shared with it) */
int64_t oracle_k_from_rho(int64_t d, double rho);
void oracle_ef_add(const float *g, const float *r, float *x, int64_t n);
int oracle_topk_select(const float *x, int64_t n, int64_t k, int64_t *sel);
int oracle_sparsify(const float *g, const float *r, int64_t n, int64_t k, int64_t index_base,
                    int32_t *idx_out, float *val_out, float *r_out);
int64_t oracle_rank(const float *x, int64_t n, int64_t i);
int oracle_update(float *w, float *b, int64_t d, int32_t P, const int32_t *idx,
                  const float *val, int64_t stride, const int64_t *nnz, float lr, float mu,
                  float wd);
int oracle_aggregate(float *out, int64_t d, int32_t P, const int32_t *idx, const float *val,
                     int64_t stride, const int64_t *nnz);

static int fails = 0;
#define CHECK(e)                                                           \
    do {                                                                   \
        if (!(e)) {                                                        \
            fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #e); \
            ++fails;                                                       \
        }                                                                  \
    } while (0)

static uint64_t state = 0x9E3779B97F4A7C15ull;
static uint32_t next32(void) {
    state ^= state << 13;
    state ^= state >> 7;
    state ^= state << 17;
    return (uint32_t)(state >> 32);
}

/* values drawn from a small alphabet so that ties are common */
static float draw(int kind) {
    static const float alphabet[] = {0.0f, -0.0f, 1.0f, -1.0f, 0.5f, -2.0f, 3.0e-39f,
                                     -3.0e-39f, 1.0e30f, INFINITY, -INFINITY, 7.25f};
    if (kind == 0) return alphabet[next32() % (sizeof alphabet / sizeof alphabet[0])];
    return ((float)(int32_t)next32()) * 1e-9f;
}

static void selection_cases(void) {
    for (int trial = 0; trial < 300; ++trial) {
        const int64_t n = (int64_t)(next32() % 40);
        const int kind = trial % 2;
        float *g = malloc((size_t)(n + 1) * sizeof(float));
        float *r = malloc((size_t)(n + 1) * sizeof(float));
        float *x = malloc((size_t)(n + 1) * sizeof(float));
        float *ro = malloc((size_t)(n + 1) * sizeof(float));
        int64_t *sel = malloc((size_t)(n + 1) * sizeof(int64_t));
        int32_t *idx = malloc((size_t)(n + 1) * sizeof(int32_t));
        float *val = malloc((size_t)(n + 1) * sizeof(float));
        for (int64_t i = 0; i < n; ++i) {
            g[i] = draw(kind);
            r[i] = (next32() % 3 == 0) ? draw(kind) : 0.0f;
        }
        oracle_ef_add(g, r, x, n);
        for (int64_t k = 0; k <= n; ++k) {
            int rc = oracle_topk_select(x, n, k, sel);
            int has_nan = 0;
            for (int64_t i = 0; i < n; ++i) has_nan |= isnan(x[i]);
            if (has_nan) {
                CHECK(rc == 2);
                continue;
            }
            CHECK(rc == 0);
            /* ascending, and exactly the positions of rank < k */
            int64_t j = 0;
            for (int64_t i = 0; i < n; ++i) {
                const int chosen = j < k && sel[j] == i;
                CHECK(chosen == (oracle_rank(x, n, i) < k));
                if (chosen) ++j;
            }
            CHECK(j == k);
            rc = oracle_sparsify(g, r, n, k, 1000, idx, val, ro);
            CHECK(rc == 0);
            for (int64_t q = 0; q < k; ++q) {
                CHECK(idx[q] == (int32_t)(sel[q] + 1000));
                CHECK(memcmp(&val[q], &x[sel[q]], sizeof(float)) == 0);
                CHECK(ro[sel[q]] == 0.0f && !signbit(ro[sel[q]]));
            }
        }
        CHECK(oracle_topk_select(x, n, n + 1, sel) == 1);
        CHECK(oracle_topk_select(x, n, -1, sel) == 1);
        CHECK(oracle_rank(x, n, n) == -1);
        free(g); free(r); free(x); free(ro); free(sel); free(idx); free(val);
    }
    float one = 1.0f;
    int32_t idx1;
    float v1, r1;
    CHECK(oracle_sparsify(&one, &one, 1, 1, 2147483647LL, &idx1, &v1, &r1) == 4);
    CHECK(oracle_sparsify(&one, &one, 1, 1, -1, &idx1, &v1, &r1) == 4);
}

static void update_cases(void) {
    enum { D = 64, P = 5, S = 12 };
    int32_t idx[P * S];
    float val[P * S];
    int64_t nnz[P] = {12, 0, 7, 12, 1};
    for (int p = 0; p < P; ++p) {
        int32_t cur = 0;
        for (int j = 0; j < S; ++j) {
            cur += (int32_t)(next32() % 3);   /* ascending, repeats allowed */
            idx[p * S + j] = cur < D ? cur : D - 1;
            val[p * S + j] = (float)((int)(next32() % 17) - 8) * 0.25f;
        }
    }
    float G[D], w[D], b[D], w2[D];
    CHECK(oracle_aggregate(G, D, P, idx, val, S, nnz) == 0);
    /* dyadic values: the sum is exact, so any order must give it */
    for (int i = 0; i < D; ++i) {
        double s = 0.0;
        for (int p = 0; p < P; ++p)
            for (int64_t j = 0; j < nnz[p]; ++j)
                if (idx[p * S + j] == i) s += val[p * S + j];
        CHECK((double)G[i] == s);
    }
    for (int i = 0; i < D; ++i) {
        w[i] = w2[i] = (float)i * 0.125f;
        b[i] = 0.0f;
    }
    CHECK(oracle_update(w, b, D, P, idx, val, S, nnz, 0.5f, 0.5f, 0.0f) == 0);
    for (int i = 0; i < D; ++i) CHECK(w[i] == w2[i] - 0.5f * G[i] && b[i] == G[i]);
    CHECK(oracle_update(w2, NULL, D, P, idx, val, S, nnz, 0.5f, 0.0f, 0.0f) == 0);
    CHECK(oracle_update(w2, NULL, D, P, idx, val, S, nnz, 0.5f, 0.9f, 0.0f) == 1);
    nnz[1] = 13;
    CHECK(oracle_aggregate(G, D, P, idx, val, S, nnz) == 1);
    nnz[1] = 0;
    idx[3] = D;
    CHECK(oracle_aggregate(G, D, P, idx, val, S, nnz) == 4);
    CHECK(oracle_update(w, b, D, P, idx, val, S, nnz, 0.5f, 0.5f, 0.0f) == 4);
    CHECK(oracle_aggregate(G, 0, 0, idx, val, 0, nnz) == 0);
}

int main(void) {
    CHECK(oracle_k_from_rho(1 << 20, 0.001) == 1049);
    CHECK(oracle_k_from_rho(0, 0.5) == 0);
    CHECK(oracle_k_from_rho(10, 0.0) == -1);
    CHECK(oracle_k_from_rho(10, NAN) == -1);
    selection_cases();
    update_cases();
    printf("oracle driver: %d failed checks\n", fails);
    return fails;
}
