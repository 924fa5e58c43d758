/*
 * Exercises every entry point of the CPU oracle (and the seeded input
 * generator) on small shapes, including the edge cases of its conventions,
 * so that a build with AddressSanitizer and UndefinedBehaviorSanitizer can
 * catch out-of-bounds accesses, overflow and uninitialised reads.  Test
 * infrastructure only; tests/test_oracle_sanitizers.py compiles and runs it.
 * Exit status 0 when every call returns what its contract says.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int oracle_decode(const float *q, const float *K, const float *V, const int32_t *len,
                  float scale, double *out, int B, int h_q, int h_kv, int n_max, int d_k,
                  int d_v, const uint8_t *head_mask, int threads);
int64_t oracle_decode_weights(const float *q, const float *K, const float *V,
                              const int32_t *len, float scale, int b, int h, int B, int h_q,
                              int h_kv, int n_max, int d_k, int d_v, double *weights,
                              double *out_row);
int oracle_append(float *K, float *V, const float *k_new, const float *v_new, int32_t *len,
                  int B, int h_kv, int n_max, int d_k, int d_v);
int oracle_decode_multi(const float *q, const float *K, const float *V, const int32_t *len,
                        float scale, double *out, int B, int h_q, int h_kv, int n_max,
                        int d_k, int d_v, int T, int threads);
int oracle_append_rows(float *K, float *V, const float *k_new, const float *v_new,
                       int32_t *len, int B, int h_kv, int n_max, int d_k, int d_v, int T);
void workload_normal_f32(uint64_t seed, uint32_t stream, int64_t offset, float *out,
                         int64_t count, int threads);

static int failures = 0;

#define EXPECT(cond, what)                                        \
    do {                                                          \
        if (!(cond)) {                                            \
            fprintf(stderr, "FAILED: %s (line %d)\n", what, __LINE__); \
            ++failures;                                           \
        }                                                         \
    } while (0)

static float *normals(uint32_t stream, int64_t n)
{
    float *p = malloc((size_t)(n > 0 ? n : 1) * sizeof(float));
    workload_normal_f32(7, stream, 0, p, n, 2);
    return p;
}

/* One shape: decode (all heads, then a head mask), the weights entry, T
 * appends, and the multi-row forms. */
static void run_shape(int B, int h_q, int h_kv, int n_max, int d_k, int d_v, int T,
                      const int32_t *len0)
{
    const int64_t nk = (int64_t)B * h_kv * n_max * d_k, nv = (int64_t)B * h_kv * n_max * d_v;
    float *q = normals(1, (int64_t)B * h_q * T * d_k);
    float *K = normals(2, nk), *V = normals(3, nv);
    float *kn = normals(4, (int64_t)B * h_kv * T * d_k), *vn = normals(5, (int64_t)B * h_kv * T * d_v);
    int32_t *len = malloc((size_t)B * sizeof(int32_t));
    memcpy(len, len0, (size_t)B * sizeof(int32_t));
    double *out = malloc((size_t)B * h_q * T * d_v * sizeof(double));
    const float scale = 1.0f / sqrtf((float)d_k);

    EXPECT(oracle_decode(q, K, V, len, scale, out, B, h_q, h_kv, n_max, d_k, d_v, NULL, 2) == 0,
           "decode");
    for (int64_t i = 0; i < (int64_t)B * h_q * d_v; ++i) EXPECT(isfinite(out[i]), "finite output");
    uint8_t *mask = calloc((size_t)B * h_q, 1);
    mask[0] = 1;
    EXPECT(oracle_decode(q, K, V, len, scale, out, B, h_q, h_kv, n_max, d_k, d_v, mask, 1) == 0,
           "masked decode");
    free(mask);

    double *w = malloc((size_t)n_max * sizeof(double)), *row = malloc((size_t)d_v * sizeof(double));
    for (int b = 0; b < B; ++b) {
        const int64_t n = oracle_decode_weights(q, K, V, len, scale, b, h_q - 1, B, h_q, h_kv,
                                                n_max, d_k, d_v, w, row);
        EXPECT(n >= 0 && n <= n_max, "weights row count");
        double sum = 0.0;
        for (int64_t l = 0; l < n; ++l) sum += w[l];
        EXPECT(n == 0 || fabs(sum - 1.0) < 1e-12, "weights sum to one");
    }
    EXPECT(oracle_decode_weights(q, K, V, len, scale, B, 0, B, h_q, h_kv, n_max, d_k, d_v, w,
                                 row) == -1, "weights: b out of range");
    free(w);
    free(row);

    for (int t = 0; t < T; ++t)
        EXPECT(oracle_append(K, V, kn, vn, len, B, h_kv, n_max, d_k, d_v) == 0, "append");
    EXPECT(oracle_decode_multi(q, K, V, len, scale, out, B, h_q, h_kv, n_max, d_k, d_v, T, 2) == 0,
           "decode_multi");
    EXPECT(oracle_append_rows(K, V, kn, vn, len, B, h_kv, n_max, d_k, d_v, T) == 0, "append_rows");
    for (int b = 0; b < B; ++b) {
        if (len0[b] < 0 || len0[b] >= n_max)      /* appends there do nothing */
            EXPECT(len[b] == len0[b], "len unchanged outside [0, n_max)");
        else
            EXPECT(len[b] == (len0[b] + 2 * T < n_max ? len0[b] + 2 * T : n_max),
                   "len advanced by the rows that fit");
    }

    free(q); free(K); free(V); free(kn); free(vn); free(len); free(out);
}

int main(void)
{
    const int32_t l1[] = {5};
    run_shape(1, 1, 1, 8, 4, 4, 1, l1);
    const int32_t l2[] = {0, 17, 64};                 /* empty, ragged, full */
    run_shape(3, 8, 2, 64, 16, 8, 3, l2);
    const int32_t l3[] = {-3, 100, 31};               /* negative, beyond n_max, one short */
    run_shape(3, 6, 3, 32, 8, 12, 2, l3);
    const int32_t l4[] = {40, 1};
    run_shape(2, 32, 1, 48, 32, 32, 4, l4);          /* MQA, several rows per step */

    /* shape errors are reported, not crashed on */
    float x = 0.f;
    double o = 0.0;
    int32_t l = 1;
    EXPECT(oracle_decode(&x, &x, &x, &l, 1.f, &o, 1, 3, 2, 1, 1, 1, NULL, 1) == -1,
           "h_kv must divide h_q");
    EXPECT(oracle_decode(&x, &x, &x, &l, 1.f, &o, 0, 1, 1, 1, 1, 1, NULL, 1) == -1, "B >= 1");
    EXPECT(oracle_append(&x, &x, &x, &x, &l, 1, 0, 1, 1, 1) == -1, "h_kv >= 1");
    EXPECT(oracle_append_rows(&x, &x, &x, &x, &l, 1, 1, 1, 1, 1, 0) == -1, "T >= 1");

    if (failures) {
        fprintf(stderr, "%d check(s) failed\n", failures);
        return 1;
    }
    printf("oracle sanitizer driver: all checks passed\n");
    return 0;
}
