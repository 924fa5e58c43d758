/*
 * oracle.c -- plain, slow, obviously correct CPU reference for single-query
 * decode attention over a KV cache and for the per-step KV append.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path links, loads or
 * calls this file.  Only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg use it.  It shares no code, header, table or helper with
 * the HIP library: the only thing the two sides have in common is the memory
 * layout convention they both read (row-major, contiguous fp32).
 *
 * Arithmetic: inputs are fp32 as stored; every product, sum, max and exp is
 * done in fp64 (libm exp), results are fp64.  No blocking, fusion, online
 * softmax or reordering: each (batch, query head) follows Algorithm 1 (the
 * single-query decode step of the DNF section) in the paper's order -- all scores,
 * then the max, then the exponentials, then Z, then the weights, then the
 * weighted sum.
 *
 * Layout (row-major, the ONF offset rule of the section "ONF Stride
 * Arithmetic": element <l,j> of an <n,d_k> slab lives at l*d_k + j):
 *   q   [B][h_q][d_k]
 *   K   [B][h_kv][n_max][d_k]
 *   V   [B][h_kv][n_max][d_v]
 *   len [B]            number of valid cache rows of sequence b
 *   out [B][h_q][d_v]  (fp64)
 *
 * Multi-row decode (oracle_decode_multi): q [B][h_q][T][d_k] and
 * out [B][h_q][T][d_v]; the T query rows are the cache's last T positions.
 *
 * Readings of points the paper leaves open (each also stated beside the code
 * that implements it):
 *   - scale multiplies the dot product once, eq. (1); it is always passed in.
 *   - query head h reads KV head floor(h*h_kv/h_q), eq. (10) / Fig. 3.
 *   - rows used are 0 .. clamp(len[b],0,n_max)-1; an empty cache gives 0.
 *   - append writes row len[b] then increments len[b] (the pre-allocated
 *     cache of the multi-step section); at len[b] >= n_max (or len[b] < 0) it
 *     does nothing.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

/* Number of cache rows the decode of sequence b reads.  The paper's cache
 * holds exactly _t rows; a count outside [0, n_max] cannot describe a
 * cache of capacity n_max, so it is clamped. */
static int64_t rows_used(int32_t len_b, int n_max)
{
    if (len_b < 0) return 0;
    if (len_b > n_max) return n_max;
    return len_b;
}

/*
 * Algorithm 1 for one query vector against one <n, d_k> / <n, d_v> slab.
 *   Step I   (eq. 1): s[l] = scale * sum_j q[j] * K[l*d_k + j]
 *   Step II  (eq. 2): m = max_l s[l]; e[l] = exp(s[l] - m); Z = sum_l e[l];
 *                     a[l] = e[l] / Z
 *   Step III (eq. 3): out[d] = sum_l a[l] * V[l*d_v + d]
 * s and a are O(n) scratch supplied by the caller (a may alias nothing).
 * If a_out is non-NULL the weights a[0..n) are copied there.
 */
static void decode_one_query(const float *q, const float *Kslab,
                             const float *Vslab, int64_t n, int d_k, int d_v,
                             double scale, double *out, double *s, double *e,
                             double *a_out)
{
    if (n == 0) {
        /* Empty cache: Algorithm 1 has no rows to weight.  The result is
         * defined as the zero vector (what the paper's C kernel, which starts
         * from a zeroed output, gives). */
        for (int d = 0; d < d_v; ++d) out[d] = 0.0;
        return;
    }

    /* Step I -- scores, K read row by row in its natural layout. */
    for (int64_t l = 0; l < n; ++l) {
        const float *Krow = Kslab + l * (int64_t)d_k;
        double dot = 0.0;
        for (int j = 0; j < d_k; ++j) dot += (double)q[j] * (double)Krow[j];
        s[l] = scale * dot;
    }

    /* Step II -- numerically stable softmax. */
    double m = -INFINITY;
    for (int64_t l = 0; l < n; ++l)
        if (s[l] > m) m = s[l];
    for (int64_t l = 0; l < n; ++l) e[l] = exp(s[l] - m);
    double Z = 0.0;
    for (int64_t l = 0; l < n; ++l) Z += e[l];
    for (int64_t l = 0; l < n; ++l) e[l] = e[l] / Z;   /* e now holds a */
    if (a_out)
        for (int64_t l = 0; l < n; ++l) a_out[l] = e[l];

    /* Step III -- weighted sum, V read row by row. */
    for (int d = 0; d < d_v; ++d) out[d] = 0.0;
    for (int64_t l = 0; l < n; ++l) {
        const float *Vrow = Vslab + l * (int64_t)d_v;
        for (int d = 0; d < d_v; ++d) out[d] += e[l] * (double)Vrow[d];
    }
}

/* psi-selection of the KV head for query head h, eq. (10):
 * g_kv = floor(h * h_kv / h_q).  With h_kv dividing h_q this gives the
 * contiguous groups of Fig. 3 / the worked GQA example. */
static int kv_head_of(int h, int h_q, int h_kv)
{
    return (int)(((int64_t)h * h_kv) / h_q);
}

/*
 * Decode attention for every (b, h) with head_mask[b*h_q+h] != 0 (all of
 * them when head_mask is NULL).  Returns 0, or -1 on a shape error or an
 * allocation failure.  threads <= 0 means the OpenMP default.
 */
int oracle_decode(const float *q, const float *K, const float *V,
                  const int32_t *len, float scale, double *out, int B, int h_q,
                  int h_kv, int n_max, int d_k, int d_v,
                  const uint8_t *head_mask, int threads)
{
    if (B < 1 || h_q < 1 || h_kv < 1 || n_max < 1 || d_k < 1 || d_v < 1)
        return -1;
    if (h_q % h_kv != 0) return -1;   /* "h_kv divides h_q" (GQA section) */

    const double sc = (double)scale;
    int failed = 0;
    const int64_t units = (int64_t)B * h_q;

#ifdef _OPENMP
    if (threads <= 0) threads = omp_get_max_threads();
#pragma omp parallel num_threads(threads) reduction(| : failed)
#endif
    {
        double *s = (double *)malloc(sizeof(double) * (size_t)n_max);
        double *e = (double *)malloc(sizeof(double) * (size_t)n_max);
        if (!s || !e) failed = 1;
#ifdef _OPENMP
#pragma omp for schedule(dynamic, 1)
#endif
        for (int64_t u = 0; u < units; ++u) {
            if (!s || !e) continue;
            if (head_mask && !head_mask[u]) continue;
            const int b = (int)(u / h_q);
            const int h = (int)(u % h_q);
            const int g = kv_head_of(h, h_q, h_kv);
            const int64_t n = rows_used(len[b], n_max);
            const float *qv = q + ((int64_t)b * h_q + h) * d_k;
            const float *Ks = K + ((int64_t)b * h_kv + g) * n_max * d_k;
            const float *Vs = V + ((int64_t)b * h_kv + g) * n_max * d_v;
            decode_one_query(qv, Ks, Vs, n, d_k, d_v, sc,
                             out + ((int64_t)b * h_q + h) * d_v, s, e, NULL);
        }
        free(s);
        free(e);
    }
    (void)threads;
    return failed ? -1 : 0;
}

/*
 * The softmax weights a[0..n) of one (b, h) (Step II output) and its output
 * row.  Returns n (rows used), or -1 on error.  Debug entry for invariant
 * tests (the weights of Algorithm 1 sum to one).
 */
int64_t oracle_decode_weights(const float *q, const float *K, const float *V,
                              const int32_t *len, float scale, int b, int h,
                              int B, int h_q, int h_kv, int n_max, int d_k,
                              int d_v, double *weights, double *out_row)
{
    if (b < 0 || b >= B || h < 0 || h >= h_q || h_q % h_kv != 0) return -1;
    const int g = kv_head_of(h, h_q, h_kv);
    const int64_t n = rows_used(len[b], n_max);
    double *s = (double *)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1));
    double *e = (double *)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1));
    if (!s || !e) { free(s); free(e); return -1; }
    decode_one_query(q + ((int64_t)b * h_q + h) * d_k,
                     K + ((int64_t)b * h_kv + g) * n_max * d_k,
                     V + ((int64_t)b * h_kv + g) * n_max * d_v, n, d_k, d_v,
                     (double)scale, out_row, s, e, weights);
    free(s);
    free(e);
    return n;
}

/*
 * KV append, eqs. (6)-(7): K_{t+1} = K_t # k_t, V_{t+1} = V_t # v_t.
 * For every (b, g): the new rows are written at row t = len[b], i.e. at the
 * ONF offsets t*d_k + j and t*d_v + d of the slab (worked example: t=2,
 * d_k=3 lands at 6, 7, 8); no existing row moves.  Then len[b] += 1.
 * Rows are copied as bytes, so every bit pattern (NaN payloads included)
 * is preserved.  A full cache (len[b] >= n_max) or a negative count is left
 * untouched.
 *   k_new [B][h_kv][d_k], v_new [B][h_kv][d_v]
 */
int oracle_append(float *K, float *V, const float *k_new, const float *v_new,
                  int32_t *len, int B, int h_kv, int n_max, int d_k, int d_v)
{
    if (B < 1 || h_kv < 1 || n_max < 1 || d_k < 1 || d_v < 1) return -1;
    for (int b = 0; b < B; ++b) {
        const int32_t t = len[b];
        if (t < 0 || t >= n_max) continue;
        for (int g = 0; g < h_kv; ++g) {
            float *Ks = K + ((int64_t)b * h_kv + g) * n_max * d_k;
            float *Vs = V + ((int64_t)b * h_kv + g) * n_max * d_v;
            memcpy(Ks + (int64_t)t * d_k, k_new + ((int64_t)b * h_kv + g) * d_k,
                   sizeof(float) * (size_t)d_k);
            memcpy(Vs + (int64_t)t * d_v, v_new + ((int64_t)b * h_kv + g) * d_v,
                   sizeof(float) * (size_t)d_v);
        }
        len[b] = t + 1;
    }
    return 0;
}

/*
 * Decode with T query rows per (b, h): the rank-2 query of the paper's
 * training form, softmax(scale * Q (+.x Omega<2,2>) K) (+.x Omega<2,2>) V,
 * restricted to causal visibility for a step that submits T consecutive
 * positions at once (speculative verification, chunked prefill).  The T rows
 * occupy the cache's last T positions: row r of sequence b sits at position
 *   p = clamp(len[b], 0, n_max) - T + r
 * and sees rows 0..p, itself and everything before it.  Each row is
 * therefore Algorithm 1 on the prefix of n_r = p + 1 rows (none if p < 0,
 * giving the zero vector like an empty cache).
 *   q   [B][h_q][T][d_k]
 *   out [B][h_q][T][d_v] (fp64)
 * Returns 0, or -1 on a shape error or an allocation failure.
 */
int oracle_decode_multi(const float *q, const float *K, const float *V,
                        const int32_t *len, float scale, double *out, int B,
                        int h_q, int h_kv, int n_max, int d_k, int d_v, int T,
                        int threads)
{
    if (B < 1 || h_q < 1 || h_kv < 1 || n_max < 1 || d_k < 1 || d_v < 1 || T < 1)
        return -1;
    if (h_q % h_kv != 0) return -1;

    const double sc = (double)scale;
    int failed = 0;
    const int64_t units = (int64_t)B * h_q * T;

#ifdef _OPENMP
    if (threads <= 0) threads = omp_get_max_threads();
#pragma omp parallel num_threads(threads) reduction(| : failed)
#endif
    {
        double *s = (double *)malloc(sizeof(double) * (size_t)n_max);
        double *e = (double *)malloc(sizeof(double) * (size_t)n_max);
        if (!s || !e) failed = 1;
#ifdef _OPENMP
#pragma omp for schedule(dynamic, 1)
#endif
        for (int64_t u = 0; u < units; ++u) {
            if (!s || !e) continue;
            const int r = (int)(u % T);
            const int64_t bh = u / T;
            const int b = (int)(bh / h_q);
            const int h = (int)(bh % h_q);
            const int g = kv_head_of(h, h_q, h_kv);
            /* position of query row r; it sees rows 0..pos */
            const int64_t pos = rows_used(len[b], n_max) - T + r;
            const int64_t n = pos >= 0 ? pos + 1 : 0;
            const float *qv = q + u * d_k;
            const float *Ks = K + ((int64_t)b * h_kv + g) * n_max * d_k;
            const float *Vs = V + ((int64_t)b * h_kv + g) * n_max * d_v;
            decode_one_query(qv, Ks, Vs, n, d_k, d_v, sc, out + u * d_v, s, e,
                             NULL);
        }
        free(s);
        free(e);
    }
    (void)threads;
    return failed ? -1 : 0;
}

/*
 * T rows appended in order: the single-row append above applied T times,
 * row r of every (b, g) taken from k_new[b][g][r] / v_new[b][g][r].  Each
 * application writes at the current len[b] and increments it, and does
 * nothing once the cache is full, so a sequence with room for fewer than T
 * rows keeps the first ones that fit.
 *   k_new [B][h_kv][T][d_k], v_new [B][h_kv][T][d_v]
 */
int oracle_append_rows(float *K, float *V, const float *k_new,
                       const float *v_new, int32_t *len, int B, int h_kv,
                       int n_max, int d_k, int d_v, int T)
{
    if (B < 1 || h_kv < 1 || n_max < 1 || d_k < 1 || d_v < 1 || T < 1) return -1;
    for (int r = 0; r < T; ++r) {
        for (int b = 0; b < B; ++b) {
            const int32_t t = len[b];
            if (t < 0 || t >= n_max) continue;
            for (int g = 0; g < h_kv; ++g) {
                const int64_t src = ((int64_t)b * h_kv + g) * T + r;
                float *Ks = K + ((int64_t)b * h_kv + g) * n_max * d_k;
                float *Vs = V + ((int64_t)b * h_kv + g) * n_max * d_v;
                memcpy(Ks + (int64_t)t * d_k, k_new + src * d_k,
                       sizeof(float) * (size_t)d_k);
                memcpy(Vs + (int64_t)t * d_v, v_new + src * d_v,
                       sizeof(float) * (size_t)d_v);
            }
            len[b] = t + 1;
        }
    }
    return 0;
}

/* Threads an OpenMP region in this library would use (1 without OpenMP). */
int oracle_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
