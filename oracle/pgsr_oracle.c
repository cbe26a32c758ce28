/*
 * pgsr_oracle.c -- plain, slow fp64 reference of the prefill attention that the
 * sanitized-suffix replay runs.  TEST INFRASTRUCTURE ONLY: the tests, the smoke
 * check and the benchmark's CPU-baseline leg call it; the product path never
 * links, loads or calls it, and it shares no code with the HIP library.
 *
 * What it computes (transition F of Eq. (1), Section 3.1, realised as prefill;
 * the replay loop of Algorithm 1 re-materialises the suffix by prefill, Section
 * 3.2 after Lemma 2): for every suffix query row i (absolute position
 * pos0 + i) and query head h, with G = hq / hkv and KV head g = floor(h / G):
 *
 *     s_j  = scale * sum_c q[i,h,c] * k[j,g,c]          j = 0 .. pos0 + i
 *     m    = max_j s_j
 *     w_j  = exp(s_j - m)
 *     o[i,h,c] = sum_j w_j * v[j,g,c] / sum_j w_j
 *
 * i.e. softmax attention with an inclusive causal mask at absolute positions.
 * Keys 0 .. pos0-1 are the cropped clean prefix (Lemma 1), keys pos0 .. are
 * the replayed suffix itself.  Everything is fp64; the inputs are the values
 * the storage dtype holds (fp32 or bf16 widened exactly).
 *
 * Rows are independent, so the only parallelism is an OpenMP loop over rows;
 * inside a row the sums run in plain key order.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#ifdef _OPENMP
#include <omp.h>
#endif

int pgsr_oracle_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Returns 0 on success, 1 on a bad argument, 3 if scratch memory is short.
 *   q : [n_q][hq][d]   k, v : [n_kv][hkv][d]   (row-major fp64)
 *   rows == NULL : every (i, h); o is [n_q][hq][d]
 *   rows != NULL : rows[r] = i * hq + h for r < n_rows; o is [n_rows][d]   */
int pgsr_oracle_attention(int64_t n_q, int64_t pos0, int64_t n_kv,
                          int32_t hq, int32_t hkv, int32_t d,
                          const double *q, const double *k, const double *v,
                          double scale, const int64_t *rows, int64_t n_rows,
                          double *o) {
    if (n_q < 0 || pos0 < 0 || hq <= 0 || hkv <= 0 || d <= 0 || hq % hkv != 0)
        return 1;
    if (pos0 + n_q > n_kv) return 1;
    const int64_t G = hq / hkv;
    const int64_t total = rows ? n_rows : n_q * (int64_t)hq;
    int status = 0;

#pragma omp parallel
    {
        double *s = (double *)malloc(sizeof(double) * (size_t)(n_kv > 0 ? n_kv : 1));
        double *acc = (double *)malloc(sizeof(double) * (size_t)d);
        if (!s || !acc) {
#pragma omp atomic write
            status = 3;
        }
#pragma omp for schedule(dynamic, 4)
        for (int64_t r = 0; r < total; ++r) {
            if (!s || !acc) continue;
            const int64_t row = rows ? rows[r] : r;
            const int64_t i = row / hq, h = row % hq, g = h / G;
            if (i < 0 || i >= n_q) {
#pragma omp atomic write
                status = 1;
                continue;
            }
            const int64_t last = pos0 + i;              /* inclusive causal limit */
            const double *qi = q + (i * hq + h) * d;
            double m = -INFINITY;
            for (int64_t j = 0; j <= last; ++j) {
                const double *kj = k + (j * hkv + g) * d;
                double dot = 0.0;
                for (int c = 0; c < d; ++c) dot += qi[c] * kj[c];
                s[j] = scale * dot;
                if (s[j] > m) m = s[j];
            }
            double den = 0.0;
            for (int c = 0; c < d; ++c) acc[c] = 0.0;
            for (int64_t j = 0; j <= last; ++j) {
                const double w = exp(s[j] - m);
                den += w;
                const double *vj = v + (j * hkv + g) * d;
                for (int c = 0; c < d; ++c) acc[c] += w * vj[c];
            }
            double *out = o + (rows ? r : row) * d;
            for (int c = 0; c < d; ++c) out[c] = acc[c] / den;
        }
        free(s);
        free(acc);
    }
    return status;
}
