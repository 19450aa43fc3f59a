/*
 * Oracle for the segment re-prefill attention (test infrastructure only).
 *
 * Only the tests, the smoke check and the CPU-baseline leg of the benchmark
 * load this library.  It shares no code, header or constant with the device
 * library and must never be reached from the product path.
 *
 * What it computes is the plain definition of causal grouped-query attention
 * of a new segment over a cached prefix (paper Sec. 4, performance model,
 * prefill-attention term: the segment's token number i, counting from zero,
 * sees the whole cached prefix and segment tokens 0..i, so prefix + i + 1 keys
 * in all, the quantity the work count A_j adds up).  For sequence b with segment
 * length q_b and total length kv_b (prefix_b = kv_b - q_b), query head h and
 * segment row i:
 *
 *     pos   = prefix_b + i                       (last visible key)
 *     g     = floor(h / (Hq / Hkv))              (grouped-query mapping)
 *     s_j   = scale * sum_d Q[i,h,d] * K[j,g,d]  for j = 0 .. pos
 *     m     = max_j s_j
 *     p_j   = exp(s_j - m),  l = sum_j p_j
 *     O     = sum_j p_j V[j,g,:] / l,  LSE = m + log(l)
 *
 * K and V are CONTIGUOUS in logical token order (prefix rows, then segment
 * rows); paging plays no part here.  All arithmetic is IEEE double: the bf16
 * inputs widen exactly, the exponential is libm's exp, and there is no
 * blocking, tiling or reordering beyond the definition above.  Rows are
 * independent, so OpenMP spreads them over threads without changing any
 * row's arithmetic.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* bf16 bit pattern -> double, exactly (bf16 is the top half of a float32). */
static double bf16_to_double(uint16_t b)
{
    uint32_t u = ((uint32_t)b) << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/* Index of the sequence whose query range [q_indptr[b], q_indptr[b+1]) holds t. */
static int find_seq(const int64_t *q_indptr, int B, int64_t t)
{
    int lo = 0, hi = B - 1;
    while (lo < hi) {
        int mid = (lo + hi + 1) / 2;
        if (q_indptr[mid] <= t)
            lo = mid;
        else
            hi = mid - 1;
    }
    /* skip empty sequences that share the same start */
    while (lo + 1 < B && q_indptr[lo + 1] <= t)
        lo++;
    return lo;
}

/*
 * Attention output for an explicit list of (token, head) rows.
 *
 * q        bf16 bits [sum q][Hq][D]
 * k, v     bf16 bits [sum kv][Hkv][D]; sequence b owns rows kv_indptr[b] ..
 *          kv_indptr[b+1]-1 in logical order
 * q_indptr, kv_indptr   [B+1] cumulative offsets
 * row_token, row_head   [n_rows] which outputs to compute (token indexes sum q)
 * out      [n_rows][D] double;  lse [n_rows] double (nullable)
 * n_keys   [n_rows] number of keys the row attended to (nullable)
 *
 * Returns 0, or -1 if a row names a token or head outside the inputs, or a
 * sequence with q_len > kv_len.
 */
int oracle_attn_rows(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                     int B, const int64_t *q_indptr, const int64_t *kv_indptr,
                     int Hq, int Hkv, int D, double scale,
                     int64_t n_rows, const int64_t *row_token, const int32_t *row_head,
                     double *out, double *lse, int64_t *n_keys)
{
    if (B <= 0 || Hq <= 0 || Hkv <= 0 || D <= 0 || Hq % Hkv != 0)
        return -1;
    const int G = Hq / Hkv;
    const int64_t total_q = q_indptr[B];
    int bad = 0;

#pragma omp parallel for schedule(dynamic, 4) reduction(|| : bad)
    for (int64_t r = 0; r < n_rows; r++) {
        const int64_t t = row_token[r];
        const int h = row_head[r];
        if (t < 0 || t >= total_q || h < 0 || h >= Hq) {
            bad = 1;
            continue;
        }
        const int b = find_seq(q_indptr, B, t);
        const int64_t q_len = q_indptr[b + 1] - q_indptr[b];
        const int64_t kv_len = kv_indptr[b + 1] - kv_indptr[b];
        if (q_len > kv_len) {
            bad = 1;
            continue;
        }
        const int64_t i = t - q_indptr[b];
        const int64_t pos = (kv_len - q_len) + i;
        const int g = h / G;

        double *s = (double *)malloc(sizeof(double) * (size_t)(pos + 1));
        double *qd = (double *)malloc(sizeof(double) * (size_t)D);
        const uint16_t *qrow = q + ((size_t)t * Hq + h) * D;
        for (int d = 0; d < D; d++)
            qd[d] = bf16_to_double(qrow[d]);

        double m = -INFINITY;
        for (int64_t j = 0; j <= pos; j++) {
            const uint16_t *krow = k + ((size_t)(kv_indptr[b] + j) * Hkv + g) * D;
            double acc = 0.0;
            for (int d = 0; d < D; d++)
                acc += qd[d] * bf16_to_double(krow[d]);
            s[j] = scale * acc;
            if (s[j] > m)
                m = s[j];
        }

        double l = 0.0;
        double *o = out + (size_t)r * D;
        for (int d = 0; d < D; d++)
            o[d] = 0.0;
        for (int64_t j = 0; j <= pos; j++) {
            const double p = exp(s[j] - m);
            l += p;
            const uint16_t *vrow = v + ((size_t)(kv_indptr[b] + j) * Hkv + g) * D;
            for (int d = 0; d < D; d++)
                o[d] += p * bf16_to_double(vrow[d]);
        }
        for (int d = 0; d < D; d++)
            o[d] /= l;
        if (lse)
            lse[r] = m + log(l);
        if (n_keys)
            n_keys[r] = pos + 1;
        free(s);
        free(qd);
    }
    return bad ? -1 : 0;
}

/* Number of OpenMP threads the oracle uses (for reporting the CPU baseline). */
int oracle_num_threads(void)
{
#ifdef _OPENMP
    extern int omp_get_max_threads(void);
    return omp_get_max_threads();
#else
    return 1;
#endif
}
