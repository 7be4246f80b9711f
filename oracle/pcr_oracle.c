/*
 * pcr_oracle.c -- plain fp64 CPU oracle for paged prefix-reuse prefill attention.
 *
 * TEST INFRASTRUCTURE. Only the tests, the smoke check and the benchmark's CPU
 * baseline leg may load this library. It shares no code, header or constant
 * with the HIP path: the pool layout below is restated here from its written
 * definition, not included.
 *
 * What it computes (Sec. 2.2 "Prefix KV Cache Reuse"): with exact-prefix reuse,
 * the output for the uncached suffix tokens equals the output of full prefill
 * of the whole sequence for those rows, because the cached prefix K/V are the
 * very K/V full prefill would have produced. So for every sequence b, query
 * head h and suffix row i (absolute position p_b + i) the result is causal
 * softmax attention of q over keys 0 .. p_b + i, read through the paged pool
 * (Sec. 5: non-contiguous fixed-size physical blocks mapped by a block table).
 *
 * Pool layout (one layer, one of K and V each; bf16 bit patterns):
 *   K element of (block blk, kv head g, slot o, dim x) at ((blk*Hkv + g)*bs + o)*d + x
 *   V element of (block blk, kv head g, slot o, dim x) at ((blk*Hkv + g)*d + x)*bs + o
 * Logical token t of sequence b lives in block block_tables[b][t / bs], slot t % bs.
 * GQA: query head h reads kv head h / (Hq / Hkv).
 *
 * Arithmetic: every bf16 input is widened exactly to double; scores are
 * sm_scale * <q, k>; softmax is the two-pass form (row max, then
 * exp(score - max) weights, normalised at the end); all in double.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

static double bf16_to_f64(uint16_t h)
{
    uint32_t u = (uint32_t)h << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/* Row list entry: (token index in [0, T), query head). */
typedef struct { int32_t t, h; } oracle_row;

static int seq_of_token(const int32_t *cu_suffix, int B, int32_t t)
{
    /* largest b with cu_suffix[b] <= t and cu_suffix[b+1] > t */
    int lo = 0, hi = B - 1;
    while (lo < hi) {
        int mid = (lo + hi + 1) / 2;
        if (cu_suffix[mid] <= t) lo = mid; else hi = mid - 1;
    }
    return lo;
}

/* One output row: out_row[0..d) = attention of query (t, h). Returns 0 or an error code. */
static int one_row(const uint16_t *q, int Hq, int Hkv, int d, int bs,
                   const uint16_t *pool_k, const uint16_t *pool_v, int64_t num_blocks,
                   const int32_t *block_tables, int max_blocks,
                   const int32_t *prefix_lens, const int32_t *cu_suffix, int B,
                   double sm_scale, int32_t t, int32_t h, double *out_row)
{
    const int b = seq_of_token(cu_suffix, B, t);
    const int32_t i = t - cu_suffix[b];            /* suffix row */
    const int64_t pos = (int64_t)prefix_lens[b] + i; /* absolute position of the query */
    const int64_t nkeys = pos + 1;                  /* causal, diagonal included */
    const int G = Hq / Hkv;
    const int g = h / G;
    const int32_t *bt = block_tables + (int64_t)b * max_blocks;

    if ((nkeys + bs - 1) / bs > max_blocks) return -1;

    double *score = (double *)malloc(sizeof(double) * (size_t)nkeys);
    double *qv = (double *)malloc(sizeof(double) * (size_t)d);
    double *acc = (double *)calloc((size_t)d, sizeof(double));
    if (!score || !qv || !acc) { free(score); free(qv); free(acc); return -2; }

    for (int x = 0; x < d; ++x)
        qv[x] = bf16_to_f64(q[((int64_t)t * Hq + h) * d + x]);

    int rc = 0;
    /* pass 1: scores and their maximum */
    double m = -INFINITY;
    for (int64_t j = 0; j < nkeys; ++j) {
        const int64_t blk = bt[j / bs];
        const int64_t o = j % bs;
        if (blk < 0 || blk >= num_blocks) { rc = -3; goto done; }
        const uint16_t *krow = pool_k + ((blk * Hkv + g) * bs + o) * d;
        double dot = 0.0;
        for (int x = 0; x < d; ++x) dot += qv[x] * bf16_to_f64(krow[x]);
        score[j] = sm_scale * dot;
        if (score[j] > m) m = score[j];
    }
    /* pass 2: weights exp(score - max), weighted sum of values, normaliser */
    double sum = 0.0;
    for (int64_t j = 0; j < nkeys; ++j) {
        const int64_t blk = bt[j / bs];
        const int64_t o = j % bs;
        const double w = exp(score[j] - m);
        sum += w;
        const uint16_t *vbase = pool_v + (blk * Hkv + g) * (int64_t)d * bs + o;
        for (int x = 0; x < d; ++x) acc[x] += w * bf16_to_f64(vbase[(int64_t)x * bs]);
    }
    for (int x = 0; x < d; ++x) out_row[x] = acc[x] / sum;
done:
    free(score); free(qv); free(acc);
    return rc;
}

static int check_shapes(int Hq, int Hkv, int d, int bs, int B)
{
    if (Hq <= 0 || Hkv <= 0 || d <= 0 || bs <= 0 || B < 0) return -1;
    if (Hq % Hkv != 0) return -1;
    return 0;
}

/*
 * Full output: out[T][Hq][d] (double). T = cu_suffix[B].
 * Returns 0, or a negative code (bad shape, block table too short, block id out of range).
 */
int pcr_oracle_attention(const uint16_t *q, int Hq, int Hkv, int d, int bs,
                         const uint16_t *pool_k, const uint16_t *pool_v, int64_t num_blocks,
                         const int32_t *block_tables, int max_blocks,
                         const int32_t *prefix_lens, const int32_t *cu_suffix, int B,
                         double sm_scale, double *out)
{
    if (check_shapes(Hq, Hkv, d, bs, B)) return -1;
    const int64_t T = B > 0 ? cu_suffix[B] : 0;
    const int64_t rows = T * Hq;
    int rc = 0;
#pragma omp parallel for schedule(dynamic, 4) reduction(min : rc)
    for (int64_t r = 0; r < rows; ++r) {
        const int32_t t = (int32_t)(r / Hq), h = (int32_t)(r % Hq);
        int e = one_row(q, Hq, Hkv, d, bs, pool_k, pool_v, num_blocks, block_tables, max_blocks,
                        prefix_lens, cu_suffix, B, sm_scale, t, h, out + r * d);
        if (e < rc) rc = e;
    }
    return rc;
}

/*
 * Selected rows only: out[n_rows][d] for rows[k] = (t, h). Same definition as above.
 */
int pcr_oracle_attention_rows(const uint16_t *q, int Hq, int Hkv, int d, int bs,
                              const uint16_t *pool_k, const uint16_t *pool_v, int64_t num_blocks,
                              const int32_t *block_tables, int max_blocks,
                              const int32_t *prefix_lens, const int32_t *cu_suffix, int B,
                              double sm_scale, const int32_t *rows, int64_t n_rows, double *out)
{
    if (check_shapes(Hq, Hkv, d, bs, B)) return -1;
    const int64_t T = B > 0 ? cu_suffix[B] : 0;
    int rc = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(min : rc)
    for (int64_t k = 0; k < n_rows; ++k) {
        const oracle_row *rw = (const oracle_row *)rows + k;
        int e;
        if (rw->t < 0 || rw->t >= T || rw->h < 0 || rw->h >= Hq) e = -1;
        else e = one_row(q, Hq, Hkv, d, bs, pool_k, pool_v, num_blocks, block_tables, max_blocks,
                         prefix_lens, cu_suffix, B, sm_scale, rw->t, rw->h, out + k * d);
        if (e < rc) rc = e;
    }
    return rc;
}

#ifndef PCR_ORACLE_SOURCE_SHA256
#define PCR_ORACLE_SOURCE_SHA256 "unknown"
#endif
/* SHA-256 of the source this library was built from (set by the build script). */
const char *pcr_oracle_source_sha256(void) { return PCR_ORACLE_SOURCE_SHA256; }

/* Threads for the next parallel regions (n >= 1), e.g. a one-thread timing run. */
void pcr_oracle_set_num_threads(int n)
{
#ifdef _OPENMP
    extern void omp_set_num_threads(int);
    omp_set_num_threads(n > 0 ? n : 1);
#else
    (void)n;
#endif
}

/* Number of threads the OpenMP runtime will use (for reporting). */
int pcr_oracle_num_threads(void)
{
    int n = 1;
#pragma omp parallel
    {
#pragma omp single
        {
#ifdef _OPENMP
            extern int omp_get_num_threads(void);
            n = omp_get_num_threads();
#endif
        }
    }
    return n;
}
