/*
 * attn_oracle.c -- plain, slow, obviously correct CPU oracle for the attention
 * forward pass.  TEST INFRASTRUCTURE ONLY: it is linked by the test suite, the
 * smoke check and the CPU-baseline leg of the benchmark, never by the product
 * library, and it shares no code, header or constant with the HIP path.
 *
 * What it computes (Section 2.3, Eq. (1) "eq:fa"):
 *     S = Q K^T,   P = softmax(S * scale),   O = P V
 * for every (batch b, query head hq, query row i), with
 *   - grouped-query attention (Section 2.3, the MHA/GQA paragraph): query head
 *     hq reads key/value head g = hq / (Hq / Hkv), i.e. contiguous groups of
 *     Hq/Hkv query heads share one K/V head (MHA is the case Hq == Hkv);
 *   - an optional causal mask, top-left aligned: row i sees keys j <= i;
 *   - `scale` is the float32 value the caller passes (the paper fixes it to
 *     1/sqrt(d)); it is widened to double once.
 * FlashAttention's tiled online softmax (Section 2.3.1) reaches this same
 * result in exact arithmetic -- its cross-tile fix-up step exists precisely to
 * make that so -- so the oracle is the plain definition, not the tiled
 * algorithm: a two-pass softmax in fp64 (pass 1: row maximum; pass 2:
 * exponentials, their sum and the weighted sum of V rows, then one division).
 *
 * Inputs are the raw bf16 bit patterns (uint16) of Q[B][Hq][Sq][d] and
 * K, V[B][Hkv][Skv][d], contiguous; bf16 -> double is exact.  Outputs are fp64.
 *
 * Error behaviour: returns 0 on success, -1 on a null pointer, -2 on a bad
 * shape (a dimension <= 0, Hq not a multiple of Hkv, a row index out of
 * range), -3 when scratch memory cannot be allocated.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

static double bf16_bits_to_double(uint16_t bits)
{
    uint32_t u = (uint32_t)bits << 16;   /* bf16 is the top half of an IEEE float */
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

static int check_shape(int B, int Hq, int Hkv, int Sq, int Skv, int d)
{
    if (B <= 0 || Hq <= 0 || Hkv <= 0 || Sq <= 0 || Skv <= 0 || d <= 0) return -2;
    if (Hq % Hkv != 0) return -2;
    return 0;
}

/*
 * One output row O[b, hq, i, :] written to `out` (d doubles).
 * `s` is caller-provided scratch of Skv doubles.
 */
static void attention_row(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                          int Hq, int Hkv, int Sq, int Skv, int d, int causal, double scale,
                          int b, int hq, int i, double *s, double *out)
{
    const int group = Hq / Hkv;          /* query heads per K/V head */
    const int g = hq / group;            /* K/V head read by query head hq */
    const uint16_t *qrow = q + (((int64_t)b * Hq + hq) * Sq + i) * (int64_t)d;
    const uint16_t *kh = k + ((int64_t)b * Hkv + g) * (int64_t)Skv * d;
    const uint16_t *vh = v + ((int64_t)b * Hkv + g) * (int64_t)Skv * d;

    /* the keys row i may attend to: j in [0, jend) */
    int jend = Skv;
    if (causal && i + 1 < jend) jend = i + 1;

    /* scores s_j = scale * <Q[i], K[j]> */
    for (int j = 0; j < jend; ++j) {
        const uint16_t *krow = kh + (int64_t)j * d;
        double dot = 0.0;
        for (int c = 0; c < d; ++c)
            dot += bf16_bits_to_double(qrow[c]) * bf16_bits_to_double(krow[c]);
        s[j] = scale * dot;
    }

    /* pass 1: the row maximum */
    double mx = -INFINITY;
    for (int j = 0; j < jend; ++j)
        if (s[j] > mx) mx = s[j];

    /* pass 2: exponentials, their sum, and the weighted sum of V rows */
    for (int c = 0; c < d; ++c) out[c] = 0.0;
    double l = 0.0;
    for (int j = 0; j < jend; ++j) {
        const double p = exp(s[j] - mx);
        const uint16_t *vrow = vh + (int64_t)j * d;
        l += p;
        for (int c = 0; c < d; ++c)
            out[c] += p * bf16_bits_to_double(vrow[c]);
    }
    for (int c = 0; c < d; ++c) out[c] /= l;
}

static void set_threads(int nthreads)
{
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#else
    (void)nthreads;
#endif
}

/* Number of threads the next parallel region will use (1 without OpenMP). */
int oracle_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/*
 * Full forward: o[B][Hq][Sq][d] (fp64).  nthreads <= 0 keeps the OpenMP
 * default.
 */
int oracle_attn_fwd_f64(const uint16_t *q, const uint16_t *k, const uint16_t *v, double *o,
                        int B, int Hq, int Hkv, int Sq, int Skv, int d,
                        int causal, float scale, int nthreads)
{
    if (!q || !k || !v || !o) return -1;
    int rc = check_shape(B, Hq, Hkv, Sq, Skv, d);
    if (rc) return rc;
    set_threads(nthreads);
    const double sc = (double)scale;
    const int64_t nrows = (int64_t)B * Hq * Sq;
    int failed = 0;
#pragma omp parallel
    {
        double *s = (double *)malloc(sizeof(double) * (size_t)Skv);
        if (!s) {
#pragma omp atomic write
            failed = 1;
        } else {
#pragma omp for schedule(dynamic, 16)
            for (int64_t r = 0; r < nrows; ++r) {
                const int i = (int)(r % Sq);
                const int hq = (int)((r / Sq) % Hq);
                const int b = (int)(r / ((int64_t)Sq * Hq));
                attention_row(q, k, v, Hq, Hkv, Sq, Skv, d, causal, sc, b, hq, i, s,
                              o + r * (int64_t)d);
            }
            free(s);
        }
    }
    return failed ? -3 : 0;
}

/*
 * Sampled rows: rows[3*r + 0..2] = (b, hq, i); o_rows[r][d] (fp64).  Every
 * output row depends only on its own query row, so a sampled row is exactly
 * the row of the full result.
 */
int oracle_attn_fwd_rows_f64(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                             const int64_t *rows, int64_t nrows, double *o_rows,
                             int B, int Hq, int Hkv, int Sq, int Skv, int d,
                             int causal, float scale, int nthreads)
{
    if (!q || !k || !v || !o_rows || (!rows && nrows > 0)) return -1;
    int rc = check_shape(B, Hq, Hkv, Sq, Skv, d);
    if (rc) return rc;
    for (int64_t r = 0; r < nrows; ++r) {
        const int64_t b = rows[3 * r], hq = rows[3 * r + 1], i = rows[3 * r + 2];
        if (b < 0 || b >= B || hq < 0 || hq >= Hq || i < 0 || i >= Sq) return -2;
    }
    set_threads(nthreads);
    const double sc = (double)scale;
    int failed = 0;
#pragma omp parallel
    {
        double *s = (double *)malloc(sizeof(double) * (size_t)Skv);
        if (!s) {
#pragma omp atomic write
            failed = 1;
        } else {
#pragma omp for schedule(dynamic, 1)
            for (int64_t r = 0; r < nrows; ++r)
                attention_row(q, k, v, Hq, Hkv, Sq, Skv, d, causal, sc,
                              (int)rows[3 * r], (int)rows[3 * r + 1], (int)rows[3 * r + 2],
                              s, o_rows + r * (int64_t)d);
            free(s);
        }
    }
    return failed ? -3 : 0;
}
