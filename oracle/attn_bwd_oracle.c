/*
 * attn_bwd_oracle.c -- plain, slow, obviously correct CPU oracle for the
 * attention backward pass and the row statistics it needs.  TEST
 * INFRASTRUCTURE ONLY: linked by the test suite, the smoke check and the
 * CPU-baseline leg of the benchmark, never by the product library; it shares
 * no code, header or constant with the HIP path (nor with attn_oracle.c).
 *
 * Forward (Section 2.3, Eq. "eq:fa"), per (batch b, query head hq, row i):
 *     s_ij = scale * <Q_i, K_j>            for keys j in J_i
 *     P_ij = exp(s_ij) / sum_{k in J_i} exp(s_ik)
 *     O_i  = sum_j P_ij V_j
 * with J_i = {0..Skv-1}, or {j <= i} under the top-left causal mask, and
 * query head hq reading K/V head g = hq / (Hq / Hkv) (grouped-query attention,
 * Section 2.3).
 *
 * Backward (Section 2.3, Eq. "eq:ba"), given dO = dL/dO:
 *     dV_j  = sum_i P_ij dO_i                  (dV = P^T dO)
 *     dP_ij = <dO_i, V_j>                       (dP = dO V^T)
 *     dS_ij = P_ij (dP_ij - D_i),  D_i = sum_k P_ik dP_ik
 *                                               (dS = dsoftmax(dP): the softmax
 *                                                Jacobian applied row by row)
 *     dQ_i  = scale * sum_j dS_ij K_j           (dQ = dS K)
 *     dK_j  = scale * sum_i dS_ij Q_i           (dK = dS^T Q)
 * The factor `scale` appears because S in Eq. "eq:ba" is the unscaled Q K^T
 * while the softmax sees scale * S.  Under GQA, dK and dV of K/V head g sum
 * over every query head of its group and every row.  The row statistics are
 *     lse_i = log sum_{j in J_i} exp(s_ij)      (what a forward pass keeps)
 *     D_i   = sum_j P_ij dP_ij                  (equal to <dO_i, O_i>)
 * All of it is evaluated in fp64 straight from the definitions: P from a
 * two-pass softmax (row maximum, then exponentials and their sum).
 *
 * Inputs are raw bf16 bit patterns (uint16), contiguous:
 *   q, dout [B][Hq][Sq][d];  k, v [B][Hkv][Skv][d].
 * Outputs are fp64 in the same layouts.  Return codes: 0 success, -1 a null
 * pointer, -2 a bad shape or row index, -3 scratch memory unavailable.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

static double bf(uint16_t bits)
{
    uint32_t u = (uint32_t)bits << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

static int bad_shape(int B, int Hq, int Hkv, int Sq, int Skv, int d)
{
    return B <= 0 || Hq <= 0 || Hkv <= 0 || Sq <= 0 || Skv <= 0 || d <= 0 || Hq % Hkv != 0;
}

static void threads(int n)
{
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

typedef struct {
    const uint16_t *q, *k, *v, *dout;
    int B, Hq, Hkv, Sq, Skv, d, causal;
    double scale;
} Problem;

static const uint16_t *qrow(const Problem *p, int b, int hq, int i)
{
    return p->q + (((int64_t)b * p->Hq + hq) * p->Sq + i) * (int64_t)p->d;
}
static const uint16_t *dorow(const Problem *p, int b, int hq, int i)
{
    return p->dout + (((int64_t)b * p->Hq + hq) * p->Sq + i) * (int64_t)p->d;
}
static const uint16_t *kvrow(const Problem *p, const uint16_t *t, int b, int g, int j)
{
    return t + (((int64_t)b * p->Hkv + g) * p->Skv + j) * (int64_t)p->d;
}
static int keys_of(const Problem *p, int i)   /* |J_i|: keys 0 .. end-1 */
{
    return (p->causal && i + 1 < p->Skv) ? i + 1 : p->Skv;
}

/*
 * For row (b, hq, i): the probabilities P_ij into prob[0..n), dP_ij into
 * dp[0..n) (when dp != NULL), and returns n = |J_i|; *lse and *Dsum receive
 * the row statistics (when not NULL).
 */
static int row_softmax(const Problem *p, int b, int hq, int i, double *prob, double *dp,
                       double *lse, double *Dsum)
{
    const int g = hq / (p->Hq / p->Hkv);
    const int n = keys_of(p, i);
    const uint16_t *qi = qrow(p, b, hq, i);
    for (int j = 0; j < n; ++j) {
        const uint16_t *kj = kvrow(p, p->k, b, g, j);
        double dot = 0.0;
        for (int c = 0; c < p->d; ++c) dot += bf(qi[c]) * bf(kj[c]);
        prob[j] = p->scale * dot;
    }
    double mx = -INFINITY;
    for (int j = 0; j < n; ++j)
        if (prob[j] > mx) mx = prob[j];
    double l = 0.0;
    for (int j = 0; j < n; ++j) {
        prob[j] = exp(prob[j] - mx);
        l += prob[j];
    }
    for (int j = 0; j < n; ++j) prob[j] /= l;
    if (lse) *lse = mx + log(l);
    if (dp) {
        const uint16_t *doi = dorow(p, b, hq, i);
        double D = 0.0;
        for (int j = 0; j < n; ++j) {
            const uint16_t *vj = kvrow(p, p->v, b, g, j);
            double dot = 0.0;
            for (int c = 0; c < p->d; ++c) dot += bf(doi[c]) * bf(vj[c]);
            dp[j] = dot;
            D += prob[j] * dot;
        }
        if (Dsum) *Dsum = D;
    }
    return n;
}

int oracle_bwd_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/*
 * Full backward: dq [B][Hq][Sq][d], dk and dv [B][Hkv][Skv][d] (fp64).
 * Work is split over (b, g): one thread owns a K/V head and walks every query
 * head of its group and every row, so each dK/dV row is summed in one fixed
 * order (deterministic).  dout may be NULL only if dq, dk and dv are all NULL.
 */
int oracle_attn_bwd_f64(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                        const uint16_t *dout, double *dq, double *dk, double *dv,
                        int B, int Hq, int Hkv, int Sq, int Skv, int d, int causal,
                        float scale, int nthreads)
{
    if (!q || !k || !v || !dout || !dq || !dk || !dv) return -1;
    if (bad_shape(B, Hq, Hkv, Sq, Skv, d)) return -2;
    threads(nthreads);
    const Problem P = {q, k, v, dout, B, Hq, Hkv, Sq, Skv, d, causal, (double)scale};
    const int group = Hq / Hkv;
    int failed = 0;
    memset(dk, 0, sizeof(double) * (size_t)B * Hkv * Skv * d);
    memset(dv, 0, sizeof(double) * (size_t)B * Hkv * Skv * d);
#pragma omp parallel
    {
        double *prob = (double *)malloc(sizeof(double) * (size_t)Skv);
        double *dp = (double *)malloc(sizeof(double) * (size_t)Skv);
        if (!prob || !dp) {
#pragma omp atomic write
            failed = 1;
        } else {
#pragma omp for schedule(dynamic, 1)
            for (int bg = 0; bg < B * Hkv; ++bg) {
                const int b = bg / Hkv, g = bg % Hkv;
                double *dkh = dk + (int64_t)bg * Skv * d;
                double *dvh = dv + (int64_t)bg * Skv * d;
                for (int hq = g * group; hq < (g + 1) * group; ++hq) {
                    for (int i = 0; i < Sq; ++i) {
                        double D;
                        const int n = row_softmax(&P, b, hq, i, prob, dp, NULL, &D);
                        const uint16_t *qi = qrow(&P, b, hq, i);
                        const uint16_t *doi = dorow(&P, b, hq, i);
                        double *dqi = dq + (((int64_t)b * Hq + hq) * Sq + i) * (int64_t)d;
                        for (int c = 0; c < d; ++c) dqi[c] = 0.0;
                        for (int j = 0; j < n; ++j) {
                            const double ds = prob[j] * (dp[j] - D);
                            const uint16_t *kj = kvrow(&P, k, b, g, j);
                            for (int c = 0; c < d; ++c) {
                                dqi[c] += P.scale * ds * bf(kj[c]);
                                dkh[(int64_t)j * d + c] += P.scale * ds * bf(qi[c]);
                                dvh[(int64_t)j * d + c] += prob[j] * bf(doi[c]);
                            }
                        }
                    }
                }
            }
        }
        free(prob);
        free(dp);
    }
    return failed ? -3 : 0;
}

/*
 * Row statistics of rows[n] = (b, hq, i): lse[n] and, when dout and Dsum are
 * given, D[n] = sum_j P_ij dP_ij.
 */
int oracle_attn_row_stats_f64(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                              const uint16_t *dout, const int64_t *rows, int64_t nrows,
                              double *lse, double *Dsum, int B, int Hq, int Hkv, int Sq,
                              int Skv, int d, int causal, float scale, int nthreads)
{
    if (!q || !k || !rows || !lse) return -1;
    if (Dsum && (!dout || !v)) return -1;
    if (bad_shape(B, Hq, Hkv, Sq, Skv, d)) return -2;
    for (int64_t r = 0; r < nrows; ++r) {
        const int64_t *x = rows + 3 * r;
        if (x[0] < 0 || x[0] >= B || x[1] < 0 || x[1] >= Hq || x[2] < 0 || x[2] >= Sq) return -2;
    }
    threads(nthreads);
    const Problem P = {q, k, v, dout, B, Hq, Hkv, Sq, Skv, d, causal, (double)scale};
    int failed = 0;
#pragma omp parallel
    {
        double *prob = (double *)malloc(sizeof(double) * (size_t)Skv);
        double *dp = (double *)malloc(sizeof(double) * (size_t)Skv);
        if (!prob || !dp) {
#pragma omp atomic write
            failed = 1;
        } else {
#pragma omp for schedule(dynamic, 16)
            for (int64_t r = 0; r < nrows; ++r) {
                const int64_t *x = rows + 3 * r;
                row_softmax(&P, (int)x[0], (int)x[1], (int)x[2], prob, Dsum ? dp : NULL,
                            lse + r, Dsum ? Dsum + r : NULL);
            }
        }
        free(prob);
        free(dp);
    }
    return failed ? -3 : 0;
}

/*
 * dQ rows of rows[n] = (b, hq, i) into dq[n][d]: each needs only its own row's
 * probabilities, so sampled rows are exact rows of the full dQ.
 */
int oracle_attn_bwd_dq_rows_f64(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                                const uint16_t *dout, const int64_t *rows, int64_t nrows,
                                double *dq, int B, int Hq, int Hkv, int Sq, int Skv, int d,
                                int causal, float scale, int nthreads)
{
    if (!q || !k || !v || !dout || !rows || !dq) return -1;
    if (bad_shape(B, Hq, Hkv, Sq, Skv, d)) return -2;
    for (int64_t r = 0; r < nrows; ++r) {
        const int64_t *x = rows + 3 * r;
        if (x[0] < 0 || x[0] >= B || x[1] < 0 || x[1] >= Hq || x[2] < 0 || x[2] >= Sq) return -2;
    }
    threads(nthreads);
    const Problem P = {q, k, v, dout, B, Hq, Hkv, Sq, Skv, d, causal, (double)scale};
    int failed = 0;
#pragma omp parallel
    {
        double *prob = (double *)malloc(sizeof(double) * (size_t)Skv);
        double *dp = (double *)malloc(sizeof(double) * (size_t)Skv);
        if (!prob || !dp) {
#pragma omp atomic write
            failed = 1;
        } else {
#pragma omp for schedule(dynamic, 4)
            for (int64_t r = 0; r < nrows; ++r) {
                const int64_t *x = rows + 3 * r;
                const int b = (int)x[0], hq = (int)x[1], i = (int)x[2];
                const int g = hq / (Hq / Hkv);
                double D;
                const int n = row_softmax(&P, b, hq, i, prob, dp, NULL, &D);
                double *out = dq + r * d;
                for (int c = 0; c < d; ++c) out[c] = 0.0;
                for (int j = 0; j < n; ++j) {
                    const double ds = prob[j] * (dp[j] - D);
                    const uint16_t *kj = kvrow(&P, k, b, g, j);
                    for (int c = 0; c < d; ++c) out[c] += P.scale * ds * bf(kj[c]);
                }
            }
        }
        free(prob);
        free(dp);
    }
    return failed ? -3 : 0;
}

/*
 * dK and dV rows of rows[n] = (b, g, j) into dk[n][d], dv[n][d], given the row
 * statistics lse and D of every query row [B][Hq][Sq] (from
 * oracle_attn_row_stats_f64): P_ij = exp(s_ij - lse_i), dS_ij = P_ij (dP_ij -
 * D_i), summed over the group's query heads and the rows that see key j.
 */
int oracle_attn_bwd_dkdv_rows_f64(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                                  const uint16_t *dout, const double *lse, const double *Dsum,
                                  const int64_t *rows, int64_t nrows, double *dk, double *dv,
                                  int B, int Hq, int Hkv, int Sq, int Skv, int d, int causal,
                                  float scale, int nthreads)
{
    if (!q || !k || !v || !dout || !lse || !Dsum || !rows || !dk || !dv) return -1;
    if (bad_shape(B, Hq, Hkv, Sq, Skv, d)) return -2;
    for (int64_t r = 0; r < nrows; ++r) {
        const int64_t *x = rows + 3 * r;
        if (x[0] < 0 || x[0] >= B || x[1] < 0 || x[1] >= Hkv || x[2] < 0 || x[2] >= Skv) return -2;
    }
    threads(nthreads);
    const Problem P = {q, k, v, dout, B, Hq, Hkv, Sq, Skv, d, causal, (double)scale};
    const int group = Hq / Hkv;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t r = 0; r < nrows; ++r) {
        const int64_t *x = rows + 3 * r;
        const int b = (int)x[0], g = (int)x[1], j = (int)x[2];
        const uint16_t *kj = kvrow(&P, k, b, g, j);
        const uint16_t *vj = kvrow(&P, v, b, g, j);
        double *dkr = dk + r * d, *dvr = dv + r * d;
        for (int c = 0; c < d; ++c) dkr[c] = dvr[c] = 0.0;
        for (int hq = g * group; hq < (g + 1) * group; ++hq) {
            for (int i = 0; i < Sq; ++i) {
                if (j >= keys_of(&P, i)) continue;   /* key j not in J_i */
                const uint16_t *qi = qrow(&P, b, hq, i);
                const uint16_t *doi = dorow(&P, b, hq, i);
                double s = 0.0, dp = 0.0;
                for (int c = 0; c < d; ++c) {
                    s += bf(qi[c]) * bf(kj[c]);
                    dp += bf(doi[c]) * bf(vj[c]);
                }
                const int64_t row = ((int64_t)b * Hq + hq) * Sq + i;
                const double prob = exp(P.scale * s - lse[row]);
                const double ds = prob * (dp - Dsum[row]);
                for (int c = 0; c < d; ++c) {
                    dkr[c] += P.scale * ds * bf(qi[c]);
                    dvr[c] += prob * bf(doi[c]);
                }
            }
        }
    }
    return 0;
}
