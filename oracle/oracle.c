/*
 * CPU oracle for the ShiftAddLLM reparameterized linear layer.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this library.  The product path (the
 * HIP library and its Python binding) never calls it and shares no code with
 * it.
 *
 * Everything here is the plain definition, in fp64, with no blocking, fusion or
 * reordering beyond what the definition states:
 *
 *   W_q = sum_i alpha_i b_i                        (Sec. 3, BCQ)
 *   alpha = sign(alpha) 2^P                        (Sec. 4.1, Eq. 2, one term)
 *   y = x W_q^T                                    (the layer)
 *
 * with one power-of-two factor per (plane i, output row n, group g of G
 * consecutive input columns) and the factor's sign folded into the plane, so
 *
 *   y[b][n] = sum_i sum_g 2^e[i][n][g] * sum_{k in g} s_i[n][k] * x[b][k].
 *
 * The table of Sec. 4.1 ("Queries and adds"): for every 8 consecutive
 * activations, 256 signed partial sums keyed by an 8-bit weight pattern,
 *
 *   lut[b][c][m] = sum_{j<8} (bit j of m ? +1 : -1) * x[b][8c+j],
 *
 * with bit j of the key standing for column 8c+j (least significant bit first)
 * and a set bit meaning +1.  The packed form of a plane uses the same key
 * convention: byte c of row n is sum_j [s[n][8c+j] > 0] << j.
 *
 * Activations are passed as fp64 (the exact values of the fp16 inputs).
 */
#include <math.h>
#include <stdint.h>
#include <stddef.h>

#ifdef _OPENMP
#include <omp.h>
#endif

static void set_threads(int nthreads)
{
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#else
    (void)nthreads;
#endif
}

/* Number of threads an OpenMP parallel region will use after set_threads(). */
int oracle_max_threads(int nthreads)
{
    set_threads(nthreads);
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Canonical packing: packed[i][n][c] = sum_j [signs[i][n][8c+j] > 0] << j.
 * Entries <= 0 count as -1 (bit 0). */
void oracle_pack(const int8_t *signs, int64_t q, int64_t N, int64_t K, uint8_t *packed)
{
    const int64_t C = K / 8;
    for (int64_t i = 0; i < q; ++i)
        for (int64_t n = 0; n < N; ++n)
            for (int64_t c = 0; c < C; ++c) {
                unsigned v = 0;
                for (int j = 0; j < 8; ++j)
                    if (signs[(i * N + n) * K + 8 * c + j] > 0) v |= 1u << j;
                packed[(i * N + n) * C + c] = (uint8_t)v;
            }
}

/* Inverse of oracle_pack: bit j of byte c -> +1 if set, -1 if clear. */
void oracle_unpack(const uint8_t *packed, int64_t q, int64_t N, int64_t K, int8_t *signs)
{
    const int64_t C = K / 8;
    for (int64_t i = 0; i < q; ++i)
        for (int64_t n = 0; n < N; ++n)
            for (int64_t c = 0; c < C; ++c) {
                unsigned v = packed[(i * N + n) * C + c];
                for (int j = 0; j < 8; ++j)
                    signs[(i * N + n) * K + 8 * c + j] = ((v >> j) & 1u) ? 1 : -1;
            }
}

/* Table of Sec. 4.1: lut[b][c][m] = sum_{j<8} (2*bit_j(m) - 1) * x[b][8c+j]. */
void oracle_lut(const double *x, int64_t B, int64_t K, double *lut)
{
    const int64_t C = K / 8;
    for (int64_t b = 0; b < B; ++b)
        for (int64_t c = 0; c < C; ++c)
            for (int m = 0; m < 256; ++m) {
                double s = 0.0;
                for (int j = 0; j < 8; ++j) {
                    double sign = ((m >> j) & 1) ? 1.0 : -1.0;
                    s += sign * x[b * K + 8 * c + j];
                }
                lut[(b * C + c) * 256 + m] = s;
            }
}

/*
 * The layer at one output (b, n):
 *   y       = sum_i sum_g ldexp( sum_{k in g} s_i[n][k] x[b][k], e[i][n][g] )
 *   absterm = sum_i sum_k 2^e[i][n][k/G] |x[b][k]|   (the sum of |terms|)
 * Loops run planes, then groups, then columns, each in increasing order.
 */
static void one_output(const double *xb, const int8_t *signs, const int8_t *exps,
                       int64_t q, int64_t N, int64_t K, int64_t G, int64_t n,
                       double *y, double *absterm)
{
    const int64_t NG = K / G;
    double total = 0.0, abs_total = 0.0;
    for (int64_t i = 0; i < q; ++i) {
        const int8_t *s = signs + (i * N + n) * K;
        const int8_t *e = exps + (i * N + n) * NG;
        for (int64_t g = 0; g < NG; ++g) {
            double part = 0.0, apart = 0.0;
            for (int64_t k = g * G; k < (g + 1) * G; ++k) {
                part += (double)s[k] * xb[k];
                apart += fabs(xb[k]);
            }
            total += ldexp(part, e[g]);
            abs_total += ldexp(apart, e[g]);
        }
    }
    *y = total;
    *absterm = abs_total;
}

/* signs: int8 [q][N][K] in {-1,+1}; exps: int8 [q][N][K/G]; x: fp64 [B][K];
 * y, absterm: fp64 [B][N] (absterm may be NULL). */
void oracle_shiftadd_gemm(const double *x, const int8_t *signs, const int8_t *exps,
                          int64_t q, int64_t N, int64_t K, int64_t G, int64_t B,
                          double *y, double *absterm, int nthreads)
{
    set_threads(nthreads);
#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t b = 0; b < B; ++b)
        for (int64_t n = 0; n < N; ++n) {
            double v, a;
            one_output(x + b * K, signs, exps, q, N, K, G, n, &v, &a);
            y[b * N + n] = v;
            if (absterm) absterm[b * N + n] = a;
        }
}

/* The same definition on a list of output rows (sampled checks at full sizes):
 * y[b][t], absterm[b][t] for row n = rows[t], t < nrows. */
void oracle_shiftadd_gemm_rows(const double *x, const int8_t *signs, const int8_t *exps,
                               int64_t q, int64_t N, int64_t K, int64_t G, int64_t B,
                               const int64_t *rows, int64_t nrows,
                               double *y, double *absterm, int nthreads)
{
    set_threads(nthreads);
#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t b = 0; b < B; ++b)
        for (int64_t t = 0; t < nrows; ++t) {
            double v, a;
            one_output(x + b * K, signs, exps, q, N, K, G, rows[t], &v, &a);
            y[b * nrows + t] = v;
            if (absterm) absterm[b * nrows + t] = a;
        }
}

/*
 * The layer with column-wise scaling factors ("Ours (Acc.)", Sec. 4.2: one
 * factor per plane and weight column, i.e. per input activation, here a power
 * of two by Eq. 2) at one output (b, n):
 *   y       = sum_i sum_k s_i[n][k] * ldexp(x[b][k], e[i][k])
 *   absterm = sum_i sum_k 2^e[i][k] |x[b][k]|
 * Loops run planes, then columns, in increasing order.
 */
static void one_output_col(const double *xb, const int8_t *signs, const int8_t *col_exps,
                           int64_t q, int64_t N, int64_t K, int64_t n,
                           double *y, double *absterm)
{
    double total = 0.0, abs_total = 0.0;
    for (int64_t i = 0; i < q; ++i) {
        const int8_t *s = signs + (i * N + n) * K;
        const int8_t *e = col_exps + i * K;
        for (int64_t k = 0; k < K; ++k) {
            const double xs = ldexp(xb[k], e[k]);
            total += (double)s[k] * xs;
            abs_total += fabs(xs);
        }
    }
    *y = total;
    *absterm = abs_total;
}

/* signs: int8 [q][N][K]; col_exps: int8 [q][K]; x: fp64 [B][K]; rows: NULL
 * for every output row, else the list of rows (nrows of them); y, absterm:
 * fp64 [B][rows] (absterm may be NULL). */
void oracle_shiftadd_gemm_colwise(const double *x, const int8_t *signs, const int8_t *col_exps,
                                  int64_t q, int64_t N, int64_t K, int64_t B,
                                  const int64_t *rows, int64_t nrows,
                                  double *y, double *absterm, int nthreads)
{
    const int64_t R = rows ? nrows : N;
    set_threads(nthreads);
#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t b = 0; b < B; ++b)
        for (int64_t t = 0; t < R; ++t) {
            double v, a;
            one_output_col(x + b * K, signs, col_exps, q, N, K, rows ? rows[t] : t, &v, &a);
            y[b * R + t] = v;
            if (absterm) absterm[b * R + t] = a;
        }
}

/*
 * The layer with block-wise scaling factors ("Ours (Lat.)", Sec. 4.2: 8
 * columns and a block of rows share one factor, here a power of two by Eq. 2)
 * at one output (b, n), rows in blocks of row_block:
 *   y       = sum_i sum_c ldexp( sum_{j<8} s_i[n][8c+j] x[b][8c+j], E[i][n / row_block][c] )
 *   absterm = sum_i sum_k 2^E[i][n / row_block][k / 8] |x[b][k]|
 * Loops run planes, then chunks, then columns, in increasing order.
 */
static void one_output_blk(const double *xb, const int8_t *signs, const int8_t *blk_exps,
                           int64_t q, int64_t N, int64_t K, int64_t row_block, int64_t n,
                           double *y, double *absterm)
{
    const int64_t C = K / 8, NB = (N + row_block - 1) / row_block;
    double total = 0.0, abs_total = 0.0;
    for (int64_t i = 0; i < q; ++i) {
        const int8_t *s = signs + (i * N + n) * K;
        const int8_t *e = blk_exps + (i * NB + n / row_block) * C;
        for (int64_t c = 0; c < C; ++c) {
            double part = 0.0, apart = 0.0;
            for (int64_t k = 8 * c; k < 8 * c + 8; ++k) {
                part += (double)s[k] * xb[k];
                apart += fabs(xb[k]);
            }
            total += ldexp(part, e[c]);
            abs_total += ldexp(apart, e[c]);
        }
    }
    *y = total;
    *absterm = abs_total;
}

/* signs: int8 [q][N][K]; blk_exps: int8 [q][ceil(N / row_block)][K/8]; x: fp64
 * [B][K]; rows: NULL for every output row, else nrows rows; y, absterm: fp64
 * [B][rows] (absterm may be NULL). */
void oracle_shiftadd_gemm_blockwise(const double *x, const int8_t *signs, const int8_t *blk_exps,
                                    int64_t q, int64_t N, int64_t K, int64_t row_block, int64_t B,
                                    const int64_t *rows, int64_t nrows,
                                    double *y, double *absterm, int nthreads)
{
    const int64_t R = rows ? nrows : N;
    set_threads(nthreads);
#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t b = 0; b < B; ++b)
        for (int64_t t = 0; t < R; ++t) {
            double v, a;
            one_output_blk(x + b * K, signs, blk_exps, q, N, K, row_block, rows ? rows[t] : t,
                           &v, &a);
            y[b * R + t] = v;
            if (absterm) absterm[b * R + t] = a;
        }
}

/*
 * The layer with additive power-of-two factors (Eq. 2 with T terms): the
 * factor of (plane i, row n, group g) is sum_t sg[i][n][g][t] 2^e[i][n][g][t]
 * with term signs in {-1, 0, +1} (0: no term), so that
 *   y       = sum_i sum_g sum_t sg_t ldexp( sum_{k in g} s_i[n][k] x[b][k], e_t )
 *   absterm = sum_i sum_g sum_t |sg_t| ldexp( sum_{k in g} |x[b][k]|, e_t )
 * Loops run planes, then groups, then terms, then columns.
 */
static void one_output_terms(const double *xb, const int8_t *signs, const int8_t *exps,
                             const int8_t *term_signs, int64_t T, int64_t q, int64_t N,
                             int64_t K, int64_t G, int64_t n, double *y, double *absterm)
{
    const int64_t NG = K / G;
    double total = 0.0, abs_total = 0.0;
    for (int64_t i = 0; i < q; ++i) {
        const int8_t *s = signs + (i * N + n) * K;
        for (int64_t g = 0; g < NG; ++g) {
            double part = 0.0, apart = 0.0;
            for (int64_t k = g * G; k < (g + 1) * G; ++k) {
                part += (double)s[k] * xb[k];
                apart += fabs(xb[k]);
            }
            const int64_t at = ((i * N + n) * NG + g) * T;
            for (int64_t t = 0; t < T; ++t) {
                const int sg = term_signs[at + t];
                if (sg == 0) continue;
                total += (double)sg * ldexp(part, exps[at + t]);
                abs_total += ldexp(apart, exps[at + t]);
            }
        }
    }
    *y = total;
    *absterm = abs_total;
}

/* exps, term_signs: int8 [q][N][K/G][T]; other arguments as
 * oracle_shiftadd_gemm_blockwise. */
void oracle_shiftadd_gemm_terms(const double *x, const int8_t *signs, const int8_t *exps,
                                const int8_t *term_signs, int64_t T, int64_t q, int64_t N,
                                int64_t K, int64_t G, int64_t B, const int64_t *rows,
                                int64_t nrows, double *y, double *absterm, int nthreads)
{
    const int64_t R = rows ? nrows : N;
    set_threads(nthreads);
#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t b = 0; b < B; ++b)
        for (int64_t t = 0; t < R; ++t) {
            double v, a;
            one_output_terms(x + b * K, signs, exps, term_signs, T, q, N, K, G,
                             rows ? rows[t] : t, &v, &a);
            y[b * R + t] = v;
            if (absterm) absterm[b * R + t] = a;
        }
}
