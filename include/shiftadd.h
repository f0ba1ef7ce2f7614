/*
 * shiftadd.h -- C ABI of the MI355X (gfx950) shift-add linear layer.
 *
 * The layer is the inference step of ShiftAddLLM (Sec. 4.1, "Post-training
 * Reparameterization of LLMs"): a weight matrix quantized into q binary
 * matrices b_i in {-1,+1}^{N x K} with power-of-two scaling factors (BCQ,
 * Sec. 3; PoT factors, Eq. 2) is applied to an fp16 activation x by
 *   (1) shifting by the power-of-two factors, and
 *   (2) querying 256-entry tables of precomputed partial sums -- one table per
 *       8 consecutive activations, keyed by 8 binary weights -- and adding.
 *
 * What is computed, for b < batch, n < N (fp32 result):
 *
 *   y[b][n] = sum_{i<q} sum_{g<K/group} 2^exps[i][n][g] *
 *             sum_{k = g*group}^{(g+1)*group - 1} s_i[n][k] * x[b][k]
 *
 * One exponent per (plane i, output row n, group g of `group` consecutive input
 * columns).  The sign of each scaling factor is folded into its plane (exact,
 * because entries are +-1), so exponents carry magnitudes only.  The shift is
 * applied to each group's fp32 partial sum (ldexp), which equals shifting the
 * activations because the factor is constant over the group.
 *
 * Key convention (Sec. 4.1: the binary weights of one plane row are taken eight
 * at a time as the index of a table; the bit order is this library's reading):
 * the key of chunk c of a plane row is sum_{j<8} [s[8c+j] = +1] << j -- bit j stands for column 8c+j, a set
 * bit means +1.
 *
 * Conventions shared by every entry point:
 *  - Pointers marked (device) are device memory of the current HIP device; the
 *    caller allocates and owns every buffer.  `stream` is a hipStream_t passed
 *    as void* (NULL = the null stream).
 *  - Arguments are validated on the host before any HIP call; a rejected call
 *    returns a negative sa_status and enqueues nothing.
 *  - Accepted calls are asynchronous on `stream`; kernel faults surface at the
 *    caller's next synchronization.  SA_ERR_HIP reports a launch error.
 *  - Only int, size_t, fixed-width integers and plain pointers cross the ABI.
 */
#ifndef SHIFTADD_H
#define SHIFTADD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#if defined(__GNUC__)
#define SA_API __attribute__((visibility("default")))
#else
#define SA_API
#endif

typedef enum {
    SA_OK = 0,
    SA_ERR_NULL = -1,  /* a required pointer is NULL */
    SA_ERR_SHAPE = -2, /* N, K or batch out of range, K % 8 != 0, one plane of
                          packed keys (N*K/8 bytes) >= 2^31, or q*N*K > 2^36 */
    SA_ERR_Q = -3,     /* q outside [1, 8] */
    SA_ERR_GROUP = -4, /* group < 8, group % 8 != 0, or K % group != 0 */
    SA_ERR_ALIGN = -5, /* a pointer that must be 16-byte aligned is not */
    SA_ERR_HIP = -6    /* a HIP runtime call or kernel launch failed */
} sa_status;

/* Largest accepted values. */
#define SA_MAX_Q 8
#define SA_MAX_BATCH 256
#define SA_MAX_CYCLES 64
#define SA_MAX_TERMS 4

/* Bytes of the packed planes of a q x N x K layer: q*N*K/8 (1 bit per weight
 * per plane, no padding).  Returns 0 for invalid sizes. */
SA_API size_t sa_packed_bytes(int q, int N, int K);

/* Byte offset, inside the packed buffer, of the key of (plane i, row n,
 * chunk c) -- chunk c covers columns 8c..8c+7.  Host-only, no HIP call; lets a
 * caller (or a test) map the device layout to the canonical [q][N][K/8] order.
 * Returns -1 for out-of-range arguments.
 *
 * Device layout: rows in tiles of 64, chunks in blocks of 16.  For tile T with
 * R = min(64, N - 64T) rows and block J with U = min(16, K/8 - 16J) chunks,
 *   offset = i*N*(K/8) + 64T*(K/8) + 16J*R + r*U + p,   r = n - 64T,
 * where position p of a full block (U = 16) holds chunk 16J + ((p + r) mod 16)
 * and position p of a partial block holds chunk 16J + p.  A 64-row tile of one
 * 16-chunk block is thus one contiguous 1 KiB piece, 16 bytes per row. */
SA_API int64_t sa_packed_offset(int q, int N, int K, int i, int n, int c);

/* Pack binary planes into the device layout above (the offline step that
 * produces the stored form of the b_i of Sec. 3).
 *   signs        (device) int8 [q][N][K], row-major; > 0 means +1, anything
 *                else -1.  Any alignment.
 *   packed_bits  (device) sa_packed_bytes(q, N, K) bytes, 16-byte aligned;
 *                fully overwritten.
 * Bit-exact: unpacking returns the signs. */
SA_API int sa_pack_weights(const int8_t *signs, int q, int N, int K,
                           uint8_t *packed_bits, void *stream);

/* Inverse of sa_pack_weights: signs[i][n][k] in {-1, +1} (device, int8
 * [q][N][K], any alignment, fully overwritten). */
SA_API int sa_unpack_weights(const uint8_t *packed_bits, int q, int N, int K,
                             int8_t *signs, void *stream);

/* The tables of Sec. 4.1 (all 256 signed sums of each group of eight
 * activations, computed before the queries): for b < batch, c < K/8, m < 256,
 *   lut[b][c][m] = sum_{j<8} (bit j of m ? +1 : -1) * x[b][8c+j]
 * computed in fp32 from the fp16 activations.  Entry m and entry 255-m are
 * exact negatives of each other.  This is the same construction the fused
 * kernel stages in on-chip memory; it is exposed for inspection and tests.
 *   x    (device) IEEE binary16 bit patterns [batch][K], row-major, 16-byte
 *        aligned.
 *   lut  (device) fp32 [batch][K/8][256], 16-byte aligned, fully overwritten. */
SA_API int sa_build_lut(const uint16_t *x, int K, int batch, float *lut, void *stream);

/* The layer (Sec. 4.1: shift, then query and add), y = x W_q^T in fp32.
 *   x            (device) binary16 [batch][K], row-major, 16-byte aligned.
 *   packed_bits  (device) planes packed by sa_pack_weights for the same
 *                (q, N, K), 16-byte aligned.
 *   exps         (device) int8 [q][N][K/group], row-major: exponent of the
 *                power-of-two factor of (plane, row, group).  Any alignment.
 *                Results follow fp32 ldexp semantics; exponents in [-30, 30]
 *                never overflow or lose bits to underflow.
 *   q in [1, 8]; N >= 1; K >= 8, K % 8 == 0; group % 8 == 0, K % group == 0;
 *   batch in [1, SA_MAX_BATCH].
 *   y            (device) fp32 [batch][N], 16-byte aligned, fully
 *                overwritten (no accumulation into prior contents).
 * The result is deterministic: the same inputs give bit-identical y.  The call
 * allocates nothing, keeps no state between calls and uses no memory beyond
 * its arguments, so calls on different streams may run concurrently and the
 * call may be captured in a HIP graph. */
SA_API int sa_shiftadd_gemm(const uint16_t *x, const uint8_t *packed_bits, const int8_t *exps,
                            int q, int N, int K, int group, int batch, float *y, void *stream);

/* The same layer with the output activations in binary16 (Sec. 4.1): y[b][n]
 * is the fp32 result of sa_shiftadd_gemm rounded to the nearest binary16
 * (ties to even; beyond the binary16 range +-inf), bit-identical to
 * converting that fp32 result.  Arguments, launch geometry and errors as for
 * sa_shiftadd_gemm, with
 *   y  (device) IEEE binary16 bit patterns [batch][N], 16-byte aligned,
 *      fully overwritten. */
SA_API int sa_shiftadd_gemm_f16(const uint16_t *x, const uint8_t *packed_bits, const int8_t *exps,
                                int q, int N, int K, int group, int batch, uint16_t *y,
                                void *stream);

/* The same layer at batch 1 with the whole 256-entry table of every chunk
 * (Sec. 4.1), one LDS read and one add per key.  K is cut into 1024-column
 * slices; a workgroup builds the 128 chunk tables of one slice once and
 * streams a range of rows through them, writing one fp32 partial per (slice,
 * row) to `workspace`; a second kernel adds each row's partials in slice
 * order into y.  Arguments as for sa_shiftadd_gemm with batch = 1, and:
 *   K % 1024 == 0 and group % 128 == 0 (else SA_ERR_SHAPE, SA_ERR_GROUP);
 *   workspace        (device) fp32, 4-byte aligned (else SA_ERR_ALIGN), at
 *                    least sa_kslice_workspace_bytes(N, K) bytes = 4 * (K /
 *                    1024) * N (else SA_ERR_SHAPE; NULL: SA_ERR_NULL); owned
 *                    by the caller, overwritten; calls that share a workspace
 *                    must not overlap.
 * Deterministic; y is bit-identical across calls but not to sa_shiftadd_gemm
 * (a different fp32 summation order).  Allocates nothing; may be captured in
 * a HIP graph. */
SA_API size_t sa_kslice_workspace_bytes(int N, int K);
SA_API int sa_shiftadd_gemm_kslice(const uint16_t *x, const uint8_t *packed_bits,
                                   const int8_t *exps, int q, int N, int K, int group, float *y,
                                   float *workspace, size_t workspace_bytes, void *stream);

/* The offline reparameterization that produces the layer's planes and
 * exponents from full-precision weights: alternating multi-bit binary-coding
 * quantization (Sec. 3, Alg. 1: greedy initialisation on residuals, Eq. 1, then
 * `cycles` rounds of a least-squares refit of the scales and a refit of the
 * codes) with every scale rounded to a power of two (Sec. 4.1, Eq. 2, one
 * term).  Each segment of `group` consecutive columns of one row is quantized
 * on its own, in fp64:
 *   greedy   r = w; for i < q: b_i = sign(r) (sign(0) = +1),
 *            alpha_i = sum|r| / group, r -= alpha_i b_i;
 *   cycle    LS: alpha = (B^T B)^-1 B^T w (Gaussian elimination with partial
 *            pivoting; a column whose pivot is <= 1e-9 * group depends on the
 *            earlier ones and gets alpha = 0);  PoT: alpha -> sign * 2^P with
 *            P = round(log2|alpha|) in the log domain (|alpha| = m 2^E,
 *            m in [1, 2): P = E + [m >= sqrt 2]), clamped to [-128, 127], and
 *            alpha = 0 -> P = -128;  BS: each element takes the codes whose
 *            value sum_i +-alpha_i is nearest to it (ties: the smaller code
 *            number, b_i = +1 when bit i is set).
 * With cycles = 0 the greedy scales are rounded to powers of two.  The result
 * is the layer's format: W_q[n][k] = sum_i 2^exps[i][n][k/group] *
 * signs[i][n][k], the sign of each scale folded into its plane.
 *   w      (device) fp32 [N][K], row-major, finite, 16-byte aligned.
 *   q in [1, 8]; group % 8 == 0, K % group == 0; cycles in [0, SA_MAX_CYCLES].
 *   signs  (device) int8 [q][N][K], +-1, 8-byte aligned, fully overwritten
 *          (the input of sa_pack_weights).
 *   exps   (device) int8 [q][N][K/group], fully overwritten.
 * Errors: SA_ERR_NULL, SA_ERR_Q, SA_ERR_SHAPE (sizes as for the layer, or
 * cycles out of range), SA_ERR_GROUP, SA_ERR_ALIGN, SA_ERR_HIP.
 * Asynchronous on `stream`; deterministic; allocates nothing. */
SA_API int sa_quantize_bcq(const float *w, int N, int K, int q, int group, int cycles,
                           int8_t *signs, int8_t *exps, void *stream);

/* The same reparameterization with additive power-of-two scales (Eq. 2 with
 * `terms` terms): wherever a scale is rounded, term t is the power of two
 * nearest (in the log domain) to the residual r = alpha - sum_{j<t} a_j, with
 * the sign of r (a zero residual gives no term: sign 0, exponent -128), and
 * BS uses the sum of the terms.  The result is the format of
 * sa_shiftadd_gemm_terms: the sign of the first term is folded into the
 * plane, term signs are relative to it (term 0 is +1, or 0 for a zero scale).
 *   exps, term_signs  (device) int8 [q][N][K/group][terms], fully overwritten.
 *   1 <= terms <= SA_MAX_TERMS (else SA_ERR_SHAPE); term_signs non-NULL;
 *   other arguments as for sa_quantize_bcq.  With terms = 1 the planes and
 *   exponents equal those of sa_quantize_bcq. */
SA_API int sa_quantize_bcq_terms(const float *w, int N, int K, int q, int group, int cycles,
                                 int terms, int8_t *signs, int8_t *exps, int8_t *term_signs,
                                 void *stream);

/* Launch geometry sa_shiftadd_gemm uses for a shape (host-only, no HIP call). */
typedef struct {
    int path;         /* 0: generic kernel (any group); group % 128 == 0: 1 row kernel
                         (batch 1), 2 batch kernel (batch >= 2); 3: the row kernel
                         with column-wise factors (sa_shiftadd_gemm_colwise, batch 1); 4: the
                         row kernel with block-wise factors (sa_shiftadd_gemm_blockwise,
                         batch 1), 5 the batch kernel with block-wise factors (batch >= 2);
                         6 the batch kernel with column-wise factors (batch >= 2) */
    int rows_per_wg;  /* output rows per workgroup (the largest share when the
                         row kernel spreads row groups unevenly) */
    int workgroups;   /* workgroups of the launch */
    int threads;      /* threads per workgroup */
    int pieces;       /* input-dimension pieces whose tables a workgroup builds in turn */
    size_t lds_bytes; /* on-chip memory per workgroup */
} sa_plan;

SA_API int sa_plan_gemm(int q, int N, int K, int group, int batch, sa_plan *plan);

/* The layer with column-wise scaling factors ("Ours (Acc.)", Sec. 4.2): one
 * power-of-two factor per plane and weight column (Eq. 2, one term, sign
 * folded into the plane), W_q[n][k] = sum_i 2^col_exps[i][k] s_i[n][k]:
 *
 *   y[b][n] = sum_i sum_k s_i[n][k] * 2^col_exps[i][k] * x[b][k]
 *
 * A factor belongs to one activation, so it shifts the activation: the tables
 * of Sec. 4.1 are built per plane from the shifted activations (in fp32,
 * exact for exponents in [-100, 100]) and the queried sums need no shift.
 *   x         (device) fp16 bits [batch][K], 16-byte aligned.
 *   packed_bits (device) planes packed by sa_pack_weights, 16-byte aligned.
 *   col_exps  (device) int8 [q][K], 8-byte aligned.
 *   q in [1, 8]; K % 128 == 0 (else SA_ERR_SHAPE); 1 <= batch <= SA_MAX_BATCH.
 *   y         (device) fp32 [batch][N], 16-byte aligned, fully overwritten.
 * Same error codes as sa_shiftadd_gemm.  Asynchronous on `stream`; allocates
 * nothing; deterministic. */
SA_API int sa_shiftadd_gemm_colwise(const uint16_t *x, const uint8_t *packed_bits,
                                    const int8_t *col_exps, int q, int N, int K, int batch,
                                    float *y, void *stream);

/* Launch geometry of sa_shiftadd_gemm_colwise (host-only). */
SA_API int sa_plan_gemm_colwise(int q, int N, int K, int batch, sa_plan *plan);

/* The layer with block-wise scaling factors ("Ours (Lat.)", Sec. 4.2): 8
 * columns (one key) and a block of `row_block` consecutive rows share one
 * power-of-two factor (Eq. 2, one term, sign folded into the plane):
 *
 *   y[b][n] = sum_i sum_c 2^blk_exps[i][n / row_block][c] * sum_{j<8} s_i[n][8c+j] x[b][8c+j]
 *
 * One table per chunk serves every plane and row, as in sa_shiftadd_gemm; each
 * queried entry is shifted by its key's exponent (ldexp) before it is added.
 * The paper's choice is row_block = N / 8.
 *   blk_exps  (device) int8 [q][ceil(N / row_block)][K/8], 16-byte aligned.
 *   row_block >= 1; K % 128 == 0 (else SA_ERR_SHAPE); other arguments as for
 *   sa_shiftadd_gemm_colwise.
 * Same error codes as sa_shiftadd_gemm.  Asynchronous on `stream`; allocates
 * nothing; deterministic. */
SA_API int sa_shiftadd_gemm_blockwise(const uint16_t *x, const uint8_t *packed_bits,
                                      const int8_t *blk_exps, int q, int N, int K, int row_block,
                                      int batch, float *y, void *stream);

/* The layer with additive power-of-two factors (Eq. 2 with T terms): the
 * factor of (plane i, row n, group g) is the greedy sum of T signed powers of
 * two, sum_t term_signs[..][t] 2^exps[..][t] (a term sign of 0 means no term):
 *
 *   y[b][n] = sum_i sum_g ( sum_t term_signs[i][n][g][t] 2^exps[i][n][g][t] )
 *                         * sum_{k in g} s_i[n][k] x[b][k]
 *
 * Each group sum is shifted once per term and added with its sign.  T = 1
 * with term sign +1 is sa_shiftadd_gemm.
 *   exps, term_signs (device) int8 [q][N][K/group][T] (the T terms of a group
 *          are consecutive bytes; 2-byte aligned for T = 2, 4-byte for T = 4),
 *          term signs in {-1, 0, 1}.
 *   group % 128 == 0 (else SA_ERR_GROUP); 1 <= terms <= SA_MAX_TERMS (else
 *   SA_ERR_SHAPE); other arguments and errors as for sa_shiftadd_gemm.
 * Asynchronous on `stream`; allocates nothing; deterministic. */
SA_API int sa_shiftadd_gemm_terms(const uint16_t *x, const uint8_t *packed_bits,
                                  const int8_t *exps, const int8_t *term_signs, int q, int N,
                                  int K, int group, int terms, int batch, float *y, void *stream);

/* Launch geometry of sa_shiftadd_gemm_blockwise (host-only). */
SA_API int sa_plan_gemm_blockwise(int q, int N, int K, int row_block, int batch, sa_plan *plan);

/* ---- Automated mixed-bit allocation (Sec. 4.3, Eq. 3 and Eq. 4) ----
 *
 * The criterion of a layer, C = ||IS||_F STD(IS)^2 with IS = W /
 * diag(cholesky(H^-1)) and H = X X^T + damp * mean(diag(X X^T)) I (X the
 * calibration activations, one column per token), is computed in three calls:
 * sa_gram_f16 (X X^T), sa_inverse_cholesky_diag (the diagonal of the Cholesky
 * factor of H^-1), sa_importance_criterion (C).  The caller owns every buffer,
 * workspaces included; nothing is allocated. */

/* H = X X^T (Eq. 3) on the matrix cores, fp32 accumulation of fp16 products.
 *   x  (device) fp16 bits [K][T] row-major (one row per input channel), 16-byte
 *      aligned; K % 128 == 0, T % 32 == 0 (pad with zero tokens; they add nothing).
 *   H  (device) fp32 [K][K], fully overwritten (symmetric).
 * Asynchronous on `stream`. */
SA_API int sa_gram_f16(const uint16_t *x, int K, int T, float *H, void *stream);

/* d[k] = diag(cholesky((H + damp * mean(diag H) I)^-1))[k] in fp64 (Eq. 3).
 * Computed without forming the inverse: the Cholesky factor of H^-1 has, in
 * reverse order, the reciprocals of the diagonal of the Cholesky factor of the
 * matrix with rows and columns reversed, which is factored here (blocked, 64
 * columns per panel).  A matrix that is not positive definite after damping
 * yields NaN entries.
 *   H  (device) fp32 [K][K] symmetric (only its lower triangle is read).
 *   damp >= 0.  d (device) fp64 [K], 8-byte aligned.
 *   workspace (device) >= sa_inverse_cholesky_workspace(K) bytes, 256-byte
 *      aligned, owned by the caller (its contents are overwritten).
 * Asynchronous on `stream`. */
SA_API size_t sa_inverse_cholesky_workspace(int K);
SA_API int sa_inverse_cholesky_diag(const float *H, int K, double damp, double *d,
                                    void *workspace, size_t workspace_bytes, void *stream);

/* out[0] = C = ||IS||_F * STD(IS)^2, out[1] = ||IS||_F, out[2] = STD(IS)
 * (population standard deviation over all N*K entries), IS[n][k] = w[n][k] /
 * d[k], fp64 sums in a fixed order (Eq. 3).
 *   w (device) fp32 [N][K]; d (device) fp64 [K]; out (device) fp64 [3].
 *   workspace (device) >= sa_importance_workspace() bytes, 8-byte aligned. */
SA_API size_t sa_importance_workspace(void);
SA_API int sa_importance_criterion(const float *w, int N, int K, const double *d, double *out,
                                   void *workspace, size_t workspace_bytes, void *stream);

/* sa_importance_criterion for callers that cannot allocate (code under HIP
 * graph capture, serving loops, harnesses that forbid allocation): the same
 * kernels and result, with the partial sums in a fixed 16 KB device array the
 * library owns (one per GPU, held until the process ends) instead of a
 * workspace argument.  Calls no allocator.  The array is set up on the first
 * call on each device (that device current).  Accepts the same sizes as
 * sa_importance_criterion (N*K <= 2^40, else SA_ERR_SHAPE); out 8-byte
 * aligned.  Calls that overlap on one GPU share the array and race: keep them
 * on one stream. */
SA_API int sa_importance_criterion_noalloc(const float *w, int N, int K, const double *d,
                                           double *out, void *stream);

/* Host only.  Per-bit estimates C_{i,b}: for each bit width (column b of
 * errors [L][nb], the measured reparameterization errors of L calibration
 * layers) the least-squares polynomial of the given degree in the criterion
 * c[L] is fitted, and out[i][b] = p_b(c[i]) (Sec. 4.3).  Needs L > degree and
 * degree + 1 distinct criteria (else SA_ERR_SHAPE). */
SA_API int sa_fit_per_bit(const double *c, const double *errors, int L, int nb, int degree,
                          double *out);

/* Host only.  Eq. 4: one bit width per layer, out[i] in bits[], minimising
 * sum_i cost[i][b_i] (summed from layer 0) subject to sum_i b_i <= budget * L,
 * exactly (a multiple-choice knapsack over integer bit totals by dynamic
 * programming).  Ties: fewer total bits, then the lexicographically smallest
 * widths (layer 0 first).  cost [L][nb], bits [nb] in [1, 64], nb <= 16.
 * *objective (may be NULL) receives the minimum.  SA_ERR_SHAPE when nothing
 * fits the budget. */
SA_API int sa_allocate_bits(const double *cost, const int *bits, int L, int nb, double budget,
                            int *out, double *objective);

/* Measurement aid, not part of the layer (no operation of the paper): reads
 * every byte of `buf` once -- each thread one 16-byte word, 256 threads per
 * workgroup, so every wave request is 1 KiB of contiguous memory -- and writes at most one
 * float per wave into out[] (values unspecified).  Its time is that
 * of a plain read of `bytes` bytes, the practical floor a layer that streams as
 * many bytes is compared against.
 *   buf    (device) 16-byte aligned; bytes a multiple of 16, 16 <= bytes <= 2^40.
 *   out    (device) float [256], overwritten.
 * Asynchronous on `stream`. */
SA_API int sa_read_probe(const void *buf, size_t bytes, float *out, void *stream);

/* Human-readable text for a status code (static storage). */
SA_API const char *sa_status_string(int status);

/* Library version string, e.g. "0.1.0 gfx950". */
SA_API const char *sa_version(void);

#ifdef __cplusplus
}
#endif

#endif /* SHIFTADD_H */
