/*
 * repops_ref.h -- CPU oracle for the RepOps operators of
 * "Verde: Verification via Refereed Delegation for Machine Learning Programs"
 * (arXiv 2502.19405), Section 3.
 *
 * TEST INFRASTRUCTURE ONLY.  This library is a plain, slow, scalar-C statement
 * of what each reproducible operator computes: the exact sequence of IEEE-754
 * binary32 operations.  Only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg may load it.  It shares no code, header, table or constant
 * with the GPU library; the two meet only on the seeded input buffers.
 *
 * Conventions (all functions):
 *   - host pointers, row-major storage, leading dimensions and strides in
 *     elements (not bytes);
 *   - the canonical order is passed as plain integers:
 *       k_block   B >= 0: contraction block length; 0 = one block (the paper's
 *                 matrix-multiplication listing taken literally);
 *       k_inner   0 = fused multiply-add  p = fma(a, b, p)
 *                 1 = multiply then add   p = p + RN(a*b);
 *       row_width W, a power of two in [1, 1024];
 *       row_combine 0 = strided tree, 1 = blocked left-to-right;
 *   - nthreads <= 0 uses every online CPU; threads split independent outputs or
 *     rows only, never one output's operation sequence;
 *   - every function returns 0 on success and a negative value on a bad argument.
 *
 * Parity pins and the readings of the paper that fix each order are stated
 * beside each definition in repops_ref.c.
 */
#ifndef REPOPS_REF_H
#define REPOPS_REF_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define REF_INNER_FMA 0
#define REF_INNER_MUL_ADD 1
#define REF_ROW_TREE 0
#define REF_ROW_BLOCKED 1

/* Bit mask of failed floating-point environment checks (0 = all good):
 * 1 = fmaf is not single-rounding, 2 = subnormals are flushed,
 * 4 = rounding mode is not to-nearest-even, 8 = excess precision in use. */
int repops_ref_env_check(void);

/* Number of threads a call with nthreads <= 0 uses. */
int repops_ref_default_threads(void);

/* One canonical contraction: sum over k of a[k*inc_a] * b[k*inc_b]. */
float repops_ref_dot(int64_t k_block, int k_inner, int64_t K,
                     const float *a, int64_t inc_a, const float *b, int64_t inc_b);

/* C[i][j] = dot(A[i][:], B[:][j]) (+ bias[j]).  trans_a: A is stored K x M
 * (A[i][k] at A[k*lda+i]); trans_b: B is stored N x K (B[k][j] at B[j*ldb+k]). */
int repops_ref_matmul(int64_t k_block, int k_inner, int64_t m, int64_t n, int64_t k,
                      const float *A, int64_t lda, int trans_a,
                      const float *B, int64_t ldb, int trans_b,
                      const float *bias, float *C, int64_t ldc, int nthreads);

/* Same outputs as repops_ref_matmul, but only at the npts positions
 * (rows[p], cols[p]); out[p] receives C[rows[p]][cols[p]]. */
int repops_ref_matmul_at(int64_t k_block, int k_inner, int64_t m, int64_t n, int64_t k,
                         const float *A, int64_t lda, int trans_a,
                         const float *B, int64_t ldb, int trans_b,
                         const float *bias, int64_t npts, const int64_t *rows,
                         const int64_t *cols, float *out);

/* Batched product over (b0, b1) in [0,batch0) x [0,batch1); operand origins
 * A + b0*sa0 + b1*sa1 (likewise B, C); C = alpha * dot. */
int repops_ref_bmm(int64_t k_block, int k_inner, int64_t batch0, int64_t batch1,
                   int64_t m, int64_t n, int64_t k,
                   const float *A, int64_t sa0, int64_t sa1, int64_t lda, int trans_a,
                   const float *B, int64_t sb0, int64_t sb1, int64_t ldb, int trans_b,
                   float alpha, float *C, int64_t sc0, int64_t sc1, int64_t ldc, int nthreads);

/* Sampled bmm outputs: out[p] = C at batch (b0[p], b1[p]), row rows[p], col cols[p]. */
int repops_ref_bmm_at(int64_t k_block, int k_inner, int64_t batch0, int64_t batch1,
                      int64_t m, int64_t n, int64_t k,
                      const float *A, int64_t sa0, int64_t sa1, int64_t lda, int trans_a,
                      const float *B, int64_t sb0, int64_t sb1, int64_t ldb, int trans_b,
                      float alpha, int64_t npts, const int64_t *b0, const int64_t *b1,
                      const int64_t *rows, const int64_t *cols, float *out);

/* Fixed-order sum of x[0..n) (squares = 1: sum of fma(x,x,.) terms). */
float repops_ref_rowsum(int row_width, int row_combine, int64_t n, const float *x, int squares);

/* Reproducible exp and tanh-form GELU, element by element. */
float repops_ref_exp1(float x);
float repops_ref_gelu1(float x);
int repops_ref_exp(int64_t n, const float *x, float *y, int nthreads);
int repops_ref_gelu(int64_t n, const float *x, float *y, int nthreads);

/* Row softmax; causal_period > 0 masks column j of row r when j > r % period. */
int repops_ref_softmax_rows(int row_width, int row_combine, int64_t rows, int64_t cols,
                            const float *X, int64_t ldx, float *Y, int64_t ldy,
                            int64_t causal_period, int nthreads);

/* Row LayerNorm with biased variance; gamma/beta may be NULL (the op is skipped);
 * mean_out/rstd_out may be NULL. */
int repops_ref_layernorm_rows(int row_width, int row_combine, int64_t rows, int64_t cols,
                              const float *X, int64_t ldx, const float *gamma,
                              const float *beta, float eps, float *Y, int64_t ldy,
                              float *mean_out, float *rstd_out, int nthreads);

/* ---- Llama-block operators ---- */

/* Reproducible sin and cos of one argument (both results; NaN for non-finite x). */
void repops_ref_sincos1(float x, float *sin_out, float *cos_out);
/* Elementwise; s or c may be NULL. */
int repops_ref_sincos(int64_t n, const float *x, float *s, float *c, int nthreads);

/* Rotary embedding (rotate-half pairing) of `heads` heads of head_dim values per
 * row; position of row r = (period > 0 ? r % period : r) + offset; inverse = 1
 * rotates by -angle (the backward). */
int repops_ref_rope(int64_t rows, int64_t heads, int64_t head_dim, const float *X, int64_t ldx,
                    const float *inv_freq, int64_t period, int64_t offset, int inverse,
                    float *Y, int64_t ldy, int nthreads);

/* RMSNorm rows; gamma may be NULL; rstd_out may be NULL. */
int repops_ref_rmsnorm_rows(int row_width, int row_combine, int64_t rows, int64_t cols,
                            const float *X, int64_t ldx, const float *gamma, float eps,
                            float *Y, int64_t ldy, float *rstd_out, int nthreads);
/* RMSNorm backward from the forward's rstd; dX / dgamma may be NULL. */
int repops_ref_rmsnorm_backward_rows(int row_width, int row_combine, int64_t k_block,
                                     int64_t rows, int64_t cols, const float *X, int64_t ldx,
                                     const float *dY, int64_t lddy, const float *rstd,
                                     const float *gamma, float *dX, int64_t lddx, float *dgamma,
                                     int nthreads);

/* SiLU, the SiLU-gated unit silu(g) * u, and its backward. */
float repops_ref_silu1(float x);
float repops_ref_silu_grad1(float x);
int repops_ref_silu(int64_t n, const float *x, float *y, int nthreads);
int repops_ref_swiglu(int64_t n, const float *g, const float *u, float *y, int nthreads);
int repops_ref_swiglu_backward(int64_t n, const float *g, const float *u, const float *dy,
                               float *dg, float *du, int nthreads);

/* erf and the erf-form GELU x * Phi(x) with its derivative (elementwise). */
float repops_ref_erf1(float x);
float repops_ref_gelu_erf1(float x);
float repops_ref_gelu_erf_grad1(float x);
int repops_ref_erf(int64_t n, const float *x, float *y, int nthreads);
int repops_ref_gelu_erf(int64_t n, const float *x, float *y, int nthreads);
int repops_ref_gelu_erf_backward(int64_t n, const float *x, const float *dy, float *dx,
                                 int nthreads);

/* ---- tensor commitments ---- */

/* SHA-256 (FIPS 180-4) of len bytes. */
void repops_ref_sha256(const void *msg, uint64_t len, uint8_t out[32]);
/* RFC 6962 Merkle Tree Hash over the chunk_bytes-sized chunks of data (last
 * chunk shorter); nbytes = 0 gives SHA-256 of the empty string. */
int repops_ref_commit(const void *data, uint64_t nbytes, uint64_t chunk_bytes, uint8_t out[32]);

/* ---- training-step operators ---- */

/* dX = Y * (dY - rowsum(Y * dY)) per row; masked columns (causal_period > 0:
 * j > r % period) are skipped in the sum and get dX = +0. */
int repops_ref_softmax_backward_rows(int row_width, int row_combine, int64_t rows, int64_t cols,
                                     const float *Y, int64_t ldy, const float *dY, int64_t lddy,
                                     float *dX, int64_t lddx, int64_t causal_period, int nthreads);

/* LayerNorm backward from the forward's mean / rstd; gamma may be NULL.  dX,
 * dgamma, dbeta may each be NULL (not computed).  dgamma/dbeta reduce over rows
 * with the contraction rule and block length k_block. */
int repops_ref_layernorm_backward_rows(int row_width, int row_combine, int64_t k_block,
                                       int64_t rows, int64_t cols,
                                       const float *X, int64_t ldx, const float *dY, int64_t lddy,
                                       const float *mean, const float *rstd, const float *gamma,
                                       float *dX, int64_t lddx, float *dgamma, float *dbeta,
                                       int nthreads);

/* Column sums over rows with the contraction rule (the bias gradient). */
int repops_ref_colsum_rows(int64_t k_block, int64_t rows, int64_t cols, const float *X,
                           int64_t ldx, float *out, int nthreads);

/* d gelu(x) / dx and dX = dY * gelu'(X). */
float repops_ref_gelu_grad1(float x);
int repops_ref_gelu_backward(int64_t n, const float *x, const float *dy, float *dx, int nthreads);

/* One Adam (decoupled = 0) or AdamW (decoupled = 1) step, in place; step >= 1. */
int repops_ref_adam_step(int64_t n, float *param, const float *grad, float *exp_avg,
                         float *exp_avg_sq, float lr, float beta1, float beta2, float eps,
                         float weight_decay, int64_t step, int decoupled, int nthreads);
/* out6 = {1 - b1, 1 - b2, lr / (1 - b1^t), sqrt(1 - b2^t), 1 - lr*wd, b1^t}, each
 * computed in binary64 and rounded once to binary32. */
int repops_ref_adam_scalars(float lr, float beta1, float beta2, float weight_decay, int64_t step,
                            float *out6);

#ifdef __cplusplus
}
#endif
#endif
