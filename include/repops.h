/*
 * repops.h -- C ABI of librepops, bitwise-reproducible fp32 operators for
 * AMD Instinct MI355X (gfx950).
 *
 * The operators are those of RepOps in "Verde: Verification via Refereed
 * Delegation for Machine Learning Programs" (arXiv 2502.19405), Section 3:
 * every output is produced by one fixed sequence of IEEE-754 binary32
 * operations that depends only on the problem sizes and on the canonical-order
 * descriptor below -- never on the launch configuration, tile sizes, strides,
 * transposition, the GPU model or the run.  Two calls with the same order
 * descriptor and the same logical inputs return the same bits.
 *
 * General conventions
 *   - All tensor pointers are DEVICE pointers owned by the caller; the library
 *     allocates no device memory and keeps no mutable global state.
 *   - Storage is row-major; leading dimensions and batch strides count
 *     elements (float), not bytes.
 *   - Calls are asynchronous on `hip_stream` (a hipStream_t; NULL means the
 *     null stream).  Device faults surface at the caller's next
 *     synchronisation.  Calls are thread-safe.
 *   - On any error nothing is enqueued and a nonzero repops_status_t is
 *     returned.  Zero-sized problems (m, n, rows, batch or element count 0)
 *     succeed without launching anything.
 *   - `launch` selects speed only and may be NULL (automatic choice).  A
 *     launch configuration never changes an output bit.
 *   - Inputs are expected finite; infinities and NaNs propagate
 *     deterministically, but only "NaN in, NaN out" is promised for them.
 */
#ifndef REPOPS_H
#define REPOPS_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define REPOPS_ABI_VERSION 2u

typedef int32_t repops_status_t;
enum {
    REPOPS_OK = 0,
    REPOPS_ERR_NULL = 1,   /* a required pointer is NULL */
    REPOPS_ERR_SHAPE = 2,  /* negative size, or a size the operator cannot take */
    REPOPS_ERR_STRIDE = 3, /* leading dimension smaller than the row it holds */
    REPOPS_ERR_ALIAS = 4,  /* output overlaps an input where that is not allowed */
    REPOPS_ERR_ORDER = 5,  /* unknown or unsupported order descriptor; never silently replaced */
    REPOPS_ERR_LAUNCH = 6, /* launch configuration invalid for this call */
    REPOPS_ERR_HIP = 7,    /* the HIP runtime rejected the kernel launch */
    REPOPS_ERR_VALUE = 8,  /* a scalar argument outside its domain */
    REPOPS_ERR_WORKSPACE = 9, /* workspace NULL or smaller than the size the query returns */
    REPOPS_ERR_SCRATCH = 10   /* the problem needs more than the fixed scratch of a
                                 no-allocation entry point (REPOPS_NOALLOC_SCRATCH_BYTES) */
};

/*
 * Canonical-order descriptor: selects the BITS.
 *
 * Contraction (matmul, bmm) -- Section 3.2, matrix-multiplication listing: the
 * output indices run in any order, the contraction index k in one fixed order.
 * For an output with terms (a_k, b_k), k = 0..K-1:
 *     for each block beta = 0, 1, ... of k_block consecutive k (last one short):
 *         P = +0;  for k in the block, ascending:  P = fma(a_k, b_k, P)
 *                                         (k_inner MUL_ADD: P = P + RN(a_k*b_k))
 *     acc = +0;  for beta ascending:  acc = acc + P_beta
 * k_block = 0 is a single block: the listing itself.
 *
 * Row reductions (softmax, LayerNorm) -- not fixed by the paper; the order is a
 * function of the row length n and row_width W only:
 *     STRIDED_TREE: q[l] = +0 for l < W; x_j is added to q[j mod W] in
 *         ascending j; then for s = W/2, ..., 1: q[l] = q[l] + q[l+s] (l < s);
 *         the sum is q[0].
 *     BLOCKED_LTR: the contraction rule with additions, blocks of W elements.
 *     For LayerNorm's sum of squares the term update is q = fma(d, d, q).
 *
 * version 1 also freezes the operation sequences of exp, GELU, softmax and
 * LayerNorm documented at each function below.
 */
typedef struct repops_order {
    uint32_t version;     /* must be 1 */
    uint32_t k_block;     /* contraction block length; 0 = unblocked; default 64 */
    uint32_t k_inner;     /* REPOPS_K_FMA (default) or REPOPS_K_MUL_ADD */
    uint32_t k_combine;   /* REPOPS_COMBINE_LTR (only value in version 1) */
    uint32_t row_width;   /* W: power of two in [1, 1024]; default 64 */
    uint32_t row_combine; /* REPOPS_ROW_STRIDED_TREE (default) or REPOPS_ROW_BLOCKED_LTR */
    uint32_t reserved[2]; /* must be 0 */
} repops_order_t;

enum { REPOPS_K_FMA = 0, REPOPS_K_MUL_ADD = 1 };
enum { REPOPS_COMBINE_LTR = 0 };
enum { REPOPS_ROW_STRIDED_TREE = 0, REPOPS_ROW_BLOCKED_LTR = 1 };

/*
 * Launch descriptor: selects the SPEED only.
 *   kind AUTO (0): the library chooses.
 *   matmul / bmm:
 *     GEMM_SIMPLE (1): one output per thread, operands read from global memory.
 *     GEMM_TILED  (2): LDS-staged tiles, per-lane FMA chains; p[0] = index into
 *         the table reported by repops_gemm_config_name().  Needs k_block = 0
 *         or k_block a multiple of the configuration's k tile.
 *     GEMM_MFMA   (3): matrix-core tiles whose single-term updates equal the
 *         FMA chain; p[0] = index into the same table.  Needs k_inner FMA.
 *   softmax_rows / layernorm_rows (and rmsnorm_rows):
 *     ROWS_GENERIC (1): any supported order descriptor.
 *     ROWS_WAVE    (2): STRIDED_TREE with W = 64; rows held in registers.
 *         p[0] = rows per block, one of 1, 2, 4, 8; p[1] = waves per row:
 *         0 or 1 for one 64-lane wave per row (rows up to 4096 columns), or
 *         2, 4, 8 for one row per block split over that many waves (then
 *         p[0] = 1, and a row takes at most 2048 * p[1] columns).  Each lane
 *         still folds its terms in column order, so the bits do not depend on
 *         p[].  AUTO takes one wave per row up to 1024 columns and splits
 *         wider rows (at most 16 values per lane where 8 waves allow it).
 *   gelu / exp:
 *     ELEMENTWISE (1): p[0] = threads per block (multiple of 64, <= 1024),
 *         p[1] = maximum number of blocks (0 = as many as needed).
 * Unused p[] entries must be 0.
 */
typedef struct repops_launch {
    uint32_t kind;
    uint32_t p[7];
} repops_launch_t;

enum {
    REPOPS_LAUNCH_AUTO = 0,
    REPOPS_LAUNCH_GEMM_SIMPLE = 1,
    REPOPS_LAUNCH_GEMM_TILED = 2,
    REPOPS_LAUNCH_GEMM_MFMA = 3,
    REPOPS_LAUNCH_ROWS_GENERIC = 1,
    REPOPS_LAUNCH_ROWS_WAVE = 2,
    REPOPS_LAUNCH_ELEMENTWISE = 1
};

/* Fills *order with version 1, k_block 64, FMA, left-to-right, W 64, strided tree. */
void repops_order_default(repops_order_t *order);
const char *repops_status_str(repops_status_t status);
uint32_t repops_abi_version(void);

/* Number of entries in the tiled / matrix-core configuration tables, and a
 * static description of entry `index` ("BMxBNxBK/TMxTN", NULL if out of range). */
int32_t repops_gemm_config_count(uint32_t kind);
const char *repops_gemm_config_name(uint32_t kind, uint32_t index);

/*
 * repops_matmul -- C = A.B (+ bias), Section 3.2 (matrix multiplication).
 *   m, n, k   logical sizes: A is m x k, B is k x n, C is m x n; k = 0 gives
 *             C = +0 (or bias).
 *   A, lda    trans_a = 0: A[i][kk] at A[i*lda + kk] (lda >= k);
 *             trans_a = 1: A stored k x m, A[i][kk] at A[kk*lda + i] (lda >= m).
 *   B, ldb    trans_b = 0: B[kk][j] at B[kk*ldb + j] (ldb >= n);
 *             trans_b = 1: B stored n x k, B[kk][j] at B[j*ldb + kk] (ldb >= k).
 *   bias      NULL or [n]: C[i][j] = acc + bias[j], one rounded addition after
 *             the contraction.
 *   C, ldc    output, ldc >= n; must not overlap A, B or bias (REPOPS_ERR_ALIAS).
 */
repops_status_t repops_matmul(const repops_order_t *order, int64_t m, int64_t n, int64_t k,
                              const float *A, int64_t lda, int32_t trans_a,
                              const float *B, int64_t ldb, int32_t trans_b,
                              const float *bias, float *C, int64_t ldc,
                              const repops_launch_t *launch, void *hip_stream);

/*
 * repops_matmul_gelu -- H = A.B (+ bias) and G = GELU(H), the feed-forward
 * layer's first product and activation (Section 3.2's matrix multiplication,
 * then Section 3.1's reproducible elementwise GELU, tanh form), in one pass:
 * the threads that write an output of H also write its GELU into G.  H takes
 * exactly the bits repops_matmul gives for the same arguments, and G exactly
 * the bits repops_gelu gives for that H, under every launch descriptor.
 *   Arguments as for repops_matmul, with H, ldh in the place of C, ldc.
 *   G, ldg    [m x n] output, ldg >= n; must not overlap H, A, B or bias
 *             (REPOPS_ERR_ALIAS); NULL is REPOPS_ERR_NULL unless m or n is 0.
 */
repops_status_t repops_matmul_gelu(const repops_order_t *order, int64_t m, int64_t n, int64_t k,
                                   const float *A, int64_t lda, int32_t trans_a,
                                   const float *B, int64_t ldb, int32_t trans_b,
                                   const float *bias, float *H, int64_t ldh, float *G,
                                   int64_t ldg, const repops_launch_t *launch, void *hip_stream);

/*
 * repops_matmul_gelu_backward -- C = GELU'(X) * (A.B), the input gradient of
 * the feed-forward layer's GELU taken straight from the product that makes its
 * output gradient (Section 3.2's matrix multiplication, then the reproducible
 * GELU backward of Section 3.1's elementwise functions, as the training graph
 * of Section 2.2 chains them): C[i][j] = RN(P[i][j] * gelu'(X[i][j])) with
 * P the product repops_matmul gives and gelu' the tanh-form derivative, so C
 * has exactly the bits of repops_matmul followed by repops_gelu_backward(X, P)
 * under every launch descriptor.
 *   Arguments as for repops_matmul without bias.
 *   X, ldx    [m x n] forward input of the GELU, ldx >= n; C must not overlap
 *             it (REPOPS_ERR_ALIAS); NULL is REPOPS_ERR_NULL unless m or n is 0.
 */
repops_status_t repops_matmul_gelu_backward(const repops_order_t *order, int64_t m, int64_t n,
                                            int64_t k, const float *A, int64_t lda,
                                            int32_t trans_a, const float *B, int64_t ldb,
                                            int32_t trans_b, const float *X, int64_t ldx,
                                            float *C, int64_t ldc, const repops_launch_t *launch,
                                            void *hip_stream);

/*
 * repops_matmul_grouped -- several independent products C_p = A_p.B_p (+ bias_p)
 * in one call, Section 3.2 (matrix multiplication) as for repops_matmul: each
 * product's outputs take exactly the bits repops_matmul gives for the same
 * arguments (repops_matmul_gelu_backward's where gelu_in is set).  The products run concurrently (one launch whose workgroups cover
 * every product's output tiles, the products with the longest contraction
 * first), so that products with few output tiles share the compute units:
 * the weight and input gradients of a linear layer are the intended use.
 *   count   0 .. REPOPS_MAX_GROUP products; descs: host array of count entries
 *           (read during the call only; may be NULL when count = 0).
 *   each desc's fields as repops_matmul's arguments; gelu_in, ld_gelu_in: NULL
 *           for a plain product, else the GELU input X of
 *           repops_matmul_gelu_backward (then bias must be NULL).
 *   No C_p may overlap its own operands or any other product's A, B, bias,
 *   gelu_in or C (REPOPS_ERR_ALIAS).
 *   launch  NULL or AUTO.  When every nonempty product has K > 0, K and k_block
 *           multiples of 16, 16-byte aligned rows and the fused order, one
 *           launch of the 128 x 128 matrix-core tile runs them all; otherwise the
 *           products run one after another with repops_matmul's automatic
 *           launch (the same bits either way).
 */
typedef struct repops_gemm_desc {
    int64_t m, n, k;
    const float *A; int64_t lda; int32_t trans_a;
    const float *B; int64_t ldb; int32_t trans_b;
    const float *bias;
    float *C; int64_t ldc;
    const float *gelu_in; int64_t ld_gelu_in;
} repops_gemm_desc_t;
#define REPOPS_MAX_GROUP 8
repops_status_t repops_matmul_grouped(const repops_order_t *order, int32_t count,
                                      const repops_gemm_desc_t *descs,
                                      const repops_launch_t *launch, void *hip_stream);

/*
 * repops_bmm -- batched product over (i0, i1) in [0,batch0) x [0,batch1), the
 * batched key-query and probability-value products of attention that Section
 * 2.2 decomposes into independent matrix products.  Batch element (i0, i1)
 * reads A + i0*sa0 + i1*sa1 and B + i0*sb0 + i1*sb1 with the matmul layout
 * rules, and writes C + i0*sc0 + i1*sc1:  C[i][j] = acc * alpha (one rounded
 * multiplication).  Strides may be 0 for A and B.  C may not overlap A or B
 * (REPOPS_ERR_ALIAS), and no two of its elements may share an address
 * (REPOPS_ERR_STRIDE), checked by a sufficient condition: taking the
 * dimensions batch0, batch1, m (stride ldc) and n (stride 1) that have more
 * than one element in increasing order of |stride|, each stride must exceed
 * the span of the ones before it -- every permutation of a dense array, such
 * as heads interleaved within the rows of a [tokens x heads*dim] output,
 * passes.
 */
repops_status_t repops_bmm(const repops_order_t *order, int64_t batch0, int64_t batch1,
                           int64_t m, int64_t n, int64_t k,
                           const float *A, int64_t sa0, int64_t sa1, int64_t lda, int32_t trans_a,
                           const float *B, int64_t sb0, int64_t sb1, int64_t ldb, int32_t trans_b,
                           float alpha, float *C, int64_t sc0, int64_t sc1, int64_t ldc,
                           const repops_launch_t *launch, void *hip_stream);

/*
 * repops_bmm_causal -- repops_bmm for the causal attention products (Section
 * 2.2's key-query and value products of a causal self-attention), with the
 * same arguments plus a mask over each batch element's rows i, columns j and
 * contraction index kk:
 *   REPOPS_CAUSAL_OUTPUT  only the outputs with j <= i are wanted: they get
 *       exactly repops_bmm's bits; outputs with j > i are unspecified (the
 *       matrix-core kernels skip output tiles that lie wholly above the
 *       diagonal and leave them unwritten).  For scores S = alpha Q K^T that a
 *       causal softmax (causal_period = m) reads only at j <= i.
 *   REPOPS_CAUSAL_A  the caller guarantees A[i][kk] is zero (either sign) for
 *       kk > i and B is finite: every output gets exactly repops_bmm's bits.
 *       The matrix-core kernels skip the k blocks of a row tile that hold only
 *       such terms -- their block partials would be +0, which leaves the
 *       accumulator unchanged.  For P V with P a causal softmax's output.
 *   Any other mask value: REPOPS_ERR_VALUE.  Everything else as repops_bmm.
 */
#define REPOPS_CAUSAL_OUTPUT 1
#define REPOPS_CAUSAL_A 2
repops_status_t repops_bmm_causal(const repops_order_t *order, int64_t batch0, int64_t batch1,
                                  int64_t m, int64_t n, int64_t k, const float *A, int64_t sa0,
                                  int64_t sa1, int64_t lda, int32_t trans_a, const float *B,
                                  int64_t sb0, int64_t sb1, int64_t ldb, int32_t trans_b,
                                  float alpha, float *C, int64_t sc0, int64_t sc1, int64_t ldc,
                                  int32_t mask, const repops_launch_t *launch, void *hip_stream);

/*
 * repops_softmax_rows -- row softmax (an operator of the DistilBERT and Llama
 * programs of Section 4.2; order fixed by the descriptor):
 *     m = max over unmasked x_j;  e_j = exp_rep(x_j - m) (masked: +0);
 *     s = row sum of e in the descriptor's row order;  r = 1 / s;  y_j = e_j * r.
 *   X, ldx / Y, ldy   rows x cols, ldx >= cols, ldy >= cols.  Y == X with
 *                     ldy == ldx (in place) is allowed; other overlap is not.
 *   causal_period     0: no mask; p > 0: row i masks columns j > i mod p.
 */
repops_status_t repops_softmax_rows(const repops_order_t *order, int64_t rows, int64_t cols,
                                    const float *X, int64_t ldx, float *Y, int64_t ldy,
                                    int64_t causal_period, const repops_launch_t *launch,
                                    void *hip_stream);

/*
 * repops_layernorm_rows -- row LayerNorm (named among DistilBERT's operators in
 * Section 4.2), biased variance:
 *     mean = rowsum(x) / n;  d_j = x_j - mean;  var = rowsum(fma(d,d,.)) / n;
 *     rstd = 1 / sqrt(var + eps);  t_j = d_j * rstd;  y_j = fma(t_j, gamma_j, beta_j).
 *   sqrt and the division are correctly rounded.  gamma / beta may be NULL:
 *   the operation is skipped (y = t, t + beta or t * gamma), which differs from
 *   passing ones / zeros in the sign of zero.  mean_out / rstd_out: NULL or
 *   [rows]; neither may overlap X, Y, gamma, beta or the other
 *   (REPOPS_ERR_ALIAS).  cols must be >= 1.  In-place as for softmax.
 */
repops_status_t repops_layernorm_rows(const repops_order_t *order, int64_t rows, int64_t cols,
                                      const float *X, int64_t ldx, const float *gamma,
                                      const float *beta, float eps, float *Y, int64_t ldy,
                                      float *mean_out, float *rstd_out,
                                      const repops_launch_t *launch, void *hip_stream);

/*
 * repops_gelu -- tanh-form GELU over n contiguous elements (Section 4.2 names
 * GeLU among DistilBERT's operators), using 0.5(1 + tanh z) = 1/(1 + exp(-2z)):
 *     u = (x*x)*x;  z = fma(0.044715f, u, x) * 0.7978846f;  w = -2*z;
 *     y = x / (1 + exp_rep(w)).
 *   Constants are the binary32 values nearest 0.044715 and sqrt(2/pi).
 *   Y == X (in place) is allowed.
 */
repops_status_t repops_gelu(const repops_order_t *order, int64_t n, const float *X, float *Y,
                            const repops_launch_t *launch, void *hip_stream);

/*
 * repops_exp -- the reproducible exp used inside softmax and GELU (Section 3.1
 * lists exp among the functions RepOps rebuilds with a controlled order),
 * exported for testing.  Cody-Waite reduction and a degree-7 Taylor polynomial:
 *     n = rint(x * log2e) (ties to even); n > 128: +inf; n < -151: +0;
 *     r = fma(n, -ln2_hi, x); r = fma(n, -ln2_lo, r);
 *     p = Horner over 1/i!, i = 7..0, with fma;
 *     y = (p * 2^floor(n/2)) * 2^(n - floor(n/2)).
 *   Y == X (in place) is allowed.
 */
repops_status_t repops_exp(const repops_order_t *order, int64_t n, const float *X, float *Y,
                           const repops_launch_t *launch, void *hip_stream);

/*
 * repops_copy -- Y = X over n contiguous elements through the elementwise
 *   kernel with no arithmetic: the streaming rate that kernel reaches, the
 *   ceiling against which the bandwidth-bound operators are measured (not an
 *   operator of the method).  Same checks, launch options and errors as
 *   repops_exp; Y == X is allowed.
 */
repops_status_t repops_copy(const repops_order_t *order, int64_t n, const float *X, float *Y,
                            const repops_launch_t *launch, void *hip_stream);

/* ------------------------------------------------------------------------
 * Training-step operators.  The training runs of Section 4.2 (Adam optimizer)
 * execute the extended graph of Section 2.2: every forward node, its backward
 * node and the optimizer update.  The paper fixes no order for these
 * operators; version 1 fixes the operation sequences documented below.
 * ------------------------------------------------------------------------ */

/*
 * repops_softmax_backward_rows -- gradient of repops_softmax_rows:
 *     s = row sum of fma(y_j, dy_j, .) over the unmasked columns, in the
 *         descriptor's row order (masked columns contribute no operation);
 *     dx_j = y_j * (dy_j - s);  masked columns: dx_j = +0.
 *   Y, ldy    the forward output (rows x cols); dY, lddy the incoming gradient.
 *   dX, lddx  output; may coincide exactly (same base and leading dimension)
 *             with Y or with dY; other overlap is REPOPS_ERR_ALIAS.
 *   causal_period  as for the forward.  Launch kinds as for softmax_rows.
 */
repops_status_t repops_softmax_backward_rows(const repops_order_t *order, int64_t rows,
                                             int64_t cols, const float *Y, int64_t ldy,
                                             const float *dY, int64_t lddy, float *dX,
                                             int64_t lddx, int64_t causal_period,
                                             const repops_launch_t *launch, void *hip_stream);

/*
 * repops_layernorm_backward_workspace -- bytes of device workspace that
 * repops_layernorm_backward_rows needs for the parameter gradients at this
 * size and order: 2 * ceil(rows / k_block) * cols floats when that is more
 * than one block of rows, else 0.
 */
repops_status_t repops_layernorm_backward_workspace(const repops_order_t *order, int64_t rows,
                                                    int64_t cols, uint64_t *bytes);

/*
 * repops_layernorm_backward_rows -- gradients of repops_layernorm_rows, from
 * the forward's mean and rstd (its mean_out / rstd_out):
 *   input gradient, per row, with the descriptor's row order:
 *     t_j = (x_j - mean) * rstd;  g_j = dy_j * gamma_j (dy_j if gamma is NULL);
 *     a = rowsum(g) / n;  b = rowsum of fma(g_j, t_j, .) / n;
 *     dx_j = rstd * ((g_j - a) - t_j * b).
 *   parameter gradients, per column j: the row index is a contraction index
 *   and takes the matmul rule with block length k_block:
 *     dgamma_j: P = fma(dy_ij, t_ij, P) over the rows of a block;
 *     dbeta_j:  P = P + dy_ij;  block partials added left to right.
 *     rows = 0 gives +0.
 *   X, ldx / dY, lddy   forward input and incoming gradient, rows x cols.
 *   mean, rstd          [rows]; gamma NULL or [cols].
 *   dX, lddx            NULL or output; may coincide exactly with X or dY.
 *   dgamma, dbeta       NULL or [cols] outputs.
 *   workspace           device memory of at least the size that
 *                       repops_layernorm_backward_workspace returns (may be NULL
 *                       when that is 0 or when dgamma and dbeta are NULL);
 *                       owned by the caller, contents on return unspecified.
 *                       REPOPS_ERR_WORKSPACE if missing or too small.
 *   No output may overlap another output, the workspace or an input (other
 *   than dX as stated).  cols must be >= 1 when rows > 0, and <= 2^24.
 *   Launch kinds (for the input gradient) as for layernorm_rows.
 */
repops_status_t repops_layernorm_backward_rows(
    const repops_order_t *order, int64_t rows, int64_t cols, const float *X, int64_t ldx,
    const float *dY, int64_t lddy, const float *mean, const float *rstd, const float *gamma,
    float *dX, int64_t lddx, float *dgamma, float *dbeta, void *workspace,
    uint64_t workspace_bytes, const repops_launch_t *launch, void *hip_stream);

/*
 * repops_layernorm_backward_rows_noalloc -- repops_layernorm_backward_rows
 * for callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the same
 * operation, arguments, launch kinds and bits, with no workspace argument.
 * The parameter gradients' block partials go to a fixed scratch array of
 * REPOPS_NOALLOC_SCRATCH_BYTES in device memory, which every device the
 * library runs on holds until the process ends; the call allocates and frees
 * nothing.  Its device address is looked up (hipGetSymbolAddress) on the
 * first call per device, with the caller's current device, which must be the
 * device of hip_stream.
 *   Limit: 2 * ceil(rows / k_block) * cols * 4 bytes (the workspace query's
 *   size) at most REPOPS_NOALLOC_SCRATCH_BYTES, e.g. 65536 x 768 or
 *   16384 x 4096 at k_block 64; beyond it REPOPS_ERR_SCRATCH, with nothing
 *   enqueued.
 *   Calls on one device share the scratch array: calls that overlap in time
 *   on that device (on different streams, or from different host threads)
 *   race and may give wrong parameter gradients; serialise them.  Every
 *   partial a call reads is written earlier in the same call, so the contents
 *   left by an earlier call never matter.
 */
#define REPOPS_NOALLOC_SCRATCH_BYTES (8ull << 20)
repops_status_t repops_layernorm_backward_rows_noalloc(
    const repops_order_t *order, int64_t rows, int64_t cols, const float *X, int64_t ldx,
    const float *dY, int64_t lddy, const float *mean, const float *rstd, const float *gamma,
    float *dX, int64_t lddx, float *dgamma, float *dbeta, const repops_launch_t *launch,
    void *hip_stream);

/*
 * repops_colsum_rows -- column sums over rows, the bias gradient of a linear
 * layer (db = ones^T dY).  The row index is a contraction index, so the
 * matmul rule applies with block length k_block: per column, chains
 * P = P + x_ij over blocks of rows from +0, block partials left to right
 * (bit-identical to repops_matmul of a ones row with X, since
 * fma(1, x, P) = P + x).  rows = 0 gives +0.
 *   X, ldx     rows x cols input; out [cols], must not overlap X.
 *   workspace  as for repops_layernorm_backward_rows (its workspace query
 *              gives the size for the same rows, cols and order).
 *   launch     NULL or AUTO.
 */
repops_status_t repops_colsum_rows(const repops_order_t *order, int64_t rows, int64_t cols,
                                   const float *X, int64_t ldx, float *out, void *workspace,
                                   uint64_t workspace_bytes, const repops_launch_t *launch,
                                   void *hip_stream);

/*
 * repops_gelu_backward -- dx = dy * gelu'(x) over n contiguous elements, the
 * derivative of repops_gelu.  With s = 1 / (1 + exp_rep(w)) from the forward's
 * sequence (y = x * s), one fixed sequence:
 *     u = x*x;  z = fma(0.044715f, u*x, x) * 0.7978846f;  s = 1 / (1 + exp_rep(-2z));
 *     om = 1 - s;  v = fma(0.134145f, u, 1);  t2 = (x*s) * om;  t3 = 1.5957692f * v;
 *     dx = dy * fma(t2, t3, s).
 *   Constants are the binary32 values nearest 0.044715, sqrt(2/pi), 0.134145
 *   and 2 sqrt(2/pi).  dX may coincide exactly with X or dY.
 */
repops_status_t repops_gelu_backward(const repops_order_t *order, int64_t n, const float *X,
                                     const float *dY, float *dX, const repops_launch_t *launch,
                                     void *hip_stream);

/*
 * repops_adam_step -- one Adam (decoupled = 0) or AdamW (decoupled = 1) update
 * of n contiguous parameters in place (Section 4.2 trains with Adam).
 *   step scalars, computed on the host in binary64 from the binary32
 *   arguments and rounded once to binary32:
 *     c1 = 1 - b1;  c2 = 1 - b2;  st = lr / (1 - b1^t);  sb = sqrt(1 - b2^t);
 *     dec = 1 - lr * wd;  b^t by binary exponentiation (square-and-multiply
 *     from the lowest bit of t).
 *   per element, binary32:
 *     wd != 0: decoupled: p = p * dec;  coupled: g = fma(wd, p, g);
 *     m = fma(b1, m, c1 * g);  v = fma(b2, v, c2 * (g * g));
 *     p = p - st * (m / (sqrt(v) / sb + eps)).
 *   param, exp_avg, exp_avg_sq   [n], updated in place; grad [n] read only;
 *                                the four must not overlap.
 *   step >= 1; 0 <= beta1, beta2 < 1; lr, eps, weight_decay finite; otherwise
 *   REPOPS_ERR_VALUE.  Launch kinds as for gelu.
 */
repops_status_t repops_adam_step(const repops_order_t *order, int64_t n, float *param,
                                 const float *grad, float *exp_avg, float *exp_avg_sq, float lr,
                                 float beta1, float beta2, float eps, float weight_decay,
                                 int64_t step, int32_t decoupled, const repops_launch_t *launch,
                                 void *hip_stream);

/* ------------------------------------------------------------------------
 * Llama-block operators (the Llama programs of Section 4.2): sin/cos for the
 * rotary embedding, RMSNorm and the SiLU-gated unit.  Section 3.1 lists the
 * math functions RepOps rebuilds with a controlled order; version 1 fixes the
 * sequences below.
 * ------------------------------------------------------------------------ */

/*
 * repops_sincos -- reproducible sin and cos of n contiguous elements (used
 * inside repops_rope; exported for testing).  Cody-Waite reduction by pi/2:
 *     n = rint(x * RN(2/pi));  r = x if n = 0, else three fused steps
 *     r = fma(n, -P_i, r) with P1 + P2 + P3 = pi/2 (each the binary32 value
 *     nearest the remainder);  u = r*r;
 *     s = fma(r*u, S(u), r), S by Horner over RN(-1/3!), RN(1/5!), RN(-1/7!), RN(1/9!);
 *     c = fma(u, C(u), 1), C by Horner over -1/2, RN(1/4!), ..., RN(-1/10!);
 *     quadrant n mod 4 selects (s, c), (c, -s), (-s, -c), (-c, s).
 *   x = +-0 gives (x, 1); non-finite x gives NaN.  Accurate to 2 ulp for
 *   |x| <= 2^17 (reproducible, less accurate, beyond).  S or C may be NULL (not
 *   both); S may equal X when C is NULL, C may equal X.
 */
repops_status_t repops_sincos(const repops_order_t *order, int64_t n, const float *X, float *S,
                              float *C, const repops_launch_t *launch, void *hip_stream);

/*
 * repops_rope -- rotary position embedding with rotate-half pairing.  Row r of
 * X holds `heads` heads of head_dim (even) values at X + r*ldx; its position is
 * p = (position_period > 0 ? r % position_period : r) + position_offset
 * (p < 2^24).  For i < head_dim/2:
 *     angle = RN(p * inv_freq[i]);  s, c = repops_sincos(angle);
 *     x1 = x[h*head_dim + i], x2 = x[h*head_dim + i + head_dim/2];
 *     inverse = 0: y1 = RN(x1 c) - RN(x2 s), y2 = RN(x2 c) + RN(x1 s);
 *     inverse = 1 (the backward): y1 = RN(x1 c) + RN(x2 s), y2 = RN(x2 c) - RN(x1 s).
 *   inv_freq   [head_dim/2], the model's frequency table (an input like a weight).
 *   Y, ldy     output rows of heads*head_dim; may coincide exactly with X.
 *   launch     AUTO or ROWS_WAVE (p[0] = rows per block: 1, 2, 4, 8).
 */
repops_status_t repops_rope(const repops_order_t *order, int64_t rows, int64_t heads,
                            int64_t head_dim, const float *X, int64_t ldx, const float *inv_freq,
                            int64_t position_period, int64_t position_offset, int32_t inverse,
                            float *Y, int64_t ldy, const repops_launch_t *launch,
                            void *hip_stream);

/*
 * repops_rmsnorm_rows -- RMSNorm over rows:
 *     ms = rowsum(fma(x_j, x_j, .)) / n in the descriptor's row order;
 *     rstd = 1 / sqrt(ms + eps);  y_j = RN(x_j rstd) * gamma_j (no product if
 *     gamma is NULL).  rstd_out NULL or [rows].  In place as for LayerNorm;
 *     cols >= 1 when rows > 0.  Launch kinds as for layernorm_rows.
 */
repops_status_t repops_rmsnorm_rows(const repops_order_t *order, int64_t rows, int64_t cols,
                                    const float *X, int64_t ldx, const float *gamma, float eps,
                                    float *Y, int64_t ldy, float *rstd_out,
                                    const repops_launch_t *launch, void *hip_stream);

/* Workspace bytes of repops_rmsnorm_backward_rows (same rule as LayerNorm's). */
repops_status_t repops_rmsnorm_backward_workspace(const repops_order_t *order, int64_t rows,
                                                  int64_t cols, uint64_t *bytes);

/*
 * repops_rmsnorm_backward_rows -- gradients of repops_rmsnorm_rows from its rstd:
 *     t_j = x_j rstd;  g_j = dy_j gamma_j (dy_j);  b = rowsum(fma(g_j, t_j, .)) / n;
 *     dx_j = rstd * (g_j - t_j b);
 *     dgamma_j: per column, the contraction rule over rows with block k_block
 *     (P = fma(dy_ij, t_ij, P), block partials left to right).
 *   Arguments, workspace, aliasing and launch as for the LayerNorm backward
 *   (no mean, no dbeta).
 */
repops_status_t repops_rmsnorm_backward_rows(
    const repops_order_t *order, int64_t rows, int64_t cols, const float *X, int64_t ldx,
    const float *dY, int64_t lddy, const float *rstd, const float *gamma, float *dX,
    int64_t lddx, float *dgamma, void *workspace, uint64_t workspace_bytes,
    const repops_launch_t *launch, void *hip_stream);

/*
 * repops_silu -- y = x / (1 + exp_rep(-x)) over n contiguous elements; Y may
 * equal X.  Launch kinds as for gelu.
 */
repops_status_t repops_silu(const repops_order_t *order, int64_t n, const float *X, float *Y,
                            const repops_launch_t *launch, void *hip_stream);

/*
 * repops_swiglu -- the SiLU-gated unit of Llama's feed-forward:
 *     y = RN(silu(g) * up).  Y may equal G or Up.
 */
repops_status_t repops_swiglu(const repops_order_t *order, int64_t n, const float *G,
                              const float *Up, float *Y, const repops_launch_t *launch,
                              void *hip_stream);

/*
 * repops_swiglu_backward -- gradients of repops_swiglu:
 *     s = 1 / (1 + exp_rep(-g));  silu'(g) = fma(g*s, 1 - s, s);
 *     dG = RN(RN(dy * up) * silu'(g));  dUp = RN(dy * silu(g)) with silu(g) as
 *     in the forward.  dG and dUp may each coincide exactly with an input and
 *     must not overlap each other.
 */
repops_status_t repops_swiglu_backward(const repops_order_t *order, int64_t n, const float *G,
                                       const float *Up, const float *dY, float *dG, float *dUp,
                                       const repops_launch_t *launch, void *hip_stream);

/* ------------------------------------------------------------------------
 * Tensor commitments.  The protocol commits to checkpoints and to the tensors
 * entering and leaving every graph node with a collision-resistant hash such
 * as SHA-256, and combines node hashes in a binary Merkle tree (Sections 2.1
 * and 2.2).  A tensor is committed as the RFC 6962 Merkle Tree Hash of its
 * bytes cut into chunks:
 *     MTH({}) = SHA-256(empty);  MTH({d}) = SHA-256(0x00 || d);
 *     MTH(D[0:n]) = SHA-256(0x01 || MTH(D[0:k]) || MTH(D[k:n])), k the largest
 *     power of two below n;
 * with SHA-256 as in FIPS 180-4.
 * ------------------------------------------------------------------------ */

/* Workspace bytes repops_commit needs for nbytes of data in chunks of
 * chunk_bytes (1 <= chunk_bytes <= 2^30): 32 per chunk plus 32 per pair. */
repops_status_t repops_commit_workspace(uint64_t nbytes, uint32_t chunk_bytes, uint64_t *bytes);

/*
 * repops_commit -- the commitment of nbytes at `data` (device; a tensor's
 * storage as it lies in memory, e.g. row-major little-endian binary32),
 * chunks of chunk_bytes (the last one shorter).  The 32-byte digest goes to
 * `digest` (device memory, SHA-256 byte order).  16-byte-aligned data with a
 * chunk size that is a multiple of 64 takes the vector path; anything else is
 * hashed byte by byte, with the same result.  workspace: device memory of at
 * least repops_commit_workspace bytes, 4-byte aligned, contents on return
 * unspecified.  digest, data and workspace must not overlap.  launch: NULL
 * or AUTO.
 */
repops_status_t repops_commit(const void *data, uint64_t nbytes, uint32_t chunk_bytes,
                              uint8_t *digest, void *workspace, uint64_t workspace_bytes,
                              const repops_launch_t *launch, void *hip_stream);

/*
 * repops_erf -- reproducible erf of n contiguous elements (used inside the
 * erf-form GELU; exported for testing).  |x| < 0.5: x * S(x*x), S by Horner
 * with fma over RN(2/sqrt(pi) (-1)^n / (n! (2n+1))), n = 0..7.  Otherwise
 * sign(x) (1 - erfc(|x|)) with erfc(z) = exp(-z^2) R(z), 0 for z >= 10.5:
 *     R on [0.5, 2.5]: degree-12 polynomial in s = z - 1.5; on [2.5, 10.5]:
 *     degree-8 polynomial in s = (1/(1 + z) - 3/16) * 9.5; each the
 *     binary32-rounded monomial coefficients of the Chebyshev interpolant of
 *     exp(z^2) erfc(z) (points cos(pi (2k+1) / (2(d+1))) in s), by Horner with fma;
 *     exp(-c x^2) = exp_rep(-(h*h) c) * exp_rep(-((x - h)(x + h)) c), h = x with
 *     its low 12 significand bits cleared.
 *   Y may equal X.
 */
repops_status_t repops_erf(const repops_order_t *order, int64_t n, const float *X, float *Y,
                           const repops_launch_t *launch, void *hip_stream);

/*
 * repops_gelu_erf -- the erf form of GELU (DistilBERT's activation, Section
 * 4.2): y = x * Phi(x), with z = |x| RN(1/sqrt 2):
 *     z < 0.5: Phi = fma(0.5, erf(x RN(1/sqrt 2)), 0.5);
 *     else q = RN(exp(-x^2/2) R(z)) * 0.5 (0 for z >= 10.5), Phi = 1 - q for
 *     x > 0 and q otherwise.
 *   Y may equal X.
 */
repops_status_t repops_gelu_erf(const repops_order_t *order, int64_t n, const float *X, float *Y,
                                const repops_launch_t *launch, void *hip_stream);

/*
 * repops_gelu_erf_backward -- dx = dy * (Phi(x) + x phi(x)) with
 * phi(x) = RN(exp(-x^2/2) * RN(1/sqrt(2 pi))):  gelu' = fma(x, phi, Phi(x)).
 *   dX may coincide exactly with X or dY.
 */
repops_status_t repops_gelu_erf_backward(const repops_order_t *order, int64_t n, const float *X,
                                         const float *dY, float *dX, const repops_launch_t *launch,
                                         void *hip_stream);

#ifdef __cplusplus
}
#endif
#endif
