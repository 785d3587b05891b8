/*
 * repops_ref.c -- CPU oracle for the RepOps operators (Verde, arXiv 2502.19405,
 * Section 3 "Reproducible Operations (RepOps) library").
 *
 * TEST INFRASTRUCTURE ONLY: loaded by the test suite, the smoke check and the
 * benchmark's CPU-baseline leg; never by the GPU library or its binding.
 *
 * Every function below is the plain statement of one operator as a fixed
 * sequence of IEEE-754 binary32 operations, written for a reader to check
 * against the paper by eye: no blocking, fusion or reordering beyond what the
 * definition states.  Threads only split independent outputs (rows), never the
 * operation sequence of one output.
 *
 * Build (strict IEEE on the host): gcc -std=c11 -O2 -ffp-contract=off
 * -fno-fast-math -mfma -fexcess-precision=standard.  -ffp-contract=off keeps
 * every a*b+c written below as two rounded operations; fmaf() is the single
 * rounding fused multiply-add.
 *
 * Where the paper fixes the order (the matrix-multiplication listing of
 * Section 3.2) the code follows it; where the paper is silent (block constant,
 * row reductions, exp, GELU, softmax, LayerNorm) the chosen reading is stated
 * at the definition.
 */
#define _GNU_SOURCE
#include "repops_ref.h"

#include <fenv.h>
#include <float.h>
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <unistd.h>

/* ------------------------------------------------------------------------- */
/* Floating-point environment                                                */
/* ------------------------------------------------------------------------- */

/* Section 3.3: RepOps assumes IEEE-754 binary32 arithmetic.  On x86-64 that
 * means SSE scalar arithmetic (no x87 excess precision), round-to-nearest-even,
 * and gradual underflow (MXCSR FTZ/DAZ clear).  Each worker thread installs the
 * default environment, which clears FTZ/DAZ a foreign library may have set. */
static void install_ieee_env(void) { fesetenv(FE_DFL_ENV); }

static float bits_to_float(uint32_t u) { float f; memcpy(&f, &u, 4); return f; }

int repops_ref_env_check(void)
{
    fenv_t saved;
    fegetenv(&saved);
    install_ieee_env();
    int bad = 0;
    /* A case where fused and unfused results differ: a = b = 1 + 2^-12 and
     * c = -(1 + 2^-11).  a*b = 1 + 2^-11 + 2^-24 exactly, so the fused result
     * is 2^-24 while RN(a*b) = 1 + 2^-11 cancels c to 0. */
    volatile float a = bits_to_float(0x3f800800u); /* 1 + 2^-12 */
    volatile float c = bits_to_float(0xbf801000u); /* -(1 + 2^-11) */
    if (fmaf(a, a, c) != bits_to_float(0x33800000u)) bad |= 1; /* 2^-24 */
    volatile float tiny = FLT_MIN;                   /* 2^-126 */
    volatile float half = 0.5f;
    if (tiny * half == 0.0f) bad |= 2;
    if (fegetround() != FE_TONEAREST) bad |= 4;
    if (FLT_EVAL_METHOD != 0) bad |= 8;
    fesetenv(&saved);
    return bad;
}

/* ------------------------------------------------------------------------- */
/* Thread helper: split [0, count) into contiguous chunks                    */
/* ------------------------------------------------------------------------- */

typedef void (*range_fn)(void *ctx, int64_t begin, int64_t end);

typedef struct {
    range_fn fn;
    void *ctx;
    int64_t begin, end;
} range_job;

static void *range_worker(void *arg)
{
    range_job *job = (range_job *)arg;
    install_ieee_env();
    job->fn(job->ctx, job->begin, job->end);
    return NULL;
}

int repops_ref_default_threads(void)
{
    long n = sysconf(_SC_NPROCESSORS_ONLN);
    return n > 0 ? (int)n : 1;
}

static void parallel_for(int nthreads, int64_t count, range_fn fn, void *ctx)
{
    if (count <= 0) return;
    if (nthreads <= 0) nthreads = repops_ref_default_threads();
    if (nthreads > 256) nthreads = 256;
    if ((int64_t)nthreads > count) nthreads = (int)count;
    fenv_t saved;
    fegetenv(&saved);
    if (nthreads == 1) {
        install_ieee_env();
        fn(ctx, 0, count);
        fesetenv(&saved);
        return;
    }
    pthread_t tid[256];
    range_job job[256];
    int started = 0;
    for (int t = 0; t < nthreads; ++t) {
        job[t].fn = fn;
        job[t].ctx = ctx;
        job[t].begin = count * t / nthreads;
        job[t].end = count * (t + 1) / nthreads;
        if (pthread_create(&tid[t], NULL, range_worker, &job[t]) == 0) {
            ++started;
        } else {
            /* Could not start a thread: run its share here. */
            tid[t] = 0;
            install_ieee_env();
            fn(ctx, job[t].begin, job[t].end);
        }
    }
    for (int t = 0; t < nthreads; ++t)
        if (tid[t]) pthread_join(tid[t], NULL);
    (void)started;
    fesetenv(&saved);
}

/* ------------------------------------------------------------------------- */
/* c1: the canonical contraction                                             */
/* ------------------------------------------------------------------------- */

/*
 * Section 3.2, the matrix-multiplication contraction: the output indices
 * (i, j) may be visited in any order; for each output a running sum over k,
 * started at zero, takes one product term at a time in one fixed order.
 *
 * Reading used here (the paper gives no block constant): the k range is cut
 * into consecutive blocks of k_block indices, the last one possibly shorter.
 * Each block's partial starts at +0 and takes its terms in ascending k; the
 * partials are then added left to right, in ascending block order, into an
 * accumulator that starts at +0.  k_block = 0 means a single block covering the
 * whole range, which is the listing itself.  The term update is a fused
 * multiply-add (k_inner = 0) or a rounded product followed by a rounded add
 * (k_inner = 1): the paper's term update may be read either way.
 */
float repops_ref_dot(int64_t k_block, int k_inner, int64_t K,
                     const float *a, int64_t inc_a, const float *b, int64_t inc_b)
{
    const int64_t blk = (k_block > 0) ? k_block : K;
    float acc = 0.0f;
    for (int64_t k0 = 0; k0 < K; k0 += blk) {
        const int64_t k1 = (k0 + blk < K) ? k0 + blk : K;
        float p = 0.0f;
        for (int64_t k = k0; k < k1; ++k) {
            const float x = a[k * inc_a];
            const float y = b[k * inc_b];
            if (k_inner == REF_INNER_FMA) {
                p = fmaf(x, y, p);
            } else {
                const float prod = x * y;
                p = p + prod;
            }
        }
        acc = acc + p;
    }
    return acc;
}

static int check_order_k(int64_t k_block, int k_inner)
{
    if (k_block < 0) return -1;
    if (k_inner != REF_INNER_FMA && k_inner != REF_INNER_MUL_ADD) return -1;
    return 0;
}

/* Logical element A[i][k] / B[k][j] and the stride that walks k. */
static const float *row_of_a(const float *A, int64_t lda, int trans_a, int64_t i, int64_t *inc)
{
    if (trans_a) { *inc = lda; return A + i; }
    *inc = 1;
    return A + i * lda;
}

static const float *col_of_b(const float *B, int64_t ldb, int trans_b, int64_t j, int64_t *inc)
{
    if (trans_b) { *inc = 1; return B + j * ldb; }
    *inc = ldb;
    return B + j;
}

/*
 * Layout only: an operand whose k walk is strided in memory (A read
 * transposed, B read as stored) is first copied into one contiguous vector per
 * output row (of A) or output column (of B), so that every dot product reads
 * memory with unit stride.  Values are copied unchanged and each output still
 * takes its terms in ascending k, so the results are the same bits.  The copy
 * covers batch0 x batch1 x count vectors of k elements: vector (b0, b1, r)
 * holds the elements at src + b0 s0 + b1 s1 + r + kk inc, kk = 0 .. k-1.
 */
typedef struct {
    const float *src; int64_t s0, s1, batch1, count, k, inc;
    float *dst;
} gather_ctx;

static void gather_range(void *vctx, int64_t v0, int64_t v1)
{
    const gather_ctx *c = (const gather_ctx *)vctx;
    for (int64_t v = v0; v < v1; ++v) {
        const int64_t r = v % c->count, b = v / c->count;
        const float *p = c->src + (b / c->batch1) * c->s0 + (b % c->batch1) * c->s1 + r;
        float *d = c->dst + v * c->k;
        for (int64_t kk = 0; kk < c->k; ++kk) d[kk] = p[kk * c->inc];
    }
}

/* Contiguous copy of a strided operand, or NULL (then the strided operand is
 * read in place: same values, same order, only slower). */
static float *gather(const float *src, int64_t s0, int64_t s1, int64_t batch0, int64_t batch1,
                     int64_t count, int64_t k, int64_t inc, int nthreads)
{
    const int64_t nvec = batch0 * batch1 * count;
    if (nvec <= 0 || k <= 0 || (uint64_t)nvec > SIZE_MAX / sizeof(float) / (uint64_t)k)
        return NULL;
    float *dst = (float *)malloc((size_t)(nvec * k) * sizeof(float));
    if (!dst) return NULL;
    gather_ctx c = {src, s0, s1, batch1, count, k, inc, dst};
    parallel_for(nthreads, nvec, gather_range, &c);
    return dst;
}

/* Epilogue (paper silent; reading used here): the scale alpha multiplies the
 * finished contraction, then the bias is added, each one rounding. */
typedef struct {
    int64_t k_block;
    int k_inner;
    int64_t n, k;
    const float *A; int64_t lda; int trans_a;
    const float *B; int64_t ldb; int trans_b;
    const float *bias;
    float *C; int64_t ldc;
    const float *Ag, *Bg;  /* contiguous copies (row i of A, column j of B) or NULL */
} matmul_ctx;

static void matmul_rows(void *vctx, int64_t i0, int64_t i1)
{
    const matmul_ctx *c = (const matmul_ctx *)vctx;
    for (int64_t i = i0; i < i1; ++i) {
        for (int64_t j = 0; j < c->n; ++j) {
            int64_t ia, ib;
            const float *a = row_of_a(c->A, c->lda, c->trans_a, i, &ia);
            const float *b = col_of_b(c->B, c->ldb, c->trans_b, j, &ib);
            if (c->Ag) { a = c->Ag + i * c->k; ia = 1; }
            if (c->Bg) { b = c->Bg + j * c->k; ib = 1; }
            float v = repops_ref_dot(c->k_block, c->k_inner, c->k, a, ia, b, ib);
            if (c->bias) v = v + c->bias[j];
            c->C[i * c->ldc + j] = v;
        }
    }
}

int repops_ref_matmul(int64_t k_block, int k_inner, int64_t m, int64_t n, int64_t k,
                      const float *A, int64_t lda, int trans_a,
                      const float *B, int64_t ldb, int trans_b,
                      const float *bias, float *C, int64_t ldc, int nthreads)
{
    if (check_order_k(k_block, k_inner) || m < 0 || n < 0 || k < 0) return -1;
    if (m == 0 || n == 0) return 0;
    if (!C || (k > 0 && (!A || !B))) return -2;
    float *Ag = (k > 0 && trans_a) ? gather(A, 0, 0, 1, 1, m, k, lda, nthreads) : NULL;
    float *Bg = (k > 0 && !trans_b) ? gather(B, 0, 0, 1, 1, n, k, ldb, nthreads) : NULL;
    matmul_ctx c = {k_block, k_inner, n, k, A, lda, trans_a, B, ldb, trans_b, bias, C, ldc,
                    Ag, Bg};
    parallel_for(nthreads, m, matmul_rows, &c);
    free(Ag);
    free(Bg);
    return 0;
}

int repops_ref_matmul_at(int64_t k_block, int k_inner, int64_t m, int64_t n, int64_t k,
                         const float *A, int64_t lda, int trans_a,
                         const float *B, int64_t ldb, int trans_b,
                         const float *bias, int64_t npts, const int64_t *rows,
                         const int64_t *cols, float *out)
{
    if (check_order_k(k_block, k_inner) || m < 0 || n < 0 || k < 0 || npts < 0) return -1;
    fenv_t saved;
    fegetenv(&saved);
    install_ieee_env();
    for (int64_t p = 0; p < npts; ++p) {
        const int64_t i = rows[p], j = cols[p];
        if (i < 0 || i >= m || j < 0 || j >= n) { fesetenv(&saved); return -3; }
        int64_t ia, ib;
        const float *a = row_of_a(A, lda, trans_a, i, &ia);
        const float *b = col_of_b(B, ldb, trans_b, j, &ib);
        float v = repops_ref_dot(k_block, k_inner, k, a, ia, b, ib);
        if (bias) v = v + bias[j];
        out[p] = v;
    }
    fesetenv(&saved);
    return 0;
}

/* Batched product (Section 2.2 names the attention key-query product as an
 * operator that decomposes into independent matrix products): every batch
 * element is one matrix product with the same per-output order, followed by
 * one rounded multiplication by alpha. */
typedef struct {
    int64_t k_block;
    int k_inner;
    int64_t batch1, m, n, k;
    const float *A; int64_t sa0, sa1, lda; int trans_a;
    const float *B; int64_t sb0, sb1, ldb; int trans_b;
    float alpha;
    float *C; int64_t sc0, sc1, ldc;
    const float *Ag, *Bg;  /* contiguous copies (per batch element: rows of A, columns of B) or NULL */
} bmm_ctx;

static float bmm_one(const bmm_ctx *c, int64_t b0, int64_t b1, int64_t i, int64_t j)
{
    const float *Ab = c->A + b0 * c->sa0 + b1 * c->sa1;
    const float *Bb = c->B + b0 * c->sb0 + b1 * c->sb1;
    int64_t ia, ib;
    const float *a = row_of_a(Ab, c->lda, c->trans_a, i, &ia);
    const float *b = col_of_b(Bb, c->ldb, c->trans_b, j, &ib);
    const int64_t bz = b0 * c->batch1 + b1;
    if (c->Ag) { a = c->Ag + (bz * c->m + i) * c->k; ia = 1; }
    if (c->Bg) { b = c->Bg + (bz * c->n + j) * c->k; ib = 1; }
    const float v = repops_ref_dot(c->k_block, c->k_inner, c->k, a, ia, b, ib);
    return v * c->alpha;
}

static void bmm_rows(void *vctx, int64_t r0, int64_t r1)
{
    const bmm_ctx *c = (const bmm_ctx *)vctx;
    for (int64_t r = r0; r < r1; ++r) {
        /* r enumerates (b0, b1, i) */
        const int64_t i = r % c->m;
        const int64_t b = r / c->m;
        const int64_t b1 = b % c->batch1, b0 = b / c->batch1;
        float *Cb = c->C + b0 * c->sc0 + b1 * c->sc1;
        for (int64_t j = 0; j < c->n; ++j) Cb[i * c->ldc + j] = bmm_one(c, b0, b1, i, j);
    }
}

int repops_ref_bmm(int64_t k_block, int k_inner, int64_t batch0, int64_t batch1,
                   int64_t m, int64_t n, int64_t k,
                   const float *A, int64_t sa0, int64_t sa1, int64_t lda, int trans_a,
                   const float *B, int64_t sb0, int64_t sb1, int64_t ldb, int trans_b,
                   float alpha, float *C, int64_t sc0, int64_t sc1, int64_t ldc, int nthreads)
{
    if (check_order_k(k_block, k_inner) || batch0 < 0 || batch1 < 0 || m < 0 || n < 0 || k < 0)
        return -1;
    if (batch0 == 0 || batch1 == 0 || m == 0 || n == 0) return 0;
    float *Ag = (k > 0 && trans_a) ? gather(A, sa0, sa1, batch0, batch1, m, k, lda, nthreads)
                                   : NULL;
    float *Bg = (k > 0 && !trans_b) ? gather(B, sb0, sb1, batch0, batch1, n, k, ldb, nthreads)
                                    : NULL;
    bmm_ctx c = {k_block, k_inner, batch1, m, n, k, A, sa0, sa1, lda, trans_a,
                 B, sb0, sb1, ldb, trans_b, alpha, C, sc0, sc1, ldc, Ag, Bg};
    parallel_for(nthreads, batch0 * batch1 * m, bmm_rows, &c);
    free(Ag);
    free(Bg);
    return 0;
}

int repops_ref_bmm_at(int64_t k_block, int k_inner, int64_t batch0, int64_t batch1,
                      int64_t m, int64_t n, int64_t k,
                      const float *A, int64_t sa0, int64_t sa1, int64_t lda, int trans_a,
                      const float *B, int64_t sb0, int64_t sb1, int64_t ldb, int trans_b,
                      float alpha, int64_t npts, const int64_t *b0, const int64_t *b1,
                      const int64_t *rows, const int64_t *cols, float *out)
{
    if (check_order_k(k_block, k_inner) || batch0 < 0 || batch1 < 0 || m < 0 || n < 0 || k < 0)
        return -1;
    bmm_ctx c = {k_block, k_inner, batch1, m, n, k, A, sa0, sa1, lda, trans_a,
                 B, sb0, sb1, ldb, trans_b, alpha, NULL, 0, 0, 0, NULL, NULL};
    fenv_t saved;
    fegetenv(&saved);
    install_ieee_env();
    for (int64_t p = 0; p < npts; ++p) {
        if (b0[p] < 0 || b0[p] >= batch0 || b1[p] < 0 || b1[p] >= batch1 || rows[p] < 0 ||
            rows[p] >= m || cols[p] < 0 || cols[p] >= n) {
            fesetenv(&saved);
            return -3;
        }
        out[p] = bmm_one(&c, b0[p], b1[p], rows[p], cols[p]);
    }
    fesetenv(&saved);
    return 0;
}

/* ------------------------------------------------------------------------- */
/* c2: fixed-order row reduction                                             */
/* ------------------------------------------------------------------------- */

/*
 * The paper fixes no order for row reductions; Section 3.2 only asks that the
 * order-critical dimension be serialised or synchronised in a fixed way.
 * Reading used here, a function of the row length n and the constant W only:
 *
 *   strided tree (row_combine 0): W partials q[l] start at +0; element x[j]
 *   is added to q[j mod W] in ascending j; then for s = W/2, W/4, ..., 1 each
 *   q[l] with l < s becomes q[l] + q[l+s]; the result is q[0].
 *
 *   blocked left-to-right (row_combine 1): the c1 rule with addition, blocks of
 *   W consecutive elements, block partials added left to right.
 *
 * Terms: kind 0 adds a_j (q + a_j); kind 1 is a sum of squares, fma(a_j, a_j, q);
 * kind 2 an inner product, fma(a_j, b_j, q).  Positions j >= valid contribute
 * no operation (masked columns), but keep their place in the order.
 */
static float term2(float q, const float *a, const float *b, int64_t j, int kind)
{
    if (kind == 0) return q + a[j];
    if (kind == 1) return fmaf(a[j], a[j], q);
    return fmaf(a[j], b[j], q);
}

static float rowsum_terms(int row_width, int row_combine, int64_t n, int64_t valid,
                          const float *a, const float *b, int kind)
{
    const int64_t W = row_width;
    if (row_combine == REF_ROW_BLOCKED) {
        float acc = 0.0f;
        for (int64_t j0 = 0; j0 < n; j0 += W) {
            float p = 0.0f;
            for (int64_t j = j0; j < j0 + W && j < n; ++j)
                if (j < valid) p = term2(p, a, b, j, kind);
            acc = acc + p;
        }
        return acc;
    }
    float q[1024];
    for (int64_t l = 0; l < W; ++l) q[l] = 0.0f;
    for (int64_t j = 0; j < n; ++j)
        if (j < valid) q[j % W] = term2(q[j % W], a, b, j, kind);
    for (int64_t s = W / 2; s >= 1; s /= 2)
        for (int64_t l = 0; l < s; ++l) q[l] = q[l] + q[l + s];
    return q[0];
}

float repops_ref_rowsum(int row_width, int row_combine, int64_t n, const float *x, int squares)
{
    return rowsum_terms(row_width, row_combine, n, n, x, NULL, squares ? 1 : 0);
}

static int check_order_rows(int row_width, int row_combine)
{
    if (row_width < 1 || row_width > 1024 || (row_width & (row_width - 1))) return -1;
    if (row_combine != REF_ROW_TREE && row_combine != REF_ROW_BLOCKED) return -1;
    return 0;
}

/* ------------------------------------------------------------------------- */
/* c4: reproducible exp                                                      */
/* ------------------------------------------------------------------------- */

/*
 * Section 3.1: RepOps rebuilds exp (and the other math functions) so that the
 * operation order is controlled.  The paper gives no algorithm; the one used
 * here is Cody and Waite's additive argument reduction followed by the degree-7
 * Taylor polynomial of exp, evaluated by Horner's rule with fused multiply-adds:
 *
 *   n = rint(x * log2 e)                (nearest integer, ties to even)
 *   r = (x - n*ln2_hi) - n*ln2_lo       (two fused steps)
 *   p = sum_{i<=7} r^i / i!             (Horner, highest coefficient first)
 *   exp(x) = p * 2^n, applied as (p * 2^floor(n/2)) * 2^(n - floor(n/2))
 *
 * The split scaling keeps both powers of two normal, so the first product is
 * exact and the second rounds once, giving correctly handled overflow and
 * subnormal results.  Constants are the binary32 values nearest their
 * definitions: log2 e; ln2_hi = RN(ln 2); ln2_lo = RN(ln 2 - ln2_hi);
 * coefficients RN(1/i!).
 */
static const float EXP_LOG2E = 0x1.715476p+0f;
static const float EXP_LN2_HI = 0x1.62e43p-1f;
static const float EXP_LN2_LO = -0x1.05c61p-29f;
static const float EXP_C[8] = {
    0x1p+0f,        /* 1/0! */
    0x1p+0f,        /* 1/1! */
    0x1p-1f,        /* 1/2! */
    0x1.555556p-3f, /* 1/3! */
    0x1.555556p-5f, /* 1/4! */
    0x1.111112p-7f, /* 1/5! */
    0x1.6c16c2p-10f,/* 1/6! */
    0x1.a01a02p-13f /* 1/7! */
};

/* 2^e for an integer e in [-126, 127], built from the exponent field. */
static float pow2i(int e)
{
    return bits_to_float((uint32_t)(e + 127) << 23);
}

float repops_ref_exp1(float x)
{
    if (isnan(x)) return x;
    const float t = x * EXP_LOG2E;
    const float nf = rintf(t);
    if (nf > 128.0f) return INFINITY;
    if (nf < -151.0f) return 0.0f;
    float r = fmaf(nf, -EXP_LN2_HI, x);
    r = fmaf(nf, -EXP_LN2_LO, r);
    float p = EXP_C[7];
    for (int i = 6; i >= 0; --i) p = fmaf(p, r, EXP_C[i]);
    const int n = (int)nf;
    const int n1 = (n >= 0) ? n / 2 : -((-n + 1) / 2); /* floor(n / 2) */
    const int n2 = n - n1;
    const float y = p * pow2i(n1);
    return y * pow2i(n2);
}

/* ------------------------------------------------------------------------- */
/* c5: tanh-form GELU                                                        */
/* ------------------------------------------------------------------------- */

/*
 * GELU appears among the DistilBERT operators of Section 4.2.  The tanh form
 * 0.5*x*(1 + tanh(z)), z = sqrt(2/pi)*(x + 0.044715*x^3), is rewritten with the
 * identity 0.5*(1 + tanh z) = 1 / (1 + exp(-2z)), which avoids the cancellation
 * in 1 + tanh z for negative z:
 *
 *   u = (x*x)*x;  z = fma(0.044715, u, x) * sqrt(2/pi);  w = -2*z (exact)
 *   y = x / (1 + exp_rep(w))
 *
 * Constants: RN(0.044715) and RN(sqrt(2/pi)).
 */
static const float GELU_C = 0x1.6e4e26p-5f;
static const float GELU_SQ = 0x1.988454p-1f;

float repops_ref_gelu1(float x)
{
    float u = x * x;
    u = u * x;
    float z = fmaf(GELU_C, u, x);
    z = z * GELU_SQ;
    const float w = z * -2.0f;
    const float e = repops_ref_exp1(w);
    const float d = 1.0f + e;
    return x / d;
}

typedef struct {
    const float *x;
    float *y;
    int which; /* 0 = exp, 1 = gelu */
} ew_ctx;

static void ew_range(void *vctx, int64_t i0, int64_t i1)
{
    const ew_ctx *c = (const ew_ctx *)vctx;
    if (c->which == 0)
        for (int64_t i = i0; i < i1; ++i) c->y[i] = repops_ref_exp1(c->x[i]);
    else
        for (int64_t i = i0; i < i1; ++i) c->y[i] = repops_ref_gelu1(c->x[i]);
}

int repops_ref_exp(int64_t n, const float *x, float *y, int nthreads)
{
    if (n < 0) return -1;
    ew_ctx c = {x, y, 0};
    parallel_for(nthreads, n, ew_range, &c);
    return 0;
}

int repops_ref_gelu(int64_t n, const float *x, float *y, int nthreads)
{
    if (n < 0) return -1;
    ew_ctx c = {x, y, 1};
    parallel_for(nthreads, n, ew_range, &c);
    return 0;
}

/* ------------------------------------------------------------------------- */
/* c6: row softmax                                                           */
/* ------------------------------------------------------------------------- */

/*
 * Softmax is not named in the paper; it is one of the operators needed to run
 * the DistilBERT and Llama programs of Section 4.2.  Reading used here:
 *
 *   m   = maximum of the unmasked entries (first maximum kept on ties);
 *   e_j = exp_rep(x_j - m) for unmasked j, +0 for masked j;
 *   s   = fixed-order row sum of e (c2, masked terms included as +0);
 *   r   = 1 / s, once per row;  y_j = e_j * r.
 *
 * The causal mask of row i keeps columns j <= i mod causal_period.
 */
typedef struct {
    int W, combine;
    int64_t cols;
    const float *X; int64_t ldx;
    float *Y; int64_t ldy;
    int64_t period;
} softmax_ctx;

static void softmax_range(void *vctx, int64_t r0, int64_t r1)
{
    const softmax_ctx *c = (const softmax_ctx *)vctx;
    float *e = (float *)malloc(sizeof(float) * (size_t)(c->cols > 0 ? c->cols : 1));
    if (!e) abort();
    for (int64_t r = r0; r < r1; ++r) {
        const float *x = c->X + r * c->ldx;
        float *y = c->Y + r * c->ldy;
        const int64_t valid = (c->period > 0) ? (r % c->period) + 1 : c->cols;
        const int64_t nv = valid < c->cols ? valid : c->cols;
        float m = -INFINITY;
        for (int64_t j = 0; j < nv; ++j) m = (x[j] > m) ? x[j] : m;
        for (int64_t j = 0; j < c->cols; ++j) {
            if (j < nv) {
                const float d = x[j] - m;
                e[j] = repops_ref_exp1(d);
            } else {
                e[j] = 0.0f;
            }
        }
        const float s = repops_ref_rowsum(c->W, c->combine, c->cols, e, 0);
        const float rs = 1.0f / s;
        for (int64_t j = 0; j < c->cols; ++j) y[j] = e[j] * rs;
    }
    free(e);
}

int repops_ref_softmax_rows(int row_width, int row_combine, int64_t rows, int64_t cols,
                            const float *X, int64_t ldx, float *Y, int64_t ldy,
                            int64_t causal_period, int nthreads)
{
    if (check_order_rows(row_width, row_combine) || rows < 0 || cols < 0 || causal_period < 0)
        return -1;
    softmax_ctx c = {row_width, row_combine, cols, X, ldx, Y, ldy, causal_period};
    parallel_for(nthreads, rows, softmax_range, &c);
    return 0;
}

/* ------------------------------------------------------------------------- */
/* c7: row LayerNorm                                                         */
/* ------------------------------------------------------------------------- */

/*
 * LayerNorm is named among the DistilBERT operators of Section 4.2; the paper
 * gives no formula or order.  Reading used here (biased variance, as in the
 * usual LayerNorm definition):
 *
 *   mean = rowsum(x) / n;  d_j = x_j - mean;
 *   var  = rowsum of fma(d, d, .) / n;
 *   rstd = 1 / sqrt(var + eps)   (correctly rounded sqrt and division);
 *   t_j  = d_j * rstd;  y_j = fma(t_j, gamma_j, beta_j).
 *
 * A missing gamma or beta skips its operation: y = t, t + beta or t * gamma.
 */
typedef struct {
    int W, combine;
    int64_t cols;
    const float *X; int64_t ldx;
    const float *gamma, *beta;
    float eps;
    float *Y; int64_t ldy;
    float *mean_out, *rstd_out;
} ln_ctx;

static void ln_range(void *vctx, int64_t r0, int64_t r1)
{
    const ln_ctx *c = (const ln_ctx *)vctx;
    float *d = (float *)malloc(sizeof(float) * (size_t)(c->cols > 0 ? c->cols : 1));
    if (!d) abort();
    const float nf = (float)c->cols;
    for (int64_t r = r0; r < r1; ++r) {
        const float *x = c->X + r * c->ldx;
        float *y = c->Y + r * c->ldy;
        const float s = repops_ref_rowsum(c->W, c->combine, c->cols, x, 0);
        const float mean = s / nf;
        for (int64_t j = 0; j < c->cols; ++j) d[j] = x[j] - mean;
        const float q = repops_ref_rowsum(c->W, c->combine, c->cols, d, 1);
        const float var = q / nf;
        const float ve = var + c->eps;
        const float sd = sqrtf(ve);
        const float rstd = 1.0f / sd;
        for (int64_t j = 0; j < c->cols; ++j) {
            const float t = d[j] * rstd;
            float v;
            if (c->gamma && c->beta) v = fmaf(t, c->gamma[j], c->beta[j]);
            else if (c->gamma) v = t * c->gamma[j];
            else if (c->beta) v = t + c->beta[j];
            else v = t;
            y[j] = v;
        }
        if (c->mean_out) c->mean_out[r] = mean;
        if (c->rstd_out) c->rstd_out[r] = rstd;
    }
    free(d);
}

int repops_ref_layernorm_rows(int row_width, int row_combine, int64_t rows, int64_t cols,
                              const float *X, int64_t ldx, const float *gamma,
                              const float *beta, float eps, float *Y, int64_t ldy,
                              float *mean_out, float *rstd_out, int nthreads)
{
    if (check_order_rows(row_width, row_combine) || rows < 0 || cols < 0) return -1;
    if (rows > 0 && cols == 0) return -1; /* mean of an empty row is undefined */
    ln_ctx c = {row_width, row_combine, cols, X, ldx, gamma, beta, eps, Y, ldy, mean_out, rstd_out};
    parallel_for(nthreads, rows, ln_range, &c);
    return 0;
}

/* ========================================================================= */
/* Llama-block operators: sin/cos and rotary embedding, RMSNorm, SiLU/SwiGLU  */
/* ========================================================================= */

/*
 * The Llama programs of Section 4.2 add rotary position embeddings, RMSNorm
 * and the SiLU-gated feed-forward to the operators above.  Section 3.1 lists
 * the math functions RepOps rebuilds with a controlled order; sin and cos are
 * rebuilt here in the style of exp: Cody and Waite's additive reduction by
 * pi/2 (pi/2 split in three binary32 parts), Taylor polynomials on
 * |r| <= pi/4 by Horner's rule with fused multiply-adds, quadrant selection.
 * Reading (op sequence):
 *   non-finite x: both results NaN;  x = +-0: (sin, cos) = (x, 1);
 *   n = rint(x * RN(2/pi)) (ties to even);
 *   n = 0: r = x; else r = fma(n, -P1, x); r = fma(n, -P2, r); r = fma(n, -P3, r)
 *     with P1 = RN(pi/2), P2 = RN(pi/2 - P1), P3 = RN(pi/2 - P1 - P2);
 *   u = r*r;
 *   sin part: p = fma(S9, u, S7); p = fma(p, u, S5); p = fma(p, u, S3);
 *             s = fma(r*u, p, r)                 (S_k = RN((-1)^((k-1)/2) / k!));
 *   cos part: p = fma(C10, u, C8); p = fma(p, u, C6); p = fma(p, u, C4);
 *             p = fma(p, u, C2); c = fma(u, p, 1) (C_k = RN((-1)^(k/2) / k!));
 *   q = n - 4 floor(n/4) (exact, in {0,1,2,3}):
 *     (sin, cos) = (s, c), (c, -s), (-s, -c), (-c, s) for q = 0..3.
 * Accurate to a few ulp for |x| <= 2^17 (the angles of rotary embeddings);
 * beyond that the results stay reproducible but lose accuracy.
 */
static const float SC_TWO_OVER_PI = 0x1.45f306p-1f;
static const float SC_P1 = 0x1.921fb6p+0f;
static const float SC_P2 = -0x1.777a5cp-25f;
static const float SC_P3 = -0x1.ee59dap-50f;
static const float SC_S3 = -0x1.555556p-3f;  /* -1/3! */
static const float SC_S5 = 0x1.111112p-7f;   /* 1/5! */
static const float SC_S7 = -0x1.a01a02p-13f; /* -1/7! */
static const float SC_S9 = 0x1.71de3ap-19f;  /* 1/9! */
static const float SC_C2 = -0x1p-1f;         /* -1/2! */
static const float SC_C4 = 0x1.555556p-5f;   /* 1/4! */
static const float SC_C6 = -0x1.6c16c2p-10f; /* -1/6! */
static const float SC_C8 = 0x1.a01a02p-16f;  /* 1/8! */
static const float SC_C10 = -0x1.27e4fcp-22f; /* -1/10! */

void repops_ref_sincos1(float x, float *sin_out, float *cos_out)
{
    if (!isfinite(x)) {
        *sin_out = NAN;
        *cos_out = NAN;
        return;
    }
    if (x == 0.0f) { /* keeps the sign of zero, which the fused step would lose */
        *sin_out = x;
        *cos_out = 1.0f;
        return;
    }
    const float t = x * SC_TWO_OVER_PI;
    const float n = rintf(t);
    float r = x;
    if (n != 0.0f) {
        r = fmaf(n, -SC_P1, x);
        r = fmaf(n, -SC_P2, r);
        r = fmaf(n, -SC_P3, r);
    }
    const float u = r * r;
    float ps = fmaf(SC_S9, u, SC_S7);
    ps = fmaf(ps, u, SC_S5);
    ps = fmaf(ps, u, SC_S3);
    const float r3 = r * u;
    const float sv = fmaf(r3, ps, r);
    float pc = fmaf(SC_C10, u, SC_C8);
    pc = fmaf(pc, u, SC_C6);
    pc = fmaf(pc, u, SC_C4);
    pc = fmaf(pc, u, SC_C2);
    const float cv = fmaf(u, pc, 1.0f);
    const float quarter = n * 0.25f;
    const float fq = n - 4.0f * floorf(quarter);
    const int q = (int)fq;
    if (q == 0) { *sin_out = sv; *cos_out = cv; }
    else if (q == 1) { *sin_out = cv; *cos_out = -sv; }
    else if (q == 2) { *sin_out = -sv; *cos_out = -cv; }
    else { *sin_out = -cv; *cos_out = sv; }
}

typedef struct {
    const float *x;
    float *s, *c;
} sc_ctx;

static void sincos_range(void *vctx, int64_t i0, int64_t i1)
{
    const sc_ctx *k = (const sc_ctx *)vctx;
    for (int64_t i = i0; i < i1; ++i) {
        float sv, cv;
        repops_ref_sincos1(k->x[i], &sv, &cv);
        if (k->s) k->s[i] = sv;
        if (k->c) k->c[i] = cv;
    }
}

int repops_ref_sincos(int64_t n, const float *x, float *s, float *c, int nthreads)
{
    if (n < 0) return -1;
    sc_ctx k = {x, s, c};
    parallel_for(nthreads, n, sincos_range, &k);
    return 0;
}

/*
 * Rotary position embedding (rotate-half pairing within each head): row r of
 * X holds `heads` heads of `head_dim` (even) values; its position is
 * p = r mod period (period 0: p = r) plus offset.  For i < head_dim/2:
 *   angle = RN(p * inv_freq[i])  (p converted exactly: p < 2^24);
 *   c, s = cos_rep(angle), sin_rep(angle);
 *   x1 = X[.., i], x2 = X[.., i + head_dim/2];
 *   forward: y1 = RN(RN(x1 c) - RN(x2 s)),  y2 = RN(RN(x2 c) + RN(x1 s));
 *   inverse (the backward, rotation by -angle):
 *            y1 = RN(RN(x1 c) + RN(x2 s)),  y2 = RN(RN(x2 c) - RN(x1 s)).
 * inv_freq is the model's frequency table, an input like a weight.
 */
typedef struct {
    int64_t heads, hd, period, offset;
    const float *X; int64_t ldx;
    const float *inv_freq;
    float *Y; int64_t ldy;
    int inverse;
} rope_ctx;

static void rope_range(void *vctx, int64_t r0, int64_t r1)
{
    const rope_ctx *c = (const rope_ctx *)vctx;
    const int64_t half = c->hd / 2;
    for (int64_t r = r0; r < r1; ++r) {
        const int64_t p = (c->period > 0 ? r % c->period : r) + c->offset;
        const float pf = (float)p;
        const float *x = c->X + r * c->ldx;
        float *y = c->Y + r * c->ldy;
        for (int64_t i = 0; i < half; ++i) {
            const float angle = pf * c->inv_freq[i];
            float sv, cv;
            repops_ref_sincos1(angle, &sv, &cv);
            for (int64_t h = 0; h < c->heads; ++h) {
                const float x1 = x[h * c->hd + i], x2 = x[h * c->hd + i + half];
                const float a = x1 * cv, b = x2 * sv, d = x2 * cv, e = x1 * sv;
                if (!c->inverse) {
                    y[h * c->hd + i] = a - b;
                    y[h * c->hd + i + half] = d + e;
                } else {
                    y[h * c->hd + i] = a + b;
                    y[h * c->hd + i + half] = d - e;
                }
            }
        }
    }
}

int repops_ref_rope(int64_t rows, int64_t heads, int64_t head_dim, const float *X, int64_t ldx,
                    const float *inv_freq, int64_t period, int64_t offset, int inverse,
                    float *Y, int64_t ldy, int nthreads)
{
    if (rows < 0 || heads < 0 || head_dim < 0 || (head_dim & 1) || period < 0 || offset < 0)
        return -1;
    if (rows > 0 && (period > 0 ? period - 1 : rows - 1) + offset >= (int64_t)1 << 24) return -1;
    rope_ctx c = {heads, head_dim, period, offset, X, ldx, inv_freq, Y, ldy, inverse};
    parallel_for(nthreads, rows, rope_range, &c);
    return 0;
}

/*
 * RMSNorm (Llama's normalisation), with the row order of c2:
 *   ms = rowsum(fma(x_j, x_j, .)) / n;  rstd = 1 / sqrt(ms + eps);
 *   t_j = x_j * rstd;  y_j = t_j * gamma_j (t_j when gamma is absent).
 * Backward, from the forward's rstd:
 *   g_j = dy_j * gamma_j (dy_j);  b = rowsum(fma(g_j, t_j, .)) / n;
 *   dx_j = rstd * (g_j - t_j * b);
 *   dgamma_j = sum over rows of dy_ij * t_ij with the contraction rule
 *   (blocks of k_block rows, fma chains, block partials left to right).
 */
typedef struct {
    int W, combine;
    int64_t cols;
    const float *X; int64_t ldx;
    const float *gamma;
    float eps;
    float *Y; int64_t ldy;
    float *rstd_out;
} rms_ctx;

static void rms_range(void *vctx, int64_t r0, int64_t r1)
{
    const rms_ctx *c = (const rms_ctx *)vctx;
    const float nf = (float)c->cols;
    for (int64_t r = r0; r < r1; ++r) {
        const float *x = c->X + r * c->ldx;
        float *y = c->Y + r * c->ldy;
        const float q = rowsum_terms(c->W, c->combine, c->cols, c->cols, x, NULL, 1);
        const float ms = q / nf;
        const float ve = ms + c->eps;
        const float sd = sqrtf(ve);
        const float rstd = 1.0f / sd;
        for (int64_t j = 0; j < c->cols; ++j) {
            const float t = x[j] * rstd;
            y[j] = c->gamma ? t * c->gamma[j] : t;
        }
        if (c->rstd_out) c->rstd_out[r] = rstd;
    }
}

int repops_ref_rmsnorm_rows(int row_width, int row_combine, int64_t rows, int64_t cols,
                            const float *X, int64_t ldx, const float *gamma, float eps,
                            float *Y, int64_t ldy, float *rstd_out, int nthreads)
{
    if (check_order_rows(row_width, row_combine) || rows < 0 || cols < 0) return -1;
    if (rows > 0 && cols == 0) return -1;
    rms_ctx c = {row_width, row_combine, cols, X, ldx, gamma, eps, Y, ldy, rstd_out};
    parallel_for(nthreads, rows, rms_range, &c);
    return 0;
}

typedef struct {
    int W, combine;
    int64_t cols;
    const float *X; int64_t ldx;
    const float *dY; int64_t lddy;
    const float *rstd, *gamma;
    float *dX; int64_t lddx;
} rmsb_ctx;

static void rms_bwd_range(void *vctx, int64_t r0, int64_t r1)
{
    const rmsb_ctx *c = (const rmsb_ctx *)vctx;
    const size_t n = (size_t)(c->cols > 0 ? c->cols : 1);
    float *t = (float *)malloc(sizeof(float) * n);
    float *g = (float *)malloc(sizeof(float) * n);
    if (!t || !g) abort();
    const float nf = (float)c->cols;
    for (int64_t r = r0; r < r1; ++r) {
        const float *x = c->X + r * c->ldx;
        const float *dy = c->dY + r * c->lddy;
        float *dx = c->dX + r * c->lddx;
        const float rstd = c->rstd[r];
        for (int64_t j = 0; j < c->cols; ++j) {
            t[j] = x[j] * rstd;
            g[j] = c->gamma ? dy[j] * c->gamma[j] : dy[j];
        }
        const float b = rowsum_terms(c->W, c->combine, c->cols, c->cols, g, t, 2) / nf;
        for (int64_t j = 0; j < c->cols; ++j) {
            const float tb = t[j] * b;
            const float w = g[j] - tb;
            dx[j] = rstd * w;
        }
    }
    free(t);
    free(g);
}

typedef struct {
    int64_t k_block, rows, cols;
    const float *X; int64_t ldx;
    const float *dY; int64_t lddy;
    const float *rstd;
    float *dgamma;
} rmsp_ctx;

static void rms_param_range(void *vctx, int64_t j0, int64_t j1)
{
    const rmsp_ctx *c = (const rmsp_ctx *)vctx;
    const int64_t blk = c->k_block > 0 ? c->k_block : c->rows;
    for (int64_t j = j0; j < j1; ++j) {
        float acc = 0.0f;
        for (int64_t i0 = 0; i0 < c->rows; i0 += blk) {
            const int64_t i1 = (i0 + blk < c->rows) ? i0 + blk : c->rows;
            float pg = 0.0f;
            for (int64_t i = i0; i < i1; ++i) {
                const float t = c->X[i * c->ldx + j] * c->rstd[i];
                pg = fmaf(c->dY[i * c->lddy + j], t, pg);
            }
            acc = acc + pg;
        }
        c->dgamma[j] = acc;
    }
}

int repops_ref_rmsnorm_backward_rows(int row_width, int row_combine, int64_t k_block,
                                     int64_t rows, int64_t cols, const float *X, int64_t ldx,
                                     const float *dY, int64_t lddy, const float *rstd,
                                     const float *gamma, float *dX, int64_t lddx, float *dgamma,
                                     int nthreads)
{
    if (check_order_rows(row_width, row_combine) || k_block < 0 || rows < 0 || cols < 0)
        return -1;
    if (rows > 0 && cols == 0) return -1;
    if (dX) {
        rmsb_ctx c = {row_width, row_combine, cols, X, ldx, dY, lddy, rstd, gamma, dX, lddx};
        parallel_for(nthreads, rows, rms_bwd_range, &c);
    }
    if (dgamma) {
        rmsp_ctx p = {k_block, rows, cols, X, ldx, dY, lddy, rstd, dgamma};
        parallel_for(nthreads, cols, rms_param_range, &p);
    }
    return 0;
}

/*
 * SiLU and the SiLU-gated unit of Llama's feed-forward (op sequences):
 *   silu(x) = x / (1 + exp_rep(-x));  swiglu(g, u) = RN(silu(g) * u);
 *   backward: s = 1 / (1 + exp_rep(-g)); silu'(g) = fma(g*s, 1 - s, s)
 *     (= s + g s (1 - s));  dgate = RN(RN(dy * u) * silu'(g));
 *     dup = RN(dy * silu(g)) with silu(g) recomputed as in the forward.
 */
float repops_ref_silu1(float x)
{
    const float w = -x;
    const float d = 1.0f + repops_ref_exp1(w);
    return x / d;
}

float repops_ref_silu_grad1(float x)
{
    const float w = -x;
    const float d = 1.0f + repops_ref_exp1(w);
    const float s = 1.0f / d;
    const float om = 1.0f - s;
    const float xs = x * s;
    return fmaf(xs, om, s);
}

typedef struct {
    const float *g, *u, *dy;
    float *y, *dg, *du;
} sw_ctx;

static void silu_range(void *vctx, int64_t i0, int64_t i1)
{
    const sw_ctx *c = (const sw_ctx *)vctx;
    for (int64_t i = i0; i < i1; ++i) c->y[i] = repops_ref_silu1(c->g[i]);
}

static void swiglu_range(void *vctx, int64_t i0, int64_t i1)
{
    const sw_ctx *c = (const sw_ctx *)vctx;
    for (int64_t i = i0; i < i1; ++i) c->y[i] = repops_ref_silu1(c->g[i]) * c->u[i];
}

static void swiglu_bwd_range(void *vctx, int64_t i0, int64_t i1)
{
    const sw_ctx *c = (const sw_ctx *)vctx;
    for (int64_t i = i0; i < i1; ++i) {
        const float gi = c->g[i], ui = c->u[i], dyi = c->dy[i];
        const float dyu = dyi * ui;
        const float dgv = dyu * repops_ref_silu_grad1(gi);
        const float duv = dyi * repops_ref_silu1(gi);
        c->dg[i] = dgv;
        c->du[i] = duv;
    }
}

int repops_ref_silu(int64_t n, const float *x, float *y, int nthreads)
{
    if (n < 0) return -1;
    sw_ctx c = {x, NULL, NULL, y, NULL, NULL};
    parallel_for(nthreads, n, silu_range, &c);
    return 0;
}

int repops_ref_swiglu(int64_t n, const float *g, const float *u, float *y, int nthreads)
{
    if (n < 0) return -1;
    sw_ctx c = {g, u, NULL, y, NULL, NULL};
    parallel_for(nthreads, n, swiglu_range, &c);
    return 0;
}

int repops_ref_swiglu_backward(int64_t n, const float *g, const float *u, const float *dy,
                               float *dg, float *du, int nthreads)
{
    if (n < 0) return -1;
    sw_ctx c = {g, u, dy, NULL, dg, du};
    parallel_for(nthreads, n, swiglu_bwd_range, &c);
    return 0;
}

/*
 * erf and the erf-form ("exact") GELU, x * Phi(x) with Phi the standard normal
 * distribution function, as DistilBERT's activation (Section 4.2; Section 3.1
 * lists the math functions RepOps rebuilds).  Reading (op sequence):
 *   small arguments |z| < 0.5: erf(z) = z * S(z*z), S by Horner with fma over
 *     RN(2/sqrt(pi) (-1)^n / (n! (2n+1))), n = 0..7;
 *   otherwise erfc(z) = exp(-z^2) R(z), R(z) = exp(z^2) erfc(z) on
 *     [0.5, 2.5]: degree-12 polynomial in s = z - 1.5 (exact),
 *     [2.5, 10.5]: degree-8 polynomial in s = (1/(1 + z) - 3/16) * 9.5;
 *     each the binary32-rounded monomial coefficients of the polynomial that
 *     interpolates R at the Chebyshev points cos(pi (2k+1) / (2(d+1))) of s;
 *     erfc(z) = 0 for z >= 10.5;
 *   exp(-c x^2) (c = 1 or 1/2) without rounding x^2: h = x with the low 12
 *     bits of its significand cleared (h*h is exact), d = (x - h) * (x + h),
 *     exp(-c x^2) = exp_rep(-(h h) c) * exp_rep(-d c);
 *   erf(x) = sign(x) (1 - erfc(|x|)) for |x| >= 0.5;
 *   Phi(x): z = |x| * RN(1/sqrt 2); z < 0.5: fma(0.5, erf(x * RN(1/sqrt 2)), 0.5);
 *     else q = RN(exp(-x^2/2) R(z)) * 0.5 (0 for z >= 10.5) and
 *     Phi = 1 - q for x > 0, q otherwise (no cancellation in the lower tail);
 *   gelu(x) = x * Phi(x);  gelu'(x) = fma(x, exp(-x^2/2) * RN(1/sqrt(2 pi)), Phi(x)).
 */
static const float ERF_SMALL[8] = {
    0x1.20dd76p+0f, -0x1.812746p-2f, 0x1.ce2f22p-4f, -0x1.b82ce4p-6f,
    0x1.565bcep-8f, -0x1.c02db4p-11f, 0x1.f9a326p-14f, -0x1.f4d25cp-17f};
static const float ERFC_P1[13] = {
    0x1.494db0p-2f, -0x1.4f1988p-3f, 0x1.37ea26p-4f, -0x1.0dc542p-5f, 0x1.b6596ep-7f,
    -0x1.5135c2p-8f, 0x1.ee6646p-10f, -0x1.5c00ccp-11f, 0x1.d5624ap-13f, -0x1.243bd4p-14f,
    0x1.71a8d4p-16f, -0x1.364e28p-17f, 0x1.6a86acp-19f};
static const float ERFC_P2[9] = {
    0x1.040c3ap-3f, 0x1.565eecp-4f, 0x1.c46bacp-8f, -0x1.24aa48p-13f, -0x1.44b7dap-14f,
    0x1.7d0926p-19f, 0x1.82a7a8p-20f, -0x1.1ebc20p-23f, -0x1.dd0088p-26f};
static const float ERF_INV_SQRT2 = 0x1.6a09e6p-1f;
static const float ERF_INV_SQRT_2PI = 0x1.988454p-2f;

static float erf_small(float z)
{
    const float u = z * z;
    float p = ERF_SMALL[7];
    for (int n = 6; n >= 0; --n) p = fmaf(p, u, ERF_SMALL[n]);
    return z * p;
}

static float clear_low12(float x)
{
    uint32_t b;
    memcpy(&b, &x, 4);
    b &= 0xFFFFF000u;
    float h;
    memcpy(&h, &b, 4);
    return h;
}

static float exp_neg_sq(float x, float c)
{
    const float h = clear_low12(x);
    const float hh = h * h;
    const float a = -(hh * c);
    const float dl = x - h;
    const float ds = x + h;
    const float d = dl * ds;
    const float b = -(d * c);
    return repops_ref_exp1(a) * repops_ref_exp1(b);
}

static float erfc_scaled(float z)
{
    if (z < 2.5f) {
        const float s = z - 1.5f;
        float p = ERFC_P1[12];
        for (int j = 11; j >= 0; --j) p = fmaf(p, s, ERFC_P1[j]);
        return p;
    }
    const float t = 1.0f / (1.0f + z);
    const float s = (t - 0.1875f) * 9.5f;
    float p = ERFC_P2[8];
    for (int j = 7; j >= 0; --j) p = fmaf(p, s, ERFC_P2[j]);
    return p;
}

float repops_ref_erf1(float x)
{
    if (isnan(x)) return x;
    const float a = fabsf(x);
    if (a < 0.5f) return erf_small(x);
    const float q = (a >= 10.5f) ? 0.0f : exp_neg_sq(a, 1.0f) * erfc_scaled(a);
    const float r = 1.0f - q;
    return x < 0.0f ? -r : r;
}

static float normal_cdf(float x)
{
    const float a = fabsf(x);
    const float z = a * ERF_INV_SQRT2;
    if (z < 0.5f) {
        const float xs = x * ERF_INV_SQRT2;
        return fmaf(0.5f, erf_small(xs), 0.5f);
    }
    float q = 0.0f;
    if (!(z >= 10.5f)) {
        const float er = exp_neg_sq(a, 0.5f) * erfc_scaled(z);
        q = er * 0.5f;
    }
    return x > 0.0f ? 1.0f - q : q;
}

float repops_ref_gelu_erf1(float x)
{
    if (isnan(x)) return x;
    return x * normal_cdf(x);
}

float repops_ref_gelu_erf_grad1(float x)
{
    if (isnan(x)) return x;
    const float a = fabsf(x);
    const float e = exp_neg_sq(a, 0.5f);
    const float phi = e * ERF_INV_SQRT_2PI;
    return fmaf(x, phi, normal_cdf(x));
}

typedef struct {
    const float *x, *dy;
    float *y;
    int which; /* 0 erf, 1 gelu, 2 gelu backward */
} erf_ctx;

static void erf_range(void *vctx, int64_t i0, int64_t i1)
{
    const erf_ctx *c = (const erf_ctx *)vctx;
    for (int64_t i = i0; i < i1; ++i) {
        const float x = c->x[i];
        if (c->which == 0) c->y[i] = repops_ref_erf1(x);
        else if (c->which == 1) c->y[i] = repops_ref_gelu_erf1(x);
        else c->y[i] = c->dy[i] * repops_ref_gelu_erf_grad1(x);
    }
}

int repops_ref_erf(int64_t n, const float *x, float *y, int nthreads)
{
    if (n < 0) return -1;
    erf_ctx c = {x, NULL, y, 0};
    parallel_for(nthreads, n, erf_range, &c);
    return 0;
}

int repops_ref_gelu_erf(int64_t n, const float *x, float *y, int nthreads)
{
    if (n < 0) return -1;
    erf_ctx c = {x, NULL, y, 1};
    parallel_for(nthreads, n, erf_range, &c);
    return 0;
}

int repops_ref_gelu_erf_backward(int64_t n, const float *x, const float *dy, float *dx,
                                 int nthreads)
{
    if (n < 0) return -1;
    erf_ctx c = {x, dy, dx, 2};
    parallel_for(nthreads, n, erf_range, &c);
    return 0;
}

/* ========================================================================= */
/* Tensor commitments: SHA-256 and a Merkle tree over chunks                  */
/* ========================================================================= */

/*
 * The protocol commits to checkpoints and to the tensors entering and leaving
 * each graph node with a collision-resistant hash such as SHA-256 (Sections
 * 2.1 and 2.2), and combines node hashes with a binary Merkle tree (Section
 * 2.2, checkpoint hash format).  Reading for a tensor: its bytes as stored
 * (row-major, little-endian binary32) are cut into chunks of C bytes (the last
 * one shorter); the commitment is the Merkle Tree Hash of RFC 6962 over the
 * chunks:  MTH({}) = SHA-256(empty);  MTH({d}) = SHA-256(0x00 || d);
 * MTH(D[0:n]) = SHA-256(0x01 || MTH(D[0:k]) || MTH(D[k:n])) with k the largest
 * power of two below n.  SHA-256 is FIPS 180-4 (Section 6.2), written out
 * below from the standard.
 */
static const uint32_t SHA_K[64] = {
    0x428a2f98u, 0x71374491u, 0xb5c0fbcfu, 0xe9b5dba5u, 0x3956c25bu, 0x59f111f1u, 0x923f82a4u,
    0xab1c5ed5u, 0xd807aa98u, 0x12835b01u, 0x243185beu, 0x550c7dc3u, 0x72be5d74u, 0x80deb1feu,
    0x9bdc06a7u, 0xc19bf174u, 0xe49b69c1u, 0xefbe4786u, 0x0fc19dc6u, 0x240ca1ccu, 0x2de92c6fu,
    0x4a7484aau, 0x5cb0a9dcu, 0x76f988dau, 0x983e5152u, 0xa831c66du, 0xb00327c8u, 0xbf597fc7u,
    0xc6e00bf3u, 0xd5a79147u, 0x06ca6351u, 0x14292967u, 0x27b70a85u, 0x2e1b2138u, 0x4d2c6dfcu,
    0x53380d13u, 0x650a7354u, 0x766a0abbu, 0x81c2c92eu, 0x92722c85u, 0xa2bfe8a1u, 0xa81a664bu,
    0xc24b8b70u, 0xc76c51a3u, 0xd192e819u, 0xd6990624u, 0xf40e3585u, 0x106aa070u, 0x19a4c116u,
    0x1e376c08u, 0x2748774cu, 0x34b0bcb5u, 0x391c0cb3u, 0x4ed8aa4au, 0x5b9cca4fu, 0x682e6ff3u,
    0x748f82eeu, 0x78a5636fu, 0x84c87814u, 0x8cc70208u, 0x90befffau, 0xa4506cebu, 0xbef9a3f7u,
    0xc67178f2u};
static const uint32_t SHA_H0[8] = {0x6a09e667u, 0xbb67ae85u, 0x3c6ef372u, 0xa54ff53au,
                                   0x510e527fu, 0x9b05688cu, 0x1f83d9abu, 0x5be0cd19u};

static uint32_t rotr32(uint32_t x, int n) { return (x >> n) | (x << (32 - n)); }

/* One application of the compression function to a 64-byte block. */
static void sha_block(uint32_t H[8], const uint8_t blk[64])
{
    uint32_t W[64];
    for (int t = 0; t < 16; ++t)
        W[t] = ((uint32_t)blk[4 * t] << 24) | ((uint32_t)blk[4 * t + 1] << 16) |
               ((uint32_t)blk[4 * t + 2] << 8) | (uint32_t)blk[4 * t + 3];
    for (int t = 16; t < 64; ++t) {
        const uint32_t s0 = rotr32(W[t - 15], 7) ^ rotr32(W[t - 15], 18) ^ (W[t - 15] >> 3);
        const uint32_t s1 = rotr32(W[t - 2], 17) ^ rotr32(W[t - 2], 19) ^ (W[t - 2] >> 10);
        W[t] = W[t - 16] + s0 + W[t - 7] + s1;
    }
    uint32_t a = H[0], b = H[1], c = H[2], d = H[3], e = H[4], f = H[5], g = H[6], h = H[7];
    for (int t = 0; t < 64; ++t) {
        const uint32_t S1 = rotr32(e, 6) ^ rotr32(e, 11) ^ rotr32(e, 25);
        const uint32_t ch = (e & f) ^ (~e & g);
        const uint32_t T1 = h + S1 + ch + SHA_K[t] + W[t];
        const uint32_t S0 = rotr32(a, 2) ^ rotr32(a, 13) ^ rotr32(a, 22);
        const uint32_t maj = (a & b) ^ (a & c) ^ (b & c);
        const uint32_t T2 = S0 + maj;
        h = g; g = f; f = e; e = d + T1;
        d = c; c = b; b = a; a = T1 + T2;
    }
    H[0] += a; H[1] += b; H[2] += c; H[3] += d;
    H[4] += e; H[5] += f; H[6] += g; H[7] += h;
}

/* SHA-256 of (prefix byte if has_prefix) || msg[0..len). */
static void sha256_prefixed(int has_prefix, uint8_t prefix, const uint8_t *msg, uint64_t len,
                            uint8_t out[32])
{
    uint32_t H[8];
    memcpy(H, SHA_H0, sizeof H);
    const uint64_t total = len + (has_prefix ? 1 : 0);
    uint8_t blk[64];
    uint64_t pos = 0; /* bytes of the whole message consumed */
    int fill = 0;
    if (has_prefix) blk[fill++] = prefix;
    for (uint64_t i = 0; i < len; ++i) {
        blk[fill++] = msg[i];
        if (fill == 64) { sha_block(H, blk); fill = 0; }
    }
    pos = total;
    blk[fill++] = 0x80; /* padding: one bit, zeros, 64-bit big-endian bit length */
    if (fill > 56) {
        while (fill < 64) blk[fill++] = 0;
        sha_block(H, blk);
        fill = 0;
    }
    while (fill < 56) blk[fill++] = 0;
    const uint64_t bits = pos * 8;
    for (int i = 0; i < 8; ++i) blk[56 + i] = (uint8_t)(bits >> (56 - 8 * i));
    sha_block(H, blk);
    for (int i = 0; i < 8; ++i) {
        out[4 * i] = (uint8_t)(H[i] >> 24);
        out[4 * i + 1] = (uint8_t)(H[i] >> 16);
        out[4 * i + 2] = (uint8_t)(H[i] >> 8);
        out[4 * i + 3] = (uint8_t)H[i];
    }
}

void repops_ref_sha256(const void *msg, uint64_t len, uint8_t out[32])
{
    sha256_prefixed(0, 0, (const uint8_t *)msg, len, out);
}

/* MTH over the chunks [first, first + count) of data. */
static void mth_range(const uint8_t *data, uint64_t nbytes, uint64_t chunk, uint64_t first,
                      uint64_t count, uint8_t out[32])
{
    if (count == 1) {
        const uint64_t off = first * chunk;
        const uint64_t len = (off + chunk <= nbytes) ? chunk : nbytes - off;
        sha256_prefixed(1, 0x00, data + off, len, out);
        return;
    }
    uint64_t k = 1;
    while (k * 2 < count) k *= 2; /* largest power of two below count */
    uint8_t node[64];
    mth_range(data, nbytes, chunk, first, k, node);
    mth_range(data, nbytes, chunk, first + k, count - k, node + 32);
    sha256_prefixed(1, 0x01, node, 64, out);
}

int repops_ref_commit(const void *data, uint64_t nbytes, uint64_t chunk_bytes, uint8_t out[32])
{
    if (chunk_bytes == 0) return -1;
    if (nbytes == 0) {
        sha256_prefixed(0, 0, NULL, 0, out);
        return 0;
    }
    const uint64_t leaves = (nbytes + chunk_bytes - 1) / chunk_bytes;
    mth_range((const uint8_t *)data, nbytes, chunk_bytes, 0, leaves, out);
    return 0;
}

/* ========================================================================= */
/* Training-step operators                                                   */
/* ========================================================================= */

/*
 * The training runs of Section 4.2 (with the Adam optimizer) execute the
 * extended graph of Section 2.2: forward nodes, their backward nodes and the
 * optimizer update.  The backward operators below are the usual derivatives
 * of the forward operators above; the paper fixes no operation order for
 * them, so each reading is stated with its definition.
 */

/*
 * Softmax backward: dx = y * (dy - <y, dy>) row by row.  Reading: the inner
 * product is the fixed-order row sum of fma(y_j, dy_j, .) over the unmasked
 * columns; dx_j = y_j * (dy_j - s); masked columns get +0.
 */
typedef struct {
    int W, combine;
    int64_t cols;
    const float *Y; int64_t ldy;
    const float *dY; int64_t lddy;
    float *dX; int64_t lddx;
    int64_t period;
} smb_ctx;

static void softmax_bwd_range(void *vctx, int64_t r0, int64_t r1)
{
    const smb_ctx *c = (const smb_ctx *)vctx;
    for (int64_t r = r0; r < r1; ++r) {
        const float *y = c->Y + r * c->ldy;
        const float *dy = c->dY + r * c->lddy;
        float *dx = c->dX + r * c->lddx;
        const int64_t valid = (c->period > 0) ? (r % c->period) + 1 : c->cols;
        const int64_t nv = valid < c->cols ? valid : c->cols;
        const float s = rowsum_terms(c->W, c->combine, c->cols, nv, y, dy, 2);
        for (int64_t j = 0; j < c->cols; ++j) {
            if (j < nv) {
                const float diff = dy[j] - s;
                dx[j] = y[j] * diff;
            } else {
                dx[j] = 0.0f;
            }
        }
    }
}

int repops_ref_softmax_backward_rows(int row_width, int row_combine, int64_t rows, int64_t cols,
                                     const float *Y, int64_t ldy, const float *dY, int64_t lddy,
                                     float *dX, int64_t lddx, int64_t causal_period, int nthreads)
{
    if (check_order_rows(row_width, row_combine) || rows < 0 || cols < 0 || causal_period < 0)
        return -1;
    smb_ctx c = {row_width, row_combine, cols, Y, ldy, dY, lddy, dX, lddx, causal_period};
    parallel_for(nthreads, rows, softmax_bwd_range, &c);
    return 0;
}

/*
 * LayerNorm backward (input gradient), with the forward's saved mean and
 * rstd: t_j = (x_j - mean) * rstd exactly as in the forward; g_j = dy_j *
 * gamma_j (dy_j when gamma is absent); a = rowsum(g) / n; b = rowsum of
 * fma(g, t, .) / n; dx_j = rstd * ((g_j - a) - t_j * b).
 */
typedef struct {
    int W, combine;
    int64_t cols;
    const float *X; int64_t ldx;
    const float *dY; int64_t lddy;
    const float *mean, *rstd, *gamma;
    float *dX; int64_t lddx;
} lnb_ctx;

static void ln_bwd_range(void *vctx, int64_t r0, int64_t r1)
{
    const lnb_ctx *c = (const lnb_ctx *)vctx;
    const size_t n = (size_t)(c->cols > 0 ? c->cols : 1);
    float *t = (float *)malloc(sizeof(float) * n);
    float *g = (float *)malloc(sizeof(float) * n);
    if (!t || !g) abort();
    const float nf = (float)c->cols;
    for (int64_t r = r0; r < r1; ++r) {
        const float *x = c->X + r * c->ldx;
        const float *dy = c->dY + r * c->lddy;
        float *dx = c->dX + r * c->lddx;
        const float mean = c->mean[r], rstd = c->rstd[r];
        for (int64_t j = 0; j < c->cols; ++j) {
            const float d = x[j] - mean;
            t[j] = d * rstd;
            g[j] = c->gamma ? dy[j] * c->gamma[j] : dy[j];
        }
        const float a = rowsum_terms(c->W, c->combine, c->cols, c->cols, g, NULL, 0) / nf;
        const float b = rowsum_terms(c->W, c->combine, c->cols, c->cols, g, t, 2) / nf;
        for (int64_t j = 0; j < c->cols; ++j) {
            const float u = g[j] - a;
            const float tb = t[j] * b;
            const float w = u - tb;
            dx[j] = rstd * w;
        }
    }
    free(t);
    free(g);
}

/*
 * LayerNorm parameter gradients: dgamma_j = sum over rows i of dy_ij * t_ij,
 * dbeta_j = sum over rows of dy_ij.  Reading: the row index is a contraction
 * index, so the canonical blocked left-to-right rule of the matrix product
 * applies with the same block length (k_block): fused terms fma(dy, t, P) for
 * dgamma, plain additions for dbeta.
 */
typedef struct {
    int64_t k_block;
    int64_t rows, cols;
    const float *X; int64_t ldx;
    const float *dY; int64_t lddy;
    const float *mean, *rstd;
    float *dgamma, *dbeta;
} lnp_ctx;

static void ln_param_range(void *vctx, int64_t j0, int64_t j1)
{
    const lnp_ctx *c = (const lnp_ctx *)vctx;
    const int64_t blk = c->k_block > 0 ? c->k_block : c->rows;
    for (int64_t j = j0; j < j1; ++j) {
        float accg = 0.0f, accb = 0.0f;
        for (int64_t i0 = 0; i0 < c->rows; i0 += blk) {
            const int64_t i1 = (i0 + blk < c->rows) ? i0 + blk : c->rows;
            float pg = 0.0f, pb = 0.0f;
            for (int64_t i = i0; i < i1; ++i) {
                const float dy = c->dY[i * c->lddy + j];
                const float d = c->X[i * c->ldx + j] - c->mean[i];
                const float t = d * c->rstd[i];
                pg = fmaf(dy, t, pg);
                pb = pb + dy;
            }
            accg = accg + pg;
            accb = accb + pb;
        }
        if (c->dgamma) c->dgamma[j] = accg;
        if (c->dbeta) c->dbeta[j] = accb;
    }
}

int repops_ref_layernorm_backward_rows(int row_width, int row_combine, int64_t k_block,
                                       int64_t rows, int64_t cols,
                                       const float *X, int64_t ldx, const float *dY, int64_t lddy,
                                       const float *mean, const float *rstd, const float *gamma,
                                       float *dX, int64_t lddx, float *dgamma, float *dbeta,
                                       int nthreads)
{
    if (check_order_rows(row_width, row_combine) || k_block < 0 || rows < 0 || cols < 0)
        return -1;
    if (rows > 0 && cols == 0) return -1;
    if (dX) {
        lnb_ctx c = {row_width, row_combine, cols, X, ldx, dY, lddy, mean, rstd, gamma, dX, lddx};
        parallel_for(nthreads, rows, ln_bwd_range, &c);
    }
    if (dgamma || dbeta) {
        lnp_ctx p = {k_block, rows, cols, X, ldx, dY, lddy, mean, rstd, dgamma, dbeta};
        parallel_for(nthreads, cols, ln_param_range, &p);
    }
    return 0;
}

/*
 * Bias gradient of a linear layer: db_j = sum over rows i of dY_ij.  Reading:
 * the row index is a contraction index (the product ones^T dY), so the
 * contraction rule applies with block length k_block: per column, chains
 * P = P + dY_ij over blocks of rows from +0, block partials added left to
 * right.  Rows = 0 gives +0.
 */
typedef struct {
    int64_t k_block, rows;
    const float *X; int64_t ldx;
    float *out;
} colsum_ctx;

static void colsum_range(void *vctx, int64_t j0, int64_t j1)
{
    const colsum_ctx *c = (const colsum_ctx *)vctx;
    const int64_t blk = c->k_block > 0 ? c->k_block : c->rows;
    for (int64_t j = j0; j < j1; ++j) {
        float acc = 0.0f;
        for (int64_t i0 = 0; i0 < c->rows; i0 += blk) {
            const int64_t i1 = (i0 + blk < c->rows) ? i0 + blk : c->rows;
            float p = 0.0f;
            for (int64_t i = i0; i < i1; ++i) p = p + c->X[i * c->ldx + j];
            acc = acc + p;
        }
        c->out[j] = acc;
    }
}

int repops_ref_colsum_rows(int64_t k_block, int64_t rows, int64_t cols, const float *X,
                           int64_t ldx, float *out, int nthreads)
{
    if (k_block < 0 || rows < 0 || cols < 0) return -1;
    colsum_ctx c = {k_block, rows, X, ldx, out};
    parallel_for(nthreads, cols, colsum_range, &c);
    return 0;
}

/*
 * GELU backward (tanh form): with s = 1 / (1 + exp_rep(-2z)) the forward is
 * x * s, so d/dx = s + x s (1 - s) * 2 sqrt(2/pi) (1 + 3 * 0.044715 x^2).
 * Reading (op sequence): u = x*x; z = fma(c, u*x, x) * sq; e = exp_rep(-2z);
 * s = 1 / (1 + e); om = 1 - s; v = fma(c3, u, 1); t2 = (x*s)*om;
 * t3 = sq2 * v; dx = dy * fma(t2, t3, s).  Constants: c = RN(0.044715),
 * c3 = RN(0.134145) (= 3 * 0.044715), sq = RN(sqrt(2/pi)), sq2 = 2 * sq.
 */
static const float GELU_C3 = 0x1.12ba9ep-3f;
static const float GELU_SQ2 = 0x1.988454p+0f;

float repops_ref_gelu_grad1(float x)
{
    const float u = x * x;
    const float u3 = u * x;
    float z = fmaf(GELU_C, u3, x);
    z = z * GELU_SQ;
    const float w = z * -2.0f;
    const float e = repops_ref_exp1(w);
    const float d = 1.0f + e;
    const float s = 1.0f / d;
    const float om = 1.0f - s;
    const float v = fmaf(GELU_C3, u, 1.0f);
    const float t1 = x * s;
    const float t2 = t1 * om;
    const float t3 = GELU_SQ2 * v;
    return fmaf(t2, t3, s);
}

typedef struct {
    const float *x, *dy;
    float *dx;
} gb_ctx;

static void gelu_bwd_range(void *vctx, int64_t i0, int64_t i1)
{
    const gb_ctx *c = (const gb_ctx *)vctx;
    for (int64_t i = i0; i < i1; ++i) c->dx[i] = c->dy[i] * repops_ref_gelu_grad1(c->x[i]);
}

int repops_ref_gelu_backward(int64_t n, const float *x, const float *dy, float *dx, int nthreads)
{
    if (n < 0) return -1;
    gb_ctx c = {x, dy, dx};
    parallel_for(nthreads, n, gelu_bwd_range, &c);
    return 0;
}

/*
 * Adam / AdamW step (Kingma and Ba; decoupled weight decay of Loshchilov and
 * Hutter), the optimizer of the training runs in Section 4.2.  Reading (op
 * sequence):
 *   scalars, in binary64 from the binary32 arguments, each rounded once to
 *   binary32 at the end (1 - b^t loses most of its bits to cancellation in
 *   binary32 when b is close to 1 and t is small):
 *     pw = b^t by binary exponentiation (result *= base for each set bit of t
 *     from the lowest, base *= base after each bit); c1 = 1 - b1; c2 = 1 - b2;
 *     step = lr / (1 - b1^t); sbc2 = sqrt(1 - b2^t); dec = 1 - lr * wd.
 *   per element, binary32: decoupled: p = p * dec (when wd != 0); coupled:
 *     g = fma(wd, p, g); m = fma(b1, m, c1 * g); v = fma(b2, v, c2 * (g * g));
 *     den = sqrt(v) / sbc2 + eps; p = p - step * (m / den).
 */
typedef struct {
    float c1, c2, step, sbc2, dec, eps, wd;
    float b1, b2;
    int decoupled;
} adam_scalars;

static double pow_binary(double base, int64_t t)
{
    double result = 1.0;
    while (t > 0) {
        if (t & 1) result = result * base;
        base = base * base;
        t >>= 1;
    }
    return result;
}

static adam_scalars adam_prepare(float lr, float b1, float b2, float eps, float wd, int64_t t,
                                 int decoupled)
{
    adam_scalars s;
    const double dlr = lr, db1 = b1, db2 = b2, dwd = wd;
    s.b1 = b1;
    s.b2 = b2;
    s.c1 = (float)(1.0 - db1);
    s.c2 = (float)(1.0 - db2);
    const double bc1 = 1.0 - pow_binary(db1, t);
    const double bc2 = 1.0 - pow_binary(db2, t);
    s.step = (float)(dlr / bc1);
    s.sbc2 = (float)sqrt(bc2);
    const double lw = dlr * dwd;
    s.dec = (float)(1.0 - lw);
    s.eps = eps;
    s.wd = wd;
    s.decoupled = decoupled;
    return s;
}

typedef struct {
    adam_scalars s;
    float *p, *m, *v;
    const float *g;
} adam_ctx;

static void adam_range(void *vctx, int64_t i0, int64_t i1)
{
    const adam_ctx *c = (const adam_ctx *)vctx;
    const adam_scalars s = c->s;
    for (int64_t i = i0; i < i1; ++i) {
        float p = c->p[i], g = c->g[i];
        if (s.wd != 0.0f) {
            if (s.decoupled) p = p * s.dec;
            else g = fmaf(s.wd, p, g);
        }
        const float cg = s.c1 * g;
        const float m = fmaf(s.b1, c->m[i], cg);
        const float gg = g * g;
        const float cgg = s.c2 * gg;
        const float v = fmaf(s.b2, c->v[i], cgg);
        const float rv = sqrtf(v);
        const float q = rv / s.sbc2;
        const float den = q + s.eps;
        const float upd = m / den;
        const float su = s.step * upd;
        c->p[i] = p - su;
        c->m[i] = m;
        c->v[i] = v;
    }
}

int repops_ref_adam_step(int64_t n, float *param, const float *grad, float *exp_avg,
                         float *exp_avg_sq, float lr, float beta1, float beta2, float eps,
                         float weight_decay, int64_t step, int decoupled, int nthreads)
{
    if (n < 0 || step < 1) return -1;
    adam_ctx c;
    fenv_t saved;
    fegetenv(&saved);
    install_ieee_env();
    c.s = adam_prepare(lr, beta1, beta2, eps, weight_decay, step, decoupled);
    fesetenv(&saved);
    c.p = param;
    c.m = exp_avg;
    c.v = exp_avg_sq;
    c.g = grad;
    parallel_for(nthreads, n, adam_range, &c);
    return 0;
}

/* The step-dependent scalars, exported for the pins. */
int repops_ref_adam_scalars(float lr, float beta1, float beta2, float weight_decay, int64_t step,
                            float *out6)
{
    if (step < 1) return -1;
    fenv_t saved;
    fegetenv(&saved);
    install_ieee_env();
    const adam_scalars s = adam_prepare(lr, beta1, beta2, 0.0f, weight_decay, step, 1);
    fesetenv(&saved);
    out6[0] = s.c1;
    out6[1] = s.c2;
    out6[2] = s.step;
    out6[3] = s.sbc2;
    out6[4] = s.dec;
    out6[5] = (float)pow_binary(beta1, step);
    return 0;
}
