// C ABI of librepops: argument validation, order-descriptor checks and launch
// selection.  Every error is detected before anything is enqueued.
#include <hip/hip_runtime_api.h>
#include <math.h>
#include <stdint.h>
#include <string.h>

#include "../../include/repops.h"
#include "repops_internal.h"
#include "train_internal.h"
#include "llama_internal.h"
#include "commit_internal.h"
#include "rows_internal.h"

using repops::AdamScalars;
using repops::GemmArgs;
using repops::LnParamArgs;
using repops::RowArgs;
using repops::RowBwdArgs;

namespace {

constexpr int64_t kMaxDim = (int64_t(1) << 31) - 1;

bool order_valid(const repops_order_t* o) {
  if (!o) return false;
  if (o->version != 1) return false;
  if (o->k_inner != REPOPS_K_FMA && o->k_inner != REPOPS_K_MUL_ADD) return false;
  if (o->k_combine != REPOPS_COMBINE_LTR) return false;
  const uint32_t w = o->row_width;
  if (w < 1 || w > 1024 || (w & (w - 1)) != 0) return false;
  if (o->row_combine != REPOPS_ROW_STRIDED_TREE && o->row_combine != REPOPS_ROW_BLOCKED_LTR)
    return false;
  if (o->reserved[0] != 0 || o->reserved[1] != 0) return false;
  return true;
}

bool launch_params_zero_from(const repops_launch_t* l, int first) {
  for (int i = first; i < 7; ++i)
    if (l->p[i] != 0) return false;
  return true;
}

// Byte range [lo, hi) touched by a strided operand: `rows` rows of `cols`
// elements, leading dimension ld, replicated over two batch strides.
struct Extent {
  uintptr_t lo, hi;
};

Extent extent_of(const float* p, int64_t b0, int64_t s0, int64_t b1, int64_t s1, int64_t rows,
                 int64_t cols, int64_t ld) {
  int64_t lo = 0, hi = 0;  // element offsets, hi inclusive
  auto span = [&](int64_t count, int64_t stride) {
    if (count <= 1) return;
    const int64_t d = (count - 1) * stride;
    if (d < 0) lo += d; else hi += d;
  };
  span(b0, s0);
  span(b1, s1);
  span(rows, ld);
  hi += cols - 1;
  const uintptr_t base = reinterpret_cast<uintptr_t>(p);
  return {base + static_cast<uintptr_t>(lo * 4), base + static_cast<uintptr_t>((hi + 1) * 4)};
}

bool overlaps(Extent a, Extent b) { return a.lo < b.hi && b.lo < a.hi; }

// True when no two elements of a [b0][b1][rows][cols] array with element
// strides (s0, s1, ld, 1) share an address: taking the dimensions of more than
// one element in increasing order of |stride|, each must step past the span of
// the ones before it.  A sufficient condition (every permutation of a dense
// array passes); an output that fails it would have two batch elements write
// one address in an unspecified order.
bool elements_disjoint(int64_t b0, int64_t s0, int64_t b1, int64_t s1, int64_t rows, int64_t ld,
                       int64_t cols) {
  struct Dim {
    uint64_t size, stride;
  };
  auto mag = [](int64_t s) { return s < 0 ? 0 - static_cast<uint64_t>(s) : static_cast<uint64_t>(s); };
  Dim d[4] = {{static_cast<uint64_t>(cols), 1},
              {static_cast<uint64_t>(rows), mag(ld)},
              {static_cast<uint64_t>(b1), mag(s1)},
              {static_cast<uint64_t>(b0), mag(s0)}};
  for (int i = 1; i < 4; ++i)
    for (int j = i; j > 0 && d[j].stride < d[j - 1].stride; --j) {
      const Dim t = d[j];
      d[j] = d[j - 1];
      d[j - 1] = t;
    }
  unsigned __int128 span = 0;  // offsets the dimensions taken so far reach
  for (const Dim& x : d) {
    if (x.size <= 1) continue;
    if (x.stride <= span) return false;
    span += static_cast<unsigned __int128>(x.size - 1) * x.stride;
  }
  return true;
}

repops_status_t hip_status(hipError_t e) { return e == hipSuccess ? REPOPS_OK : REPOPS_ERR_HIP; }

repops_status_t run_gemm(const repops_order_t* order, GemmArgs& g, const repops_launch_t* launch,
                         hipStream_t stream) {
  if (!order_valid(order)) return REPOPS_ERR_ORDER;
  g.k_block = order->k_block;
  g.fused = order->k_inner == REPOPS_K_FMA ? 1 : 0;

  uint32_t kind = launch ? launch->kind : REPOPS_LAUNCH_AUTO;
  uint32_t index = 0;
  if (launch) {
    if (kind == REPOPS_LAUNCH_AUTO || kind == REPOPS_LAUNCH_GEMM_SIMPLE) {
      if (!launch_params_zero_from(launch, 0)) return REPOPS_ERR_LAUNCH;
    } else if (kind == REPOPS_LAUNCH_GEMM_TILED || kind == REPOPS_LAUNCH_GEMM_MFMA) {
      if (!launch_params_zero_from(launch, 1)) return REPOPS_ERR_LAUNCH;
      index = launch->p[0];
    } else {
      return REPOPS_ERR_LAUNCH;
    }
  }
  auto tiled_ok = [&](const repops::GemmConfig* c) {
    return c && (g.k_block == 0 || g.k_block % c->bk == 0);
  };
  auto mfma_ok = [&](const repops::GemmConfig* c) {
    return c && g.fused && (g.k_block == 0 || g.k_block % c->bk == 0);
  };
  if (kind == REPOPS_LAUNCH_AUTO) {
    // Matrix cores for the fused order (their single-term updates are the fma
    // chain), the large tile for big outputs; vector tiles for the unfused
    // order; the simple path for block lengths no tile divides.
    const int64_t outputs = g.m * g.n * g.batch0 * g.batch1;
    int mfma_pref = 0;                                  // 128 x 128 tiles, 8 waves, ring
    if (outputs <= (int64_t(1) << 20)) {
      mfma_pref = 5;                                    // small outputs: 64 x 64 tiles
    } else if (g.k <= 256) {
      // short k: the persistent ring form where each compute unit takes at
      // least four tiles in turn, else register-staged slices
      int cus = 0;
      const int64_t ring = repops::gemm_mfma_ring_tiles(g, 9, &cus);
      mfma_pref = cus > 0 && ring >= 4 * static_cast<int64_t>(cus) ? 9 : 2;
    } else if (g.causal == 2) {
      mfma_pref = 8;                                    // causal A: 64-row tiles
    }
    if (!mfma_ok(repops::gemm_mfma_config(mfma_pref))) mfma_pref = 0;
    const int tiled_pref = outputs >= (int64_t(1) << 22) ? 1 : 0;
    if (mfma_ok(repops::gemm_mfma_config(mfma_pref))) {
      kind = REPOPS_LAUNCH_GEMM_MFMA;
      index = mfma_pref;
    } else if (tiled_ok(repops::gemm_tiled_config(tiled_pref))) {
      kind = REPOPS_LAUNCH_GEMM_TILED;
      index = tiled_pref;
    } else if (tiled_ok(repops::gemm_tiled_config(0))) {
      kind = REPOPS_LAUNCH_GEMM_TILED;
      index = 0;
    } else {
      kind = REPOPS_LAUNCH_GEMM_SIMPLE;
    }
  }
  if (kind == REPOPS_LAUNCH_GEMM_SIMPLE) return hip_status(repops::launch_gemm_simple(g, stream));
  if (kind == REPOPS_LAUNCH_GEMM_TILED) {
    if (!tiled_ok(repops::gemm_tiled_config(static_cast<int>(index)))) return REPOPS_ERR_LAUNCH;
    return hip_status(repops::launch_gemm_tiled(g, static_cast<int>(index), stream));
  }
  // matrix-core path
  if (!mfma_ok(repops::gemm_mfma_config(static_cast<int>(index)))) return REPOPS_ERR_LAUNCH;
  return hip_status(repops::launch_gemm_mfma(g, static_cast<int>(index), stream));
}

repops_status_t check_operands(const GemmArgs& g) {
  if (g.batch0 < 0 || g.batch1 < 0 || g.m < 0 || g.n < 0 || g.k < 0) return REPOPS_ERR_SHAPE;
  if (g.batch0 > kMaxDim || g.batch1 > kMaxDim || g.m > kMaxDim || g.n > kMaxDim ||
      g.k > kMaxDim)
    return REPOPS_ERR_SHAPE;
  if (g.k_block < 0) return REPOPS_ERR_ORDER;
  if (g.ta != 0 && g.ta != 1) return REPOPS_ERR_SHAPE;
  if (g.tb != 0 && g.tb != 1) return REPOPS_ERR_SHAPE;
  const bool empty = g.batch0 == 0 || g.batch1 == 0 || g.m == 0 || g.n == 0;
  if (empty) return REPOPS_OK;
  if (!g.C) return REPOPS_ERR_NULL;
  if (g.k > 0 && (!g.A || !g.B)) return REPOPS_ERR_NULL;
  if (g.ldc < g.n || g.ldc < 1) return REPOPS_ERR_STRIDE;
  if (!elements_disjoint(g.batch0, g.sc0, g.batch1, g.sc1, g.m, g.ldc, g.n))
    return REPOPS_ERR_STRIDE;
  if (g.k > 0) {
    if (g.lda < (g.ta ? g.m : g.k)) return REPOPS_ERR_STRIDE;
    if (g.ldb < (g.tb ? g.k : g.n)) return REPOPS_ERR_STRIDE;
  }
  const Extent ce = extent_of(g.C, g.batch0, g.sc0, g.batch1, g.sc1, g.m, g.n, g.ldc);
  if (g.k > 0) {
    const Extent ae = g.ta ? extent_of(g.A, g.batch0, g.sa0, g.batch1, g.sa1, g.k, g.m, g.lda)
                           : extent_of(g.A, g.batch0, g.sa0, g.batch1, g.sa1, g.m, g.k, g.lda);
    const Extent be = g.tb ? extent_of(g.B, g.batch0, g.sb0, g.batch1, g.sb1, g.n, g.k, g.ldb)
                           : extent_of(g.B, g.batch0, g.sb0, g.batch1, g.sb1, g.k, g.n, g.ldb);
    if (overlaps(ce, ae) || overlaps(ce, be)) return REPOPS_ERR_ALIAS;
  }
  if (g.bias) {
    const Extent bi = extent_of(g.bias, 1, 0, 1, 0, 1, g.n, g.n);
    if (overlaps(ce, bi)) return REPOPS_ERR_ALIAS;
  }
  return REPOPS_OK;
}

// The GELU backward's forward input of a product (gelu_in): a [m x n] array
// with its own leading dimension that the output may not touch; no bias.
repops_status_t check_gelu_in(const GemmArgs& g) {
  if (!g.gelu_in || g.m == 0 || g.n == 0) return REPOPS_OK;
  if (g.bias) return REPOPS_ERR_VALUE;
  if (g.ld_gelu_in < g.n) return REPOPS_ERR_STRIDE;
  if (overlaps(extent_of(g.C, 1, 0, 1, 0, g.m, g.n, g.ldc),
               extent_of(g.gelu_in, 1, 0, 1, 0, g.m, g.n, g.ld_gelu_in)))
    return REPOPS_ERR_ALIAS;
  return REPOPS_OK;
}

// Rows: Y may equal X exactly (same base, same leading dimension); any other
// overlap is rejected.
repops_status_t check_rows(int64_t rows, int64_t cols, const float* X, int64_t ldx, const float* Y,
                           int64_t ldy, bool* empty) {
  if (rows < 0 || cols < 0 || rows > kMaxDim || cols > kMaxDim) return REPOPS_ERR_SHAPE;
  *empty = rows == 0 || cols == 0;
  if (*empty) return REPOPS_OK;
  if (!X || !Y) return REPOPS_ERR_NULL;
  if (ldx < cols || ldy < cols) return REPOPS_ERR_STRIDE;
  const Extent xe = extent_of(X, 1, 0, 1, 0, rows, cols, ldx);
  const Extent ye = extent_of(Y, 1, 0, 1, 0, rows, cols, ldy);
  if (X == Y && ldx == ldy) return REPOPS_OK;
  if (overlaps(xe, ye)) return REPOPS_ERR_ALIAS;
  return REPOPS_OK;
}

// ROWS_WAVE: p[0] = rows per block (1, 2, 4, 8); p[1] = waves per row: 0 or 1
// for one, or 2, 4, 8 for one row per block split over that many waves (needs
// p[0] = 1 and an operation with a split kernel: `split_max` non-null, giving
// the widest row it takes for a split).  *split receives the waves per row.
repops_status_t row_launch_kind(const repops_order_t* order, const repops_launch_t* launch,
                                int64_t cols, uint32_t* kind, int* wpb,
                                int64_t wave_max = repops::rows_wave_max_cols(),
                                int* split = nullptr, int64_t (*split_max)(int) = nullptr,
                                int auto_per_lane = 16, int64_t auto_wave_cols = 1024) {
  const bool wave_order =
      order->row_width == 64 && order->row_combine == REPOPS_ROW_STRIDED_TREE;
  const bool wave_fits = cols <= wave_max;
  *wpb = 4;
  if (split) *split = 1;
  if (!launch || launch->kind == REPOPS_LAUNCH_AUTO) {
    if (launch && !launch_params_zero_from(launch, 0)) return REPOPS_ERR_LAUNCH;
    *kind = (wave_order && wave_fits) ? REPOPS_LAUNCH_ROWS_WAVE : REPOPS_LAUNCH_ROWS_GENERIC;
    if (wave_order && split && split_max) {
      const int S = repops::auto_row_split(cols, auto_per_lane, auto_wave_cols);
      if (S > 1 && cols <= split_max(S)) {
        *kind = REPOPS_LAUNCH_ROWS_WAVE;
        *wpb = 1;
        *split = S;
      }
    }
    return REPOPS_OK;
  }
  if (launch->kind == REPOPS_LAUNCH_ROWS_GENERIC) {
    if (!launch_params_zero_from(launch, 0)) return REPOPS_ERR_LAUNCH;
    *kind = REPOPS_LAUNCH_ROWS_GENERIC;
    return REPOPS_OK;
  }
  if (launch->kind == REPOPS_LAUNCH_ROWS_WAVE) {
    const uint32_t w = launch->p[0], S = launch->p[1];
    if (!(w == 1 || w == 2 || w == 4 || w == 8) || !launch_params_zero_from(launch, 2))
      return REPOPS_ERR_LAUNCH;
    if (!wave_order) return REPOPS_ERR_LAUNCH;
    if (S <= 1) {
      if (!wave_fits) return REPOPS_ERR_LAUNCH;
    } else {
      if (!(S == 2 || S == 4 || S == 8) || w != 1 || !split || !split_max ||
          cols > split_max(static_cast<int>(S)))
        return REPOPS_ERR_LAUNCH;
      *split = static_cast<int>(S);
    }
    *kind = REPOPS_LAUNCH_ROWS_WAVE;
    *wpb = static_cast<int>(w);
    return REPOPS_OK;
  }
  return REPOPS_ERR_LAUNCH;
}

repops_status_t ew_launch(const repops_launch_t* launch, int* threads, int* max_blocks) {
  *threads = 256;
  *max_blocks = 0;
  if (!launch || launch->kind == REPOPS_LAUNCH_AUTO) {
    if (launch && !launch_params_zero_from(launch, 0)) return REPOPS_ERR_LAUNCH;
    return REPOPS_OK;
  }
  if (launch->kind != REPOPS_LAUNCH_ELEMENTWISE) return REPOPS_ERR_LAUNCH;
  const uint32_t t = launch->p[0];
  if (t == 0 || t > 1024 || t % 64 != 0 || !launch_params_zero_from(launch, 2))
    return REPOPS_ERR_LAUNCH;
  if (launch->p[1] > (1u << 30)) return REPOPS_ERR_LAUNCH;
  *threads = static_cast<int>(t);
  *max_blocks = static_cast<int>(launch->p[1]);
  return REPOPS_OK;
}

repops_status_t check_elementwise(const repops_order_t* order, int64_t n, const float* X,
                                  const float* Y) {
  if (!order_valid(order)) return REPOPS_ERR_ORDER;
  if (n < 0 || n > kMaxDim) return REPOPS_ERR_SHAPE;
  if (n == 0) return REPOPS_OK;
  if (!X || !Y) return REPOPS_ERR_NULL;
  if (X != Y) {
    const Extent xe = extent_of(X, 1, 0, 1, 0, 1, n, n), ye = extent_of(Y, 1, 0, 1, 0, 1, n, n);
    if (overlaps(xe, ye)) return REPOPS_ERR_ALIAS;
  }
  return REPOPS_OK;
}

// A rows x cols operand: null, stride and size checks.
repops_status_t check_matrix(const float* p, int64_t rows, int64_t cols, int64_t ld) {
  if (!p) return REPOPS_ERR_NULL;
  if (ld < cols || ld < 1) return REPOPS_ERR_STRIDE;
  (void)rows;
  return REPOPS_OK;
}

// Output `out` may coincide exactly with `in` (same base and leading
// dimension); any other overlap is an alias error.
bool bad_overlap(const float* out, int64_t ldo, Extent oe, const float* in, int64_t ldi, Extent ie) {
  if (out == in && ldo == ldi) return false;
  return overlaps(oe, ie);
}

Extent vec_extent(const void* p, int64_t n_floats) {
  return extent_of(static_cast<const float*>(p), 1, 0, 1, 0, 1, n_floats, n_floats);
}

// Adam step scalars, in binary64 from the binary32 arguments and rounded once
// to binary32 (1 - b^t cancels in binary32 when b is near 1 and t is small).
// b^t by binary exponentiation: the result is multiplied by the running power
// for each set bit of t from the lowest, and the power squared after each bit.
double pow_by_bits(double base, int64_t t) {
  double result = 1.0;
  while (t > 0) {
    if (t & 1) result = result * base;
    base = base * base;
    t >>= 1;
  }
  return result;
}

AdamScalars adam_scalars(float lr, float b1, float b2, float eps, float wd, int64_t t,
                         int decoupled) {
  AdamScalars s{};
  const double dlr = lr, db1 = b1, db2 = b2, dwd = wd;
  s.c1 = static_cast<float>(1.0 - db1);
  s.c2 = static_cast<float>(1.0 - db2);
  const double bc1 = 1.0 - pow_by_bits(db1, t);
  const double bc2 = 1.0 - pow_by_bits(db2, t);
  s.step = static_cast<float>(dlr / bc1);
  s.sbc2 = static_cast<float>(sqrt(bc2));
  const double lw = dlr * dwd;
  s.dec = static_cast<float>(1.0 - lw);
  s.eps = eps;
  s.wd = wd;
  s.b1 = b1;
  s.b2 = b2;
  s.decay = wd != 0.0f ? (decoupled ? 1 : 2) : 0;
  return s;
}

}  // namespace

extern "C" {

void repops_order_default(repops_order_t* order) {
  if (!order) return;
  memset(order, 0, sizeof(*order));
  order->version = 1;
  order->k_block = 64;
  order->k_inner = REPOPS_K_FMA;
  order->k_combine = REPOPS_COMBINE_LTR;
  order->row_width = 64;
  order->row_combine = REPOPS_ROW_STRIDED_TREE;
}

const char* repops_status_str(repops_status_t s) {
  switch (s) {
    case REPOPS_OK: return "ok";
    case REPOPS_ERR_NULL: return "null pointer";
    case REPOPS_ERR_SHAPE: return "invalid shape";
    case REPOPS_ERR_STRIDE: return "invalid stride";
    case REPOPS_ERR_ALIAS: return "output overlaps an input";
    case REPOPS_ERR_ORDER: return "unsupported order descriptor";
    case REPOPS_ERR_LAUNCH: return "invalid launch configuration";
    case REPOPS_ERR_HIP: return "HIP launch failed";
    case REPOPS_ERR_VALUE: return "invalid scalar argument";
    case REPOPS_ERR_WORKSPACE: return "workspace missing or too small";
    case REPOPS_ERR_SCRATCH:
      return "problem needs more scratch than the no-allocation entry point's fixed buffer holds";
    default: return "unknown status";
  }
}

uint32_t repops_abi_version(void) { return REPOPS_ABI_VERSION; }

int32_t repops_gemm_config_count(uint32_t kind) {
  if (kind == REPOPS_LAUNCH_GEMM_TILED) return repops::gemm_tiled_count();
  if (kind == REPOPS_LAUNCH_GEMM_MFMA) return repops::gemm_mfma_count();
  return 0;
}

const char* repops_gemm_config_name(uint32_t kind, uint32_t index) {
  const repops::GemmConfig* c = nullptr;
  if (kind == REPOPS_LAUNCH_GEMM_TILED) c = repops::gemm_tiled_config(static_cast<int>(index));
  if (kind == REPOPS_LAUNCH_GEMM_MFMA) c = repops::gemm_mfma_config(static_cast<int>(index));
  return c ? c->name : nullptr;
}

repops_status_t repops_matmul(const repops_order_t* order, int64_t m, int64_t n, int64_t k,
                              const float* A, int64_t lda, int32_t trans_a, const float* B,
                              int64_t ldb, int32_t trans_b, const float* bias, float* C,
                              int64_t ldc, const repops_launch_t* launch, void* hip_stream) {
  if (!order_valid(order)) return REPOPS_ERR_ORDER;
  GemmArgs g{};
  g.batch0 = 1; g.batch1 = 1; g.m = m; g.n = n; g.k = k;
  g.A = A; g.lda = lda; g.ta = trans_a;
  g.B = B; g.ldb = ldb; g.tb = trans_b;
  g.C = C; g.ldc = ldc;
  g.bias = bias; g.alpha = 1.0f; g.has_alpha = 0;
  g.k_block = order->k_block;
  const repops_status_t st = check_operands(g);
  if (st != REPOPS_OK) return st;
  if (m == 0 || n == 0) return REPOPS_OK;
  return run_gemm(order, g, launch, static_cast<hipStream_t>(hip_stream));
}

repops_status_t repops_matmul_gelu(const repops_order_t* order, int64_t m, int64_t n, int64_t k,
                                   const float* A, int64_t lda, int32_t trans_a, const float* B,
                                   int64_t ldb, int32_t trans_b, const float* bias, float* H,
                                   int64_t ldh, float* G, int64_t ldg,
                                   const repops_launch_t* launch, void* hip_stream) {
  if (!order_valid(order)) return REPOPS_ERR_ORDER;
  GemmArgs g{};
  g.batch0 = 1; g.batch1 = 1; g.m = m; g.n = n; g.k = k;
  g.A = A; g.lda = lda; g.ta = trans_a;
  g.B = B; g.ldb = ldb; g.tb = trans_b;
  g.C = H; g.ldc = ldh;
  g.G = G; g.ldg = ldg;
  g.bias = bias; g.alpha = 1.0f; g.has_alpha = 0;
  g.k_block = order->k_block;
  const repops_status_t st = check_operands(g);
  if (st != REPOPS_OK) return st;
  if (m == 0 || n == 0) return REPOPS_OK;
  if (!G) return REPOPS_ERR_NULL;
  if (ldg < n) return REPOPS_ERR_STRIDE;
  // G is written beside H by the same threads: it may touch no operand and
  // not H.
  const Extent ge = extent_of(G, 1, 0, 1, 0, m, n, ldg);
  if (overlaps(ge, extent_of(H, 1, 0, 1, 0, m, n, ldh))) return REPOPS_ERR_ALIAS;
  if (k > 0) {
    const Extent ae = trans_a ? extent_of(A, 1, 0, 1, 0, k, m, lda) : extent_of(A, 1, 0, 1, 0, m, k, lda);
    const Extent be = trans_b ? extent_of(B, 1, 0, 1, 0, n, k, ldb) : extent_of(B, 1, 0, 1, 0, k, n, ldb);
    if (overlaps(ge, ae) || overlaps(ge, be)) return REPOPS_ERR_ALIAS;
  }
  if (bias && overlaps(ge, extent_of(bias, 1, 0, 1, 0, 1, n, n))) return REPOPS_ERR_ALIAS;
  return run_gemm(order, g, launch, static_cast<hipStream_t>(hip_stream));
}

repops_status_t repops_matmul_gelu_backward(const repops_order_t* order, int64_t m, int64_t n,
                                            int64_t k, const float* A, int64_t lda,
                                            int32_t trans_a, const float* B, int64_t ldb,
                                            int32_t trans_b, const float* X, int64_t ldx,
                                            float* C, int64_t ldc, const repops_launch_t* launch,
                                            void* hip_stream) {
  if (!order_valid(order)) return REPOPS_ERR_ORDER;
  GemmArgs g{};
  g.batch0 = 1; g.batch1 = 1; g.m = m; g.n = n; g.k = k;
  g.A = A; g.lda = lda; g.ta = trans_a;
  g.B = B; g.ldb = ldb; g.tb = trans_b;
  g.C = C; g.ldc = ldc;
  g.gelu_in = X; g.ld_gelu_in = ldx;
  g.alpha = 1.0f; g.has_alpha = 0;
  g.k_block = order->k_block;
  repops_status_t st = check_operands(g);
  if (st != REPOPS_OK) return st;
  if (m == 0 || n == 0) return REPOPS_OK;
  if (!X) return REPOPS_ERR_NULL;
  st = check_gelu_in(g);
  if (st != REPOPS_OK) return st;
  return run_gemm(order, g, launch, static_cast<hipStream_t>(hip_stream));
}

repops_status_t repops_matmul_grouped(const repops_order_t* order, int32_t count,
                                      const repops_gemm_desc_t* descs,
                                      const repops_launch_t* launch, void* hip_stream) {
  static_assert(REPOPS_MAX_GROUP == repops::kMaxGroup, "one group size");
  if (!order_valid(order)) return REPOPS_ERR_ORDER;
  if (count < 0 || count > REPOPS_MAX_GROUP) return REPOPS_ERR_SHAPE;
  if (count == 0) return REPOPS_OK;
  if (!descs) return REPOPS_ERR_NULL;
  if (launch && (launch->kind != REPOPS_LAUNCH_AUTO || !launch_params_zero_from(launch, 0)))
    return REPOPS_ERR_LAUNCH;
  GemmArgs g[REPOPS_MAX_GROUP];
  bool live[REPOPS_MAX_GROUP];
  for (int p = 0; p < count; ++p) {
    const repops_gemm_desc_t& d = descs[p];
    g[p] = GemmArgs{};
    g[p].batch0 = 1; g[p].batch1 = 1; g[p].m = d.m; g[p].n = d.n; g[p].k = d.k;
    g[p].A = d.A; g[p].lda = d.lda; g[p].ta = d.trans_a;
    g[p].B = d.B; g[p].ldb = d.ldb; g[p].tb = d.trans_b;
    g[p].C = d.C; g[p].ldc = d.ldc;
    g[p].bias = d.bias; g[p].alpha = 1.0f; g[p].has_alpha = 0;
    g[p].gelu_in = d.gelu_in; g[p].ld_gelu_in = d.ld_gelu_in;
    g[p].k_block = order->k_block;
    g[p].fused = order->k_inner == REPOPS_K_FMA ? 1 : 0;
    repops_status_t st = check_operands(g[p]);
    if (st == REPOPS_OK) st = check_gelu_in(g[p]);
    if (st != REPOPS_OK) return st;
    live[p] = g[p].m > 0 && g[p].n > 0;
  }
  // The products run concurrently: no output may touch another product's
  // operands or output.
  for (int p = 0; p < count; ++p) {
    if (!live[p]) continue;
    const Extent ce = extent_of(g[p].C, 1, 0, 1, 0, g[p].m, g[p].n, g[p].ldc);
    for (int q = 0; q < count; ++q) {
      if (q == p || !live[q]) continue;
      if (overlaps(ce, extent_of(g[q].C, 1, 0, 1, 0, g[q].m, g[q].n, g[q].ldc)))
        return REPOPS_ERR_ALIAS;
      if (g[q].k > 0) {
        const Extent ae = g[q].ta ? extent_of(g[q].A, 1, 0, 1, 0, g[q].k, g[q].m, g[q].lda)
                                  : extent_of(g[q].A, 1, 0, 1, 0, g[q].m, g[q].k, g[q].lda);
        const Extent be = g[q].tb ? extent_of(g[q].B, 1, 0, 1, 0, g[q].n, g[q].k, g[q].ldb)
                                  : extent_of(g[q].B, 1, 0, 1, 0, g[q].k, g[q].n, g[q].ldb);
        if (overlaps(ce, ae) || overlaps(ce, be)) return REPOPS_ERR_ALIAS;
      }
      if (g[q].bias && overlaps(ce, extent_of(g[q].bias, 1, 0, 1, 0, 1, g[q].n, g[q].n)))
        return REPOPS_ERR_ALIAS;
      if (g[q].gelu_in &&
          overlaps(ce, extent_of(g[q].gelu_in, 1, 0, 1, 0, g[q].m, g[q].n, g[q].ld_gelu_in)))
        return REPOPS_ERR_ALIAS;
    }
  }
  hipStream_t s = static_cast<hipStream_t>(hip_stream);
  bool one = order->k_inner == REPOPS_K_FMA && (order->k_block == 0 || order->k_block % 16 == 0);
  int n_live = 0;
  for (int p = 0; p < count; ++p) {
    if (!live[p]) continue;
    ++n_live;
    one = one && g[p].k > 0 && repops::gemm_mfma_staged_ok(g[p], 0);
  }
  if (n_live == 0) return REPOPS_OK;
  if (!one) {
    for (int p = 0; p < count; ++p) {
      if (!live[p]) continue;
      const repops_status_t st = run_gemm(order, g[p], nullptr, s);
      if (st != REPOPS_OK) return st;
    }
    return REPOPS_OK;
  }
  // One launch: the products with the longest contraction first, so that
  // their tiles start first and the short ones fill the compute units behind
  // them.
  int idx[REPOPS_MAX_GROUP], n = 0;
  for (int p = 0; p < count; ++p)
    if (live[p]) idx[n++] = p;
  for (int a = 1; a < n; ++a)
    for (int b = a; b > 0 && g[idx[b]].k > g[idx[b - 1]].k; --b) {
      const int t = idx[b]; idx[b] = idx[b - 1]; idx[b - 1] = t;
    }
  int bm, bn;
  repops::gemm_mfma_tile(0, &bm, &bn);
  repops::GroupArgs ga{};
  ga.count = n;
  ga.first[0] = 0;
  for (int i = 0; i < n; ++i) {
    ga.g[i] = g[idx[i]];
    ga.tiles_m[i] = (ga.g[i].m + bm - 1) / bm;
    ga.tiles_n[i] = (ga.g[i].n + bn - 1) / bn;
    ga.first[i + 1] = ga.first[i] + ga.tiles_m[i] * ga.tiles_n[i];
  }
  if (ga.first[n] > kMaxDim) return REPOPS_ERR_SHAPE;
  return hip_status(repops::launch_gemm_mfma_grouped(ga, s));
}

repops_status_t repops_bmm(const repops_order_t* order, int64_t batch0, int64_t batch1, int64_t m,
                           int64_t n, int64_t k, const float* A, int64_t sa0, int64_t sa1,
                           int64_t lda, int32_t trans_a, const float* B, int64_t sb0, int64_t sb1,
                           int64_t ldb, int32_t trans_b, float alpha, float* C, int64_t sc0,
                           int64_t sc1, int64_t ldc, const repops_launch_t* launch,
                           void* hip_stream) {
  if (!order_valid(order)) return REPOPS_ERR_ORDER;
  GemmArgs g{};
  g.batch0 = batch0; g.batch1 = batch1; g.m = m; g.n = n; g.k = k;
  g.A = A; g.sa0 = sa0; g.sa1 = sa1; g.lda = lda; g.ta = trans_a;
  g.B = B; g.sb0 = sb0; g.sb1 = sb1; g.ldb = ldb; g.tb = trans_b;
  g.C = C; g.sc0 = sc0; g.sc1 = sc1; g.ldc = ldc;
  g.bias = nullptr; g.alpha = alpha; g.has_alpha = 1;
  g.k_block = order->k_block;
  const repops_status_t st = check_operands(g);
  if (st != REPOPS_OK) return st;
  if (batch0 == 0 || batch1 == 0 || m == 0 || n == 0) return REPOPS_OK;
  return run_gemm(order, g, launch, static_cast<hipStream_t>(hip_stream));
}

repops_status_t repops_bmm_causal(const repops_order_t* order, int64_t batch0, int64_t batch1,
                                  int64_t m, int64_t n, int64_t k, const float* A, int64_t sa0,
                                  int64_t sa1, int64_t lda, int32_t trans_a, const float* B,
                                  int64_t sb0, int64_t sb1, int64_t ldb, int32_t trans_b,
                                  float alpha, float* C, int64_t sc0, int64_t sc1, int64_t ldc,
                                  int32_t mask, const repops_launch_t* launch, void* hip_stream) {
  if (!order_valid(order)) return REPOPS_ERR_ORDER;
  if (mask != REPOPS_CAUSAL_OUTPUT && mask != REPOPS_CAUSAL_A) return REPOPS_ERR_VALUE;
  GemmArgs g{};
  g.batch0 = batch0; g.batch1 = batch1; g.m = m; g.n = n; g.k = k;
  g.A = A; g.sa0 = sa0; g.sa1 = sa1; g.lda = lda; g.ta = trans_a;
  g.B = B; g.sb0 = sb0; g.sb1 = sb1; g.ldb = ldb; g.tb = trans_b;
  g.C = C; g.sc0 = sc0; g.sc1 = sc1; g.ldc = ldc;
  g.bias = nullptr; g.alpha = alpha; g.has_alpha = 1;
  g.k_block = order->k_block;
  g.causal = mask;
  const repops_status_t st = check_operands(g);
  if (st != REPOPS_OK) return st;
  if (batch0 == 0 || batch1 == 0 || m == 0 || n == 0) return REPOPS_OK;
  return run_gemm(order, g, launch, static_cast<hipStream_t>(hip_stream));
}

repops_status_t repops_softmax_rows(const repops_order_t* order, int64_t rows, int64_t cols,
                                    const float* X, int64_t ldx, float* Y, int64_t ldy,
                                    int64_t causal_period, const repops_launch_t* launch,
                                    void* hip_stream) {
  if (!order_valid(order)) return REPOPS_ERR_ORDER;
  if (causal_period < 0) return REPOPS_ERR_SHAPE;
  bool empty = false;
  repops_status_t st = check_rows(rows, cols, X, ldx, Y, ldy, &empty);
  if (st != REPOPS_OK) return st;
  uint32_t kind;
  int wpb, split;
  // One wave per row measured faster up to 2048 columns here (split rows
  // beyond).
  st = row_launch_kind(order, launch, cols, &kind, &wpb, repops::rows_wave_max_cols(), &split,
                       repops::rows_split_max_cols, 16, 2048);
  if (st != REPOPS_OK || empty) return st;
  RowArgs a{};
  a.rows = rows; a.cols = cols; a.X = X; a.ldx = ldx; a.Y = Y; a.ldy = ldy;
  a.W = static_cast<int>(order->row_width);
  a.blocked = order->row_combine == REPOPS_ROW_BLOCKED_LTR;
  a.period = causal_period;
  hipStream_t s = static_cast<hipStream_t>(hip_stream);
  if (kind == REPOPS_LAUNCH_ROWS_WAVE && split > 1)
    return hip_status(repops::launch_softmax_split(a, split, s));
  if (kind == REPOPS_LAUNCH_ROWS_WAVE) return hip_status(repops::launch_softmax_wave(a, wpb, s));
  return hip_status(repops::launch_softmax_generic(a, s));
}

repops_status_t repops_layernorm_rows(const repops_order_t* order, int64_t rows, int64_t cols,
                                      const float* X, int64_t ldx, const float* gamma,
                                      const float* beta, float eps, float* Y, int64_t ldy,
                                      float* mean_out, float* rstd_out,
                                      const repops_launch_t* launch, void* hip_stream) {
  if (!order_valid(order)) return REPOPS_ERR_ORDER;
  if (rows > 0 && cols == 0) return REPOPS_ERR_SHAPE;
  if (cols > (int64_t(1) << 24)) return REPOPS_ERR_SHAPE;  // n must convert to float exactly
  bool empty = false;
  repops_status_t st = check_rows(rows, cols, X, ldx, Y, ldy, &empty);
  if (st != REPOPS_OK) return st;
  uint32_t kind;
  int wpb, split;
  st = row_launch_kind(order, launch, cols, &kind, &wpb, repops::rows_wave_max_cols(), &split,
                       repops::rows_split_max_cols);
  if (st != REPOPS_OK || empty) return st;
  const Extent ye = extent_of(Y, 1, 0, 1, 0, rows, cols, ldy);
  if (gamma && overlaps(ye, extent_of(gamma, 1, 0, 1, 0, 1, cols, cols))) return REPOPS_ERR_ALIAS;
  if (beta && overlaps(ye, extent_of(beta, 1, 0, 1, 0, 1, cols, cols))) return REPOPS_ERR_ALIAS;
  // the row statistics touch no input, not Y and not each other
  const Extent xe = extent_of(X, 1, 0, 1, 0, rows, cols, ldx);
  for (const float* stat : {static_cast<const float*>(mean_out), static_cast<const float*>(rstd_out)}) {
    if (!stat) continue;
    const Extent se = vec_extent(stat, rows);
    if (overlaps(se, ye) || overlaps(se, xe) || (gamma && overlaps(se, vec_extent(gamma, cols))) ||
        (beta && overlaps(se, vec_extent(beta, cols))))
      return REPOPS_ERR_ALIAS;
  }
  if (mean_out && rstd_out && overlaps(vec_extent(mean_out, rows), vec_extent(rstd_out, rows)))
    return REPOPS_ERR_ALIAS;
  RowArgs a{};
  a.rows = rows; a.cols = cols; a.X = X; a.ldx = ldx; a.Y = Y; a.ldy = ldy;
  a.W = static_cast<int>(order->row_width);
  a.blocked = order->row_combine == REPOPS_ROW_BLOCKED_LTR;
  a.gamma = gamma; a.beta = beta; a.eps = eps;
  a.mean_out = mean_out; a.rstd_out = rstd_out;
  hipStream_t s = static_cast<hipStream_t>(hip_stream);
  if (kind == REPOPS_LAUNCH_ROWS_WAVE && split > 1)
    return hip_status(repops::launch_layernorm_split(a, split, s));
  if (kind == REPOPS_LAUNCH_ROWS_WAVE) return hip_status(repops::launch_layernorm_wave(a, wpb, s));
  return hip_status(repops::launch_layernorm_generic(a, s));
}

repops_status_t repops_gelu(const repops_order_t* order, int64_t n, const float* X, float* Y,
                            const repops_launch_t* launch, void* hip_stream) {
  repops_status_t st = check_elementwise(order, n, X, Y);
  if (st != REPOPS_OK) return st;
  int threads, max_blocks;
  st = ew_launch(launch, &threads, &max_blocks);
  if (st != REPOPS_OK || n == 0) return st;
  return hip_status(
      repops::launch_gelu(n, X, Y, threads, max_blocks, static_cast<hipStream_t>(hip_stream)));
}

repops_status_t repops_copy(const repops_order_t* order, int64_t n, const float* X, float* Y,
                            const repops_launch_t* launch, void* hip_stream) {
  repops_status_t st = check_elementwise(order, n, X, Y);
  if (st != REPOPS_OK) return st;
  int threads, max_blocks;
  st = ew_launch(launch, &threads, &max_blocks);
  if (st != REPOPS_OK || n == 0) return st;
  return hip_status(
      repops::launch_copy(n, X, Y, threads, max_blocks, static_cast<hipStream_t>(hip_stream)));
}

repops_status_t repops_exp(const repops_order_t* order, int64_t n, const float* X, float* Y,
                           const repops_launch_t* launch, void* hip_stream) {
  repops_status_t st = check_elementwise(order, n, X, Y);
  if (st != REPOPS_OK) return st;
  int threads, max_blocks;
  st = ew_launch(launch, &threads, &max_blocks);
  if (st != REPOPS_OK || n == 0) return st;
  return hip_status(
      repops::launch_exp(n, X, Y, threads, max_blocks, static_cast<hipStream_t>(hip_stream)));
}

// ---------------------------------------------------------------------------
// Training-step operators
// ---------------------------------------------------------------------------

repops_status_t repops_softmax_backward_rows(const repops_order_t* order, int64_t rows,
                                             int64_t cols, const float* Y, int64_t ldy,
                                             const float* dY, int64_t lddy, float* dX,
                                             int64_t lddx, int64_t causal_period,
                                             const repops_launch_t* launch, void* hip_stream) {
  if (!order_valid(order)) return REPOPS_ERR_ORDER;
  if (causal_period < 0) return REPOPS_ERR_SHAPE;
  if (rows < 0 || cols < 0 || rows > kMaxDim || cols > kMaxDim) return REPOPS_ERR_SHAPE;
  const bool empty = rows == 0 || cols == 0;
  uint32_t kind;
  int wpb;
  int split;
  // One wave per row measured faster up to 4096 columns here.
  repops_status_t st = row_launch_kind(order, launch, cols, &kind, &wpb,
                                       repops::rows_wave_max_cols(), &split,
                                       repops::rows_split_max_cols, 8, 4096);
  if (st != REPOPS_OK || empty) return st;
  if ((st = check_matrix(Y, rows, cols, ldy)) != REPOPS_OK) return st;
  if ((st = check_matrix(dY, rows, cols, lddy)) != REPOPS_OK) return st;
  if ((st = check_matrix(dX, rows, cols, lddx)) != REPOPS_OK) return st;
  const Extent ye = extent_of(Y, 1, 0, 1, 0, rows, cols, ldy);
  const Extent de = extent_of(dY, 1, 0, 1, 0, rows, cols, lddy);
  const Extent xe = extent_of(dX, 1, 0, 1, 0, rows, cols, lddx);
  if (bad_overlap(dX, lddx, xe, Y, ldy, ye) || bad_overlap(dX, lddx, xe, dY, lddy, de))
    return REPOPS_ERR_ALIAS;
  RowBwdArgs a{};
  a.rows = rows; a.cols = cols;
  a.Y = Y; a.ldy = ldy; a.dY = dY; a.lddy = lddy; a.dX = dX; a.lddx = lddx;
  a.W = static_cast<int>(order->row_width);
  a.blocked = order->row_combine == REPOPS_ROW_BLOCKED_LTR;
  a.period = causal_period;
  hipStream_t s = static_cast<hipStream_t>(hip_stream);
  if (kind == REPOPS_LAUNCH_ROWS_WAVE && split > 1)
    return hip_status(repops::launch_softmax_bwd_split(a, split, s));
  if (kind == REPOPS_LAUNCH_ROWS_WAVE) return hip_status(repops::launch_softmax_bwd_wave(a, wpb, s));
  return hip_status(repops::launch_softmax_bwd_generic(a, s));
}

repops_status_t repops_layernorm_backward_workspace(const repops_order_t* order, int64_t rows,
                                                    int64_t cols, uint64_t* bytes) {
  if (!order_valid(order)) return REPOPS_ERR_ORDER;
  if (!bytes) return REPOPS_ERR_NULL;
  if (rows < 0 || cols < 0 || rows > kMaxDim || cols > (int64_t(1) << 24)) return REPOPS_ERR_SHAPE;
  const int64_t nblk = repops::layernorm_param_blocks(rows, order->k_block);
  *bytes = nblk > 1 ? static_cast<uint64_t>(2 * nblk * cols) * sizeof(float) : 0;
  return REPOPS_OK;
}

// LayerNorm and RMSNorm backward (rms: no mean input, no dbeta).
static repops_status_t norm_backward(
    bool rms, const repops_order_t* order, int64_t rows, int64_t cols, const float* X,
    int64_t ldx, const float* dY, int64_t lddy, const float* mean, const float* rstd,
    const float* gamma, float* dX, int64_t lddx, float* dgamma, float* dbeta, void* workspace,
    uint64_t workspace_bytes, const repops_launch_t* launch, void* hip_stream) {
  if (!order_valid(order)) return REPOPS_ERR_ORDER;
  if (rows < 0 || cols < 0 || rows > kMaxDim || cols > (int64_t(1) << 24)) return REPOPS_ERR_SHAPE;
  if (rows > 0 && cols == 0) return REPOPS_ERR_SHAPE;
  uint32_t kind;
  int wpb, split;
  // dX alone: one wave per row measured faster up to 2048 columns.
  repops_status_t st = row_launch_kind(order, launch, cols, &kind, &wpb,
                                       repops::rows_wave_max_cols(), &split,
                                       repops::rows_split_max_cols, 16, 2048);
  if (st != REPOPS_OK) return st;
  const bool want_params = dgamma || dbeta;
  if (cols == 0 || (rows == 0 && !want_params) || (!dX && !want_params)) return REPOPS_OK;
  uint64_t need = 0;
  if ((st = repops_layernorm_backward_workspace(order, rows, cols, &need)) != REPOPS_OK) return st;
  if (!want_params) need = 0;
  if (repops::layernorm_param_grid(rows, cols, order->k_block) > kMaxDim) return REPOPS_ERR_SHAPE;
  if (need > 0 && (!workspace || workspace_bytes < need)) return REPOPS_ERR_WORKSPACE;
  // Inputs and outputs as (extent, base, leading dimension).  No output may
  // overlap another output or an input, except that dX may coincide exactly
  // with X or with dY.
  struct Span {
    Extent e;
    const float* base;
    int64_t ld;
  };
  Span in[5], out[4];
  int nin = 0, nout = 0;
  if (rows > 0) {
    if ((st = check_matrix(X, rows, cols, ldx)) != REPOPS_OK) return st;
    if ((st = check_matrix(dY, rows, cols, lddy)) != REPOPS_OK) return st;
    if ((!rms && !mean) || !rstd) return REPOPS_ERR_NULL;
    in[nin++] = {extent_of(X, 1, 0, 1, 0, rows, cols, ldx), X, ldx};
    in[nin++] = {extent_of(dY, 1, 0, 1, 0, rows, cols, lddy), dY, lddy};
    if (!rms) in[nin++] = {vec_extent(mean, rows), mean, rows};
    in[nin++] = {vec_extent(rstd, rows), rstd, rows};
  }
  if (gamma) in[nin++] = {vec_extent(gamma, cols), gamma, cols};
  if (dX && rows > 0) {
    if ((st = check_matrix(dX, rows, cols, lddx)) != REPOPS_OK) return st;
    out[nout++] = {extent_of(dX, 1, 0, 1, 0, rows, cols, lddx), dX, lddx};
  }
  if (dgamma) out[nout++] = {vec_extent(dgamma, cols), dgamma, cols};
  if (dbeta) out[nout++] = {vec_extent(dbeta, cols), dbeta, cols};
  if (need > 0) {
    const float* w = static_cast<const float*>(workspace);
    const int64_t wn = static_cast<int64_t>(need / sizeof(float));
    out[nout++] = {vec_extent(w, wn), w, wn};
  }
  for (int i = 0; i < nout; ++i) {
    for (int j = i + 1; j < nout; ++j)
      if (overlaps(out[i].e, out[j].e)) return REPOPS_ERR_ALIAS;
    for (int j = 0; j < nin; ++j) {
      const bool is_dx = dX && rows > 0 && i == 0;
      const bool exact = out[i].base == in[j].base && out[i].ld == in[j].ld;
      if (is_dx && j < 2 && exact) continue;  // dX in place of X or dY
      if (overlaps(out[i].e, in[j].e)) return REPOPS_ERR_ALIAS;
    }
  }
  hipStream_t s = static_cast<hipStream_t>(hip_stream);
  LnParamArgs p{};
  p.rows = rows; p.cols = cols; p.k_block = order->k_block;
  p.X = X; p.ldx = ldx; p.dY = dY; p.lddy = lddy; p.mean = mean; p.rstd = rstd;
  p.dgamma = dgamma; p.dbeta = dbeta; p.ws = static_cast<float*>(workspace);
  p.rms = rms ? 1 : 0;
  RowBwdArgs a{};
  a.rows = rows; a.cols = cols;
  a.Y = X; a.ldy = ldx; a.dY = dY; a.lddy = lddy; a.dX = dX; a.lddx = lddx;
  a.W = static_cast<int>(order->row_width);
  a.blocked = order->row_combine == REPOPS_ROW_BLOCKED_LTR;
  a.mean = mean; a.rstd = rstd; a.gamma = gamma;
  a.rms = rms ? 1 : 0;
  // Both gradients on the wave path with row blocks: one fused pass over X
  // and dY (R rows staged per pass: the launch's waves per block, else a
  // choice by size).
  // (A launch that asks for split rows takes the split kernel for dX.)
  const bool explicit_split = launch && launch->kind == REPOPS_LAUNCH_ROWS_WAVE && split > 1;
  if (want_params && dX && rows > 0 && kind == REPOPS_LAUNCH_ROWS_WAVE && order->k_block >= 1 &&
      !explicit_split) {
    const bool explicit_wave = launch && launch->kind == REPOPS_LAUNCH_ROWS_WAVE;
    // Few row blocks: the blocks' rows and columns spread over about 512
    // workgroups (not in place: other workgroups read the rows dX replaces).
    repops::ColsplitPlan pl{};
    if (!explicit_wave && dX != X && dX != dY &&
        repops::layernorm_colsplit_plan(rows, cols, order->k_block, &pl))
      return hip_status(repops::launch_layernorm_bwd_colsplit(a, p, pl, s));
    const int R = repops::layernorm_fused_rows(rows, cols, order->k_block, explicit_wave ? wpb : 0);
    if (R >= 1) return hip_status(repops::launch_layernorm_bwd_fused(a, p, R, s));
  }
  // Otherwise parameter gradients first: they read X and dY, which dX may
  // overwrite.
  if (want_params) {
    if ((st = hip_status(repops::launch_layernorm_param(p, s))) != REPOPS_OK) return st;
  }
  if (!dX || rows == 0) return REPOPS_OK;
  if (kind == REPOPS_LAUNCH_ROWS_WAVE && split > 1)
    return hip_status(repops::launch_layernorm_bwd_split(a, split, s));
  if (kind == REPOPS_LAUNCH_ROWS_WAVE) return hip_status(repops::launch_layernorm_bwd_wave(a, wpb, s));
  return hip_status(repops::launch_layernorm_bwd_generic(a, s));
}

repops_status_t repops_layernorm_backward_rows(
    const repops_order_t* order, int64_t rows, int64_t cols, const float* X, int64_t ldx,
    const float* dY, int64_t lddy, const float* mean, const float* rstd, const float* gamma,
    float* dX, int64_t lddx, float* dgamma, float* dbeta, void* workspace,
    uint64_t workspace_bytes, const repops_launch_t* launch, void* hip_stream) {
  return norm_backward(false, order, rows, cols, X, ldx, dY, lddy, mean, rstd, gamma, dX, lddx,
                       dgamma, dbeta, workspace, workspace_bytes, launch, hip_stream);
}

repops_status_t repops_layernorm_backward_rows_noalloc(
    const repops_order_t* order, int64_t rows, int64_t cols, const float* X, int64_t ldx,
    const float* dY, int64_t lddy, const float* mean, const float* rstd, const float* gamma,
    float* dX, int64_t lddx, float* dgamma, float* dbeta, const repops_launch_t* launch,
    void* hip_stream) {
  static_assert(REPOPS_NOALLOC_SCRATCH_BYTES == repops::kNoallocScratchBytes,
                "the header states the scratch size");
  uint64_t need = 0;
  repops_status_t st = repops_layernorm_backward_workspace(order, rows, cols, &need);
  if (st != REPOPS_OK) return st;
  if (!dgamma && !dbeta) need = 0;
  if (need > repops::kNoallocScratchBytes) return REPOPS_ERR_SCRATCH;
  void* ws = nullptr;
  if (need > 0 && repops::noalloc_scratch(&ws) != hipSuccess) return REPOPS_ERR_HIP;
  return norm_backward(false, order, rows, cols, X, ldx, dY, lddy, mean, rstd, gamma, dX, lddx,
                       dgamma, dbeta, ws, need, launch, hip_stream);
}

repops_status_t repops_rmsnorm_backward_workspace(const repops_order_t* order, int64_t rows,
                                                  int64_t cols, uint64_t* bytes) {
  return repops_layernorm_backward_workspace(order, rows, cols, bytes);
}

repops_status_t repops_rmsnorm_backward_rows(
    const repops_order_t* order, int64_t rows, int64_t cols, const float* X, int64_t ldx,
    const float* dY, int64_t lddy, const float* rstd, const float* gamma, float* dX,
    int64_t lddx, float* dgamma, void* workspace, uint64_t workspace_bytes,
    const repops_launch_t* launch, void* hip_stream) {
  return norm_backward(true, order, rows, cols, X, ldx, dY, lddy, nullptr, rstd, gamma, dX, lddx,
                       dgamma, nullptr, workspace, workspace_bytes, launch, hip_stream);
}

repops_status_t repops_colsum_rows(const repops_order_t* order, int64_t rows, int64_t cols,
                                   const float* X, int64_t ldx, float* out, void* workspace,
                                   uint64_t workspace_bytes, const repops_launch_t* launch,
                                   void* hip_stream) {
  if (!order_valid(order)) return REPOPS_ERR_ORDER;
  if (rows < 0 || cols < 0 || rows > kMaxDim || cols > (int64_t(1) << 24)) return REPOPS_ERR_SHAPE;
  if (launch && (launch->kind != REPOPS_LAUNCH_AUTO || !launch_params_zero_from(launch, 0)))
    return REPOPS_ERR_LAUNCH;
  if (cols == 0) return REPOPS_OK;
  uint64_t need = 0;
  repops_status_t st = repops_layernorm_backward_workspace(order, rows, cols, &need);
  if (st != REPOPS_OK) return st;
  if (repops::layernorm_param_grid(rows, cols, order->k_block) > kMaxDim) return REPOPS_ERR_SHAPE;
  if (!out) return REPOPS_ERR_NULL;
  if (need > 0 && (!workspace || workspace_bytes < need)) return REPOPS_ERR_WORKSPACE;
  const Extent oe = vec_extent(out, cols);
  if (rows > 0) {
    if ((st = check_matrix(X, rows, cols, ldx)) != REPOPS_OK) return st;
    if (overlaps(oe, extent_of(X, 1, 0, 1, 0, rows, cols, ldx))) return REPOPS_ERR_ALIAS;
  }
  if (need > 0) {
    const Extent we = vec_extent(workspace, static_cast<int64_t>(need / sizeof(float)));
    if (overlaps(we, oe) || (rows > 0 && overlaps(we, extent_of(X, 1, 0, 1, 0, rows, cols, ldx))))
      return REPOPS_ERR_ALIAS;
  }
  LnParamArgs p{};
  p.rows = rows; p.cols = cols; p.k_block = order->k_block;
  p.X = X; p.ldx = ldx; p.dY = X; p.lddy = ldx;
  p.dbeta = out; p.ws = static_cast<float*>(workspace);
  p.sum_only = 1;
  return hip_status(repops::launch_layernorm_param(p, static_cast<hipStream_t>(hip_stream)));
}

repops_status_t repops_gelu_backward(const repops_order_t* order, int64_t n, const float* X,
                                     const float* dY, float* dX, const repops_launch_t* launch,
                                     void* hip_stream) {
  repops_status_t st = check_elementwise(order, n, X, dX);
  if (st != REPOPS_OK) return st;
  if ((st = check_elementwise(order, n, dY, dX)) != REPOPS_OK) return st;
  int threads, max_blocks;
  st = ew_launch(launch, &threads, &max_blocks);
  if (st != REPOPS_OK || n == 0) return st;
  return hip_status(repops::launch_gelu_bwd(n, X, dY, dX, threads, max_blocks,
                                            static_cast<hipStream_t>(hip_stream), false));
}

repops_status_t repops_adam_step(const repops_order_t* order, int64_t n, float* param,
                                 const float* grad, float* exp_avg, float* exp_avg_sq, float lr,
                                 float beta1, float beta2, float eps, float weight_decay,
                                 int64_t step, int32_t decoupled, const repops_launch_t* launch,
                                 void* hip_stream) {
  if (!order_valid(order)) return REPOPS_ERR_ORDER;
  if (n < 0 || n > kMaxDim) return REPOPS_ERR_SHAPE;
  if (step < 1 || (decoupled != 0 && decoupled != 1)) return REPOPS_ERR_VALUE;
  if (!(beta1 >= 0.0f && beta1 < 1.0f) || !(beta2 >= 0.0f && beta2 < 1.0f))
    return REPOPS_ERR_VALUE;
  if (!isfinite(lr) || !isfinite(eps) || !isfinite(weight_decay)) return REPOPS_ERR_VALUE;
  int threads, max_blocks;
  repops_status_t st = ew_launch(launch, &threads, &max_blocks);
  if (st != REPOPS_OK || n == 0) return st;
  if (!param || !grad || !exp_avg || !exp_avg_sq) return REPOPS_ERR_NULL;
  const Extent pe = vec_extent(param, n), ge = vec_extent(grad, n);
  const Extent me = vec_extent(exp_avg, n), ve = vec_extent(exp_avg_sq, n);
  if (overlaps(pe, ge) || overlaps(pe, me) || overlaps(pe, ve) || overlaps(me, ge) ||
      overlaps(me, ve) || overlaps(ve, ge))
    return REPOPS_ERR_ALIAS;
  const AdamScalars sc = adam_scalars(lr, beta1, beta2, eps, weight_decay, step, decoupled);
  return hip_status(repops::launch_adam(n, param, grad, exp_avg, exp_avg_sq, sc, threads,
                                        max_blocks, static_cast<hipStream_t>(hip_stream)));
}

// ---------------------------------------------------------------------------
// Llama-block operators
// ---------------------------------------------------------------------------

repops_status_t repops_sincos(const repops_order_t* order, int64_t n, const float* X, float* S,
                              float* C, const repops_launch_t* launch, void* hip_stream) {
  if (!order_valid(order)) return REPOPS_ERR_ORDER;
  if (n < 0 || n > kMaxDim) return REPOPS_ERR_SHAPE;
  int threads, max_blocks;
  repops_status_t st = ew_launch(launch, &threads, &max_blocks);
  if (st != REPOPS_OK || n == 0) return st;
  if (!X || (!S && !C)) return REPOPS_ERR_NULL;
  const Extent xe = vec_extent(X, n);
  if (S && S != X && overlaps(vec_extent(S, n), xe)) return REPOPS_ERR_ALIAS;
  if (C && C != X && overlaps(vec_extent(C, n), xe)) return REPOPS_ERR_ALIAS;
  if (S && C && overlaps(vec_extent(S, n), vec_extent(C, n))) return REPOPS_ERR_ALIAS;
  if (S == X && C) return REPOPS_ERR_ALIAS;  // the second output would read a written input
  return hip_status(repops::launch_sincos(n, X, S, C, threads, max_blocks,
                                          static_cast<hipStream_t>(hip_stream)));
}

repops_status_t repops_rope(const repops_order_t* order, int64_t rows, int64_t heads,
                            int64_t head_dim, const float* X, int64_t ldx, const float* inv_freq,
                            int64_t position_period, int64_t position_offset, int32_t inverse,
                            float* Y, int64_t ldy, const repops_launch_t* launch,
                            void* hip_stream) {
  if (!order_valid(order)) return REPOPS_ERR_ORDER;
  if (rows < 0 || heads < 0 || head_dim < 0 || rows > kMaxDim || heads > kMaxDim ||
      head_dim > kMaxDim || (head_dim & 1) || position_period < 0 || position_offset < 0)
    return REPOPS_ERR_SHAPE;
  if (inverse != 0 && inverse != 1) return REPOPS_ERR_VALUE;
  const int64_t cols = heads * head_dim;
  if (cols > kMaxDim) return REPOPS_ERR_SHAPE;
  const int64_t last = position_period > 0 ? position_period - 1 : rows - 1;
  if (rows > 0 && last + position_offset >= (int64_t(1) << 24))
    return REPOPS_ERR_SHAPE;  // positions must convert to binary32 exactly
  int wpb = 4;
  if (launch && launch->kind != REPOPS_LAUNCH_AUTO) {
    const uint32_t w = launch->p[0];
    if (launch->kind != REPOPS_LAUNCH_ROWS_WAVE || !(w == 1 || w == 2 || w == 4 || w == 8) ||
        !launch_params_zero_from(launch, 1))
      return REPOPS_ERR_LAUNCH;
    wpb = static_cast<int>(w);
  } else if (launch && !launch_params_zero_from(launch, 0)) {
    return REPOPS_ERR_LAUNCH;
  }
  if (rows == 0 || cols == 0) return REPOPS_OK;
  repops_status_t st;
  if ((st = check_matrix(X, rows, cols, ldx)) != REPOPS_OK) return st;
  if ((st = check_matrix(Y, rows, cols, ldy)) != REPOPS_OK) return st;
  if (!inv_freq) return REPOPS_ERR_NULL;
  const Extent xe = extent_of(X, 1, 0, 1, 0, rows, cols, ldx);
  const Extent ye = extent_of(Y, 1, 0, 1, 0, rows, cols, ldy);
  if (bad_overlap(Y, ldy, ye, X, ldx, xe)) return REPOPS_ERR_ALIAS;
  if (overlaps(ye, vec_extent(inv_freq, head_dim / 2))) return REPOPS_ERR_ALIAS;
  repops::RopeArgs a{};
  a.rows = rows; a.heads = heads; a.head_dim = head_dim;
  a.X = X; a.ldx = ldx; a.inv_freq = inv_freq;
  a.period = position_period; a.offset = position_offset; a.inverse = inverse;
  a.Y = Y; a.ldy = ldy;
  return hip_status(repops::launch_rope(a, wpb, static_cast<hipStream_t>(hip_stream)));
}

repops_status_t repops_rmsnorm_rows(const repops_order_t* order, int64_t rows, int64_t cols,
                                    const float* X, int64_t ldx, const float* gamma, float eps,
                                    float* Y, int64_t ldy, float* rstd_out,
                                    const repops_launch_t* launch, void* hip_stream) {
  if (!order_valid(order)) return REPOPS_ERR_ORDER;
  if (rows > 0 && cols == 0) return REPOPS_ERR_SHAPE;
  if (cols > (int64_t(1) << 24)) return REPOPS_ERR_SHAPE;
  bool empty = false;
  repops_status_t st = check_rows(rows, cols, X, ldx, Y, ldy, &empty);
  if (st != REPOPS_OK) return st;
  uint32_t kind;
  int wpb, split;
  // Split rows with at most 8 values per lane measured fastest here (2048 and
  // 4096 columns).
  st = row_launch_kind(order, launch, cols, &kind, &wpb, repops::rmsnorm_wave_max_cols(), &split,
                       repops::rmsnorm_split_max_cols, 8);
  if (st != REPOPS_OK || empty) return st;
  const Extent ye = extent_of(Y, 1, 0, 1, 0, rows, cols, ldy);
  if (gamma && overlaps(ye, vec_extent(gamma, cols))) return REPOPS_ERR_ALIAS;
  if (rstd_out) {
    const Extent re = vec_extent(rstd_out, rows);
    if (overlaps(re, ye) || overlaps(re, extent_of(X, 1, 0, 1, 0, rows, cols, ldx)) ||
        (gamma && overlaps(re, vec_extent(gamma, cols))))
      return REPOPS_ERR_ALIAS;
  }
  repops::RmsArgs a{};
  a.rows = rows; a.cols = cols; a.X = X; a.ldx = ldx; a.Y = Y; a.ldy = ldy;
  a.W = static_cast<int>(order->row_width);
  a.blocked = order->row_combine == REPOPS_ROW_BLOCKED_LTR;
  a.gamma = gamma; a.eps = eps; a.rstd_out = rstd_out;
  hipStream_t s = static_cast<hipStream_t>(hip_stream);
  if (kind == REPOPS_LAUNCH_ROWS_WAVE && split > 1)
    return hip_status(repops::launch_rmsnorm_split(a, split, s));
  if (kind == REPOPS_LAUNCH_ROWS_WAVE) return hip_status(repops::launch_rmsnorm_wave(a, wpb, s));
  return hip_status(repops::launch_rmsnorm_generic(a, s));
}

repops_status_t repops_silu(const repops_order_t* order, int64_t n, const float* X, float* Y,
                            const repops_launch_t* launch, void* hip_stream) {
  repops_status_t st = check_elementwise(order, n, X, Y);
  if (st != REPOPS_OK) return st;
  int threads, max_blocks;
  st = ew_launch(launch, &threads, &max_blocks);
  if (st != REPOPS_OK || n == 0) return st;
  return hip_status(
      repops::launch_silu(n, X, Y, threads, max_blocks, static_cast<hipStream_t>(hip_stream)));
}

repops_status_t repops_swiglu(const repops_order_t* order, int64_t n, const float* G,
                              const float* Up, float* Y, const repops_launch_t* launch,
                              void* hip_stream) {
  repops_status_t st = check_elementwise(order, n, G, Y);
  if (st != REPOPS_OK) return st;
  if ((st = check_elementwise(order, n, Up, Y)) != REPOPS_OK) return st;
  int threads, max_blocks;
  st = ew_launch(launch, &threads, &max_blocks);
  if (st != REPOPS_OK || n == 0) return st;
  return hip_status(repops::launch_swiglu(n, G, Up, Y, threads, max_blocks,
                                          static_cast<hipStream_t>(hip_stream)));
}

repops_status_t repops_swiglu_backward(const repops_order_t* order, int64_t n, const float* G,
                                       const float* Up, const float* dY, float* dG, float* dUp,
                                       const repops_launch_t* launch, void* hip_stream) {
  if (!order_valid(order)) return REPOPS_ERR_ORDER;
  if (n < 0 || n > kMaxDim) return REPOPS_ERR_SHAPE;
  int threads, max_blocks;
  repops_status_t st = ew_launch(launch, &threads, &max_blocks);
  if (st != REPOPS_OK || n == 0) return st;
  if (!G || !Up || !dY || !dG || !dUp) return REPOPS_ERR_NULL;
  // Outputs may coincide exactly with one input each (element i is read before
  // it is written); partial overlaps and dG/dUp overlapping each other are not
  // allowed.
  const Extent ge = vec_extent(G, n), ue = vec_extent(Up, n), de = vec_extent(dY, n);
  const Extent oge = vec_extent(dG, n), oue = vec_extent(dUp, n);
  if (overlaps(oge, oue)) return REPOPS_ERR_ALIAS;
  const float* ins[3] = {G, Up, dY};
  const Extent ine[3] = {ge, ue, de};
  for (int i = 0; i < 3; ++i) {
    if (dG != ins[i] && overlaps(oge, ine[i])) return REPOPS_ERR_ALIAS;
    if (dUp != ins[i] && overlaps(oue, ine[i])) return REPOPS_ERR_ALIAS;
  }
  return hip_status(repops::launch_swiglu_bwd(n, G, Up, dY, dG, dUp, threads, max_blocks,
                                              static_cast<hipStream_t>(hip_stream)));
}

// ---------------------------------------------------------------------------
// Tensor commitments
// ---------------------------------------------------------------------------

repops_status_t repops_commit_workspace(uint64_t nbytes, uint32_t chunk_bytes, uint64_t* bytes) {
  if (!bytes) return REPOPS_ERR_NULL;
  if (chunk_bytes == 0 || chunk_bytes > (1u << 30)) return REPOPS_ERR_SHAPE;
  if (nbytes > (uint64_t(1) << 46)) return REPOPS_ERR_SHAPE;
  *bytes = repops::commit_workspace_bytes(nbytes, chunk_bytes);
  return REPOPS_OK;
}

repops_status_t repops_commit(const void* data, uint64_t nbytes, uint32_t chunk_bytes,
                              uint8_t* digest, void* workspace, uint64_t workspace_bytes,
                              const repops_launch_t* launch, void* hip_stream) {
  uint64_t need = 0;
  repops_status_t st = repops_commit_workspace(nbytes, chunk_bytes, &need);
  if (st != REPOPS_OK) return st;
  if (launch && (launch->kind != REPOPS_LAUNCH_AUTO || !launch_params_zero_from(launch, 0)))
    return REPOPS_ERR_LAUNCH;
  if (!digest || (nbytes > 0 && !data)) return REPOPS_ERR_NULL;
  if (need > 0 && (!workspace || workspace_bytes < need)) return REPOPS_ERR_WORKSPACE;
  auto span = [](const void* p, uint64_t n) {
    const uintptr_t b = reinterpret_cast<uintptr_t>(p);
    return Extent{b, b + static_cast<uintptr_t>(n)};
  };
  const Extent de = span(digest, 32);
  if (nbytes > 0 && overlaps(de, span(data, nbytes))) return REPOPS_ERR_ALIAS;
  if (need > 0) {
    const Extent we = span(workspace, need);
    if (overlaps(we, de) || (nbytes > 0 && overlaps(we, span(data, nbytes))))
      return REPOPS_ERR_ALIAS;
  }
  if (reinterpret_cast<uintptr_t>(workspace) % 4 != 0) return REPOPS_ERR_STRIDE;
  return hip_status(repops::launch_commit(static_cast<const uint8_t*>(data), nbytes, chunk_bytes,
                                          digest, static_cast<uint32_t*>(workspace),
                                          static_cast<hipStream_t>(hip_stream)));
}

// ---------------------------------------------------------------------------
// erf and the erf-form GELU
// ---------------------------------------------------------------------------

repops_status_t repops_erf(const repops_order_t* order, int64_t n, const float* X, float* Y,
                           const repops_launch_t* launch, void* hip_stream) {
  repops_status_t st = check_elementwise(order, n, X, Y);
  if (st != REPOPS_OK) return st;
  int threads, max_blocks;
  st = ew_launch(launch, &threads, &max_blocks);
  if (st != REPOPS_OK || n == 0) return st;
  return hip_status(
      repops::launch_erf(n, X, Y, threads, max_blocks, static_cast<hipStream_t>(hip_stream)));
}

repops_status_t repops_gelu_erf(const repops_order_t* order, int64_t n, const float* X, float* Y,
                                const repops_launch_t* launch, void* hip_stream) {
  repops_status_t st = check_elementwise(order, n, X, Y);
  if (st != REPOPS_OK) return st;
  int threads, max_blocks;
  st = ew_launch(launch, &threads, &max_blocks);
  if (st != REPOPS_OK || n == 0) return st;
  return hip_status(repops::launch_gelu_erf(n, X, Y, threads, max_blocks,
                                            static_cast<hipStream_t>(hip_stream)));
}

repops_status_t repops_gelu_erf_backward(const repops_order_t* order, int64_t n, const float* X,
                                         const float* dY, float* dX, const repops_launch_t* launch,
                                         void* hip_stream) {
  repops_status_t st = check_elementwise(order, n, X, dX);
  if (st != REPOPS_OK) return st;
  if ((st = check_elementwise(order, n, dY, dX)) != REPOPS_OK) return st;
  int threads, max_blocks;
  st = ew_launch(launch, &threads, &max_blocks);
  if (st != REPOPS_OK || n == 0) return st;
  return hip_status(repops::launch_gelu_bwd(n, X, dY, dX, threads, max_blocks,
                                            static_cast<hipStream_t>(hip_stream), true));
}

}  // extern "C"
