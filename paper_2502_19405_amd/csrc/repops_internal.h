// Internal interfaces between the C ABI layer (api.cpp) and the HIP kernels.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

namespace repops {

struct GemmArgs {
  int64_t batch0, batch1, m, n, k;
  const float* A; int64_t sa0, sa1, lda; int ta;
  const float* B; int64_t sb0, sb1, ldb; int tb;
  float* C; int64_t sc0, sc1, ldc;
  float* G; int64_t ldg;  // nullable: G = gelu(C) elementwise, batch offsets as C's
  const float* gelu_in; int64_t ld_gelu_in;  // nullable: C = value * gelu'(gelu_in), offsets as C's
  const float* bias;  // nullable, [n]
  float alpha;
  int has_alpha;      // 1: C = acc * alpha
  int64_t k_block;    // 0 = one block
  int fused;          // 1: fma chain, 0: rounded product then add
  int causal;         // per batch element: 0 none; 1 outputs with j > i unspecified (the
                      // matrix-core kernels skip tiles wholly above the diagonal); 2 A is
                      // zero at kk > i (their kernels skip the all-zero k blocks)
};

struct GemmConfig {
  const char* name;
  int bm, bn, bk;
};

// Tables of compiled tile configurations.
int gemm_tiled_count();
const GemmConfig* gemm_tiled_config(int index);
int gemm_mfma_count();
const GemmConfig* gemm_mfma_config(int index);

// Several independent products in one launch of the default matrix-core tile
// (table entry 0): problem p owns tiles [first[p], first[p + 1]).  Each
// product must meet the staged kernel's conditions (gemm_mfma_staged_ok).
constexpr int kMaxGroup = 8;
struct GroupArgs {
  GemmArgs g[kMaxGroup];
  int64_t first[kMaxGroup + 1];
  int64_t tiles_m[kMaxGroup], tiles_n[kMaxGroup];
  int count;
};
bool gemm_mfma_staged_ok(const GemmArgs& g, int index);
// Tiles the persistent ring form of matrix-core entry `index` would take for
// this product (0 when it cannot); *cus receives the device's compute units,
// and the launch takes the ring form when the tiles outnumber them.
int64_t gemm_mfma_ring_tiles(const GemmArgs& g, int index, int* cus);
// Tile edge lengths of table entry `index` (for the grouped launch's tiles).
void gemm_mfma_tile(int index, int* bm, int* bn);
hipError_t launch_gemm_mfma_grouped(const GroupArgs& ga, hipStream_t s);

hipError_t launch_gemm_simple(const GemmArgs& a, hipStream_t s);
hipError_t launch_gemm_tiled(const GemmArgs& a, int index, hipStream_t s);
hipError_t launch_gemm_mfma(const GemmArgs& a, int index, hipStream_t s);

struct RowArgs {
  int64_t rows, cols;
  const float* X; int64_t ldx;
  float* Y; int64_t ldy;
  int W;              // row width
  int blocked;        // 0 = strided tree, 1 = blocked left-to-right
  // softmax
  int64_t period;     // causal period, 0 = none
  // layernorm
  const float* gamma; const float* beta; float eps;
  float* mean_out; float* rstd_out;
};

hipError_t launch_softmax_wave(const RowArgs& a, int waves_per_block, hipStream_t s);
hipError_t launch_softmax_generic(const RowArgs& a, hipStream_t s);
hipError_t launch_layernorm_wave(const RowArgs& a, int waves_per_block, hipStream_t s);
hipError_t launch_layernorm_generic(const RowArgs& a, hipStream_t s);
// Largest row length the register-resident wave kernels hold.
int64_t rows_wave_max_cols();

hipError_t launch_gelu(int64_t n, const float* x, float* y, int threads, int max_blocks,
                       hipStream_t s);
hipError_t launch_copy(int64_t n, const float* x, float* y, int threads, int max_blocks,
                      hipStream_t s);
hipError_t launch_exp(int64_t n, const float* x, float* y, int threads, int max_blocks,
                      hipStream_t s);

}  // namespace repops
