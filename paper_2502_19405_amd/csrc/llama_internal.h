// Internal interfaces of the Llama-block kernels (llama.hip) for the C ABI
// layer (api.cpp).
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

namespace repops {

struct RopeArgs {
  int64_t rows, heads, head_dim;
  const float* X; int64_t ldx;
  const float* inv_freq;  // [head_dim / 2]
  int64_t period, offset; // position of row r: (period > 0 ? r % period : r) + offset
  int inverse;            // 1: rotate by -angle (the backward)
  float* Y; int64_t ldy;
};

struct RmsArgs {
  int64_t rows, cols;
  const float* X; int64_t ldx;
  float* Y; int64_t ldy;
  int W, blocked;
  const float* gamma;  // nullable
  float eps;
  float* rstd_out;     // nullable
};

// erf and the erf-form GELU (elementwise.hip).
hipError_t launch_erf(int64_t n, const float* x, float* y, int threads, int max_blocks,
                      hipStream_t s);
hipError_t launch_gelu_erf(int64_t n, const float* x, float* y, int threads, int max_blocks,
                           hipStream_t s);

hipError_t launch_sincos(int64_t n, const float* x, float* s, float* c, int threads,
                         int max_blocks, hipStream_t st);
hipError_t launch_rope(const RopeArgs& a, int waves_per_block, hipStream_t s);
int64_t rmsnorm_wave_max_cols();
hipError_t launch_rmsnorm_wave(const RmsArgs& a, int waves_per_block, hipStream_t s);
hipError_t launch_rmsnorm_generic(const RmsArgs& a, hipStream_t s);
// One row per workgroup of S waves (S = 2, 4, 8); cols <= S * 64 * 32.
hipError_t launch_rmsnorm_split(const RmsArgs& a, int S, hipStream_t s);
int64_t rmsnorm_split_max_cols(int S);
hipError_t launch_silu(int64_t n, const float* x, float* y, int threads, int max_blocks,
                       hipStream_t s);
hipError_t launch_swiglu(int64_t n, const float* g, const float* u, float* y, int threads,
                         int max_blocks, hipStream_t s);
hipError_t launch_swiglu_bwd(int64_t n, const float* g, const float* u, const float* dy, float* dg,
                             float* du, int threads, int max_blocks, hipStream_t s);

}  // namespace repops
