// Internal interfaces of the training-step kernels (train.hip) for the C ABI
// layer (api.cpp).
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

namespace repops {

// Backward row operators.  Softmax: Y = forward output.  LayerNorm: Y = the
// forward input X, with the forward's mean / rstd and gamma (nullable).
// RMSNorm (rms = 1) runs the LayerNorm kernels with mean = +0 and the mean of
// g taken as +0: x - 0 = x and g - 0 = g exactly, which leaves
// t = x rstd and dx = rstd (g - t b), the RMSNorm gradient.
struct RowBwdArgs {
  int64_t rows, cols;
  const float* Y; int64_t ldy;
  const float* dY; int64_t lddy;
  float* dX; int64_t lddx;
  int W;
  int blocked;
  int64_t period;     // softmax causal period, 0 = none
  const float* mean; const float* rstd; const float* gamma;
  int rms;            // RMSNorm: no mean, no a term
};

hipError_t launch_softmax_bwd_wave(const RowBwdArgs& a, int waves_per_block, hipStream_t s);
hipError_t launch_softmax_bwd_generic(const RowBwdArgs& a, hipStream_t s);
hipError_t launch_layernorm_bwd_wave(const RowBwdArgs& a, int waves_per_block, hipStream_t s);
hipError_t launch_layernorm_bwd_generic(const RowBwdArgs& a, hipStream_t s);
// One row per workgroup of S waves (2, 4, 8), at most 32 values per lane.
hipError_t launch_softmax_bwd_split(const RowBwdArgs& a, int S, hipStream_t s);
hipError_t launch_layernorm_bwd_split(const RowBwdArgs& a, int S, hipStream_t s);

// LayerNorm parameter gradients over rows, blocks of k_block rows (0 = one
// block).  ws holds 2 * blocks * cols floats when there is more than one block
// (block partials in column tiles, each tile block-major).
struct LnParamArgs {
  int64_t rows, cols, k_block;
  const float* X; int64_t ldx;
  const float* dY; int64_t lddy;
  const float* mean; const float* rstd;
  float* dgamma; float* dbeta;  // nullable
  float* ws;
  int rms;            // RMSNorm: t = x * rstd (no mean)
  int sum_only;       // column sums of dY only (the bias gradient): no X, mean, rstd
};

int64_t layernorm_param_blocks(int64_t rows, int64_t k_block);
int64_t layernorm_param_grid(int64_t rows, int64_t cols, int64_t k_block);
hipError_t launch_layernorm_param(const LnParamArgs& a, hipStream_t s);
// Fused input and parameter gradients (W = 64 strided tree, cols <= 2048,
// k_block >= 1): one workgroup of R waves per block of rows.
int layernorm_fused_rows(int64_t rows, int64_t cols, int64_t k_block, int requested);
hipError_t launch_layernorm_bwd_fused(const RowBwdArgs& a, const LnParamArgs& p, int R,
                                      hipStream_t s);

// Fused input and parameter gradients for few row blocks (W = 64 strided
// tree, cols <= 1024): G workgroups per block, each with a column slice of
// the chains and a share of the rows' dX.  dX must not alias X or dY.
struct ColsplitPlan { int G, slice, swu; };
bool layernorm_colsplit_plan(int64_t rows, int64_t cols, int64_t k_block, ColsplitPlan* pl);
hipError_t launch_layernorm_bwd_colsplit(const RowBwdArgs& a, const LnParamArgs& p,
                                         const ColsplitPlan& pl, hipStream_t s);

// Device address of the fixed scratch array (kNoallocScratchBytes) on the
// current device, looked up once per device.
constexpr uint64_t kNoallocScratchBytes = uint64_t(8) << 20;
hipError_t noalloc_scratch(void** ptr);

hipError_t launch_gelu_bwd(int64_t n, const float* x, const float* dy, float* dx, int threads,
                           int max_blocks, hipStream_t s, bool erf_form);

// Step scalars of the Adam update, computed on the host.
struct AdamScalars {
  float c1, c2, step, sbc2, dec, eps, wd, b1, b2;
  int decay;  // 0 none, 1 decoupled (AdamW), 2 coupled (L2 added to the gradient)
};

hipError_t launch_adam(int64_t n, float* p, const float* g, float* m, float* v,
                       const AdamScalars& sc, int threads, int max_blocks, hipStream_t s);

}  // namespace repops
