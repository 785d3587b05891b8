// The last operations of every GEMM kernel's output, shared by the vector and
// matrix-core paths so that they cannot drift apart: the contraction's value
// scaled by alpha (batched products) and plus bias[j] (matmul), each one
// rounded operation; for the GELU backward's product, times the GELU
// derivative at the forward input (one rounded multiplication, as the
// elementwise GELU backward takes it); then the store -- and, for
// repops_matmul_gelu, the GELU of the stored value into a second array.  The
// GELU functions are the ones the elementwise kernels run, so every array has
// the bits of the separate calls.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "rep_math.h"
#include "repops_internal.h"

#pragma clang fp contract(off)

namespace repops {

// The epilogue's arithmetic with the scale and the bias value at hand (the
// same rounded operations, in the same order, as gemm_epilogue).
template <bool ALPHA, bool BIAS>
__device__ __forceinline__ float gemm_scale_bias(float acc, float alpha, float bias_j) {
  float v = acc;
  if constexpr (ALPHA) v = v * alpha;
  if constexpr (BIAS) v = v + bias_j;
  return v;
}

__device__ __forceinline__ float gemm_epilogue(const GemmArgs& g, float acc, int64_t j) {
  float v = acc;
  if (g.has_alpha) v = v * g.alpha;
  if (g.bias) v = v + g.bias[j];
  return v;
}

// Output (i, j) of one batch element (C, G and X, the GELU backward's
// forward input, already offset to it; G and X nullable).
__device__ __forceinline__ void gemm_store(const GemmArgs& g, float* C, float* G, const float* X,
                                           int64_t i, int64_t j, float acc) {
  float v = gemm_epilogue(g, acc, j);
  if (X) v = v * rep_gelu_grad(X[i * g.ld_gelu_in + j]);
  C[i * g.ldc + j] = v;
  if (G) G[i * g.ldg + j] = rep_gelu(v);
}

}  // namespace repops
