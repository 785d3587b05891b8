// The last operations of every GEMM kernel's output, shared by the vector and
// matrix-core paths so that they cannot drift apart: the contraction's value
// scaled by alpha (batched products) and plus bias[j] (matmul), each one
// rounded operation, then the store -- and, for repops_matmul_gelu, the GELU
// of the stored value into a second array (the same rep_gelu the elementwise
// kernel runs, so both arrays have the bits of the separate calls).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "rep_math.h"
#include "repops_internal.h"

#pragma clang fp contract(off)

namespace repops {

__device__ __forceinline__ float gemm_epilogue(const GemmArgs& g, float acc, int64_t j) {
  float v = acc;
  if (g.has_alpha) v = v * g.alpha;
  if (g.bias) v = v + g.bias[j];
  return v;
}

// Output (i, j) of one batch element (C and G already offset to it).
__device__ __forceinline__ void gemm_store(const GemmArgs& g, float* C, float* G, int64_t i,
                                           int64_t j, float acc) {
  const float v = gemm_epilogue(g, acc, j);
  C[i * g.ldc + j] = v;
  if (G) G[i * g.ldg + j] = rep_gelu(v);
}

}  // namespace repops
