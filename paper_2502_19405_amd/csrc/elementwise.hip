// Reproducible elementwise exp, erf, tanh-form and erf-form GELU for gfx950.
//
// Each element is independent, so the launch only decides which lane computes
// which element.  Aligned, vectorisable spans go through 16-byte loads and
// stores; the scalar loop covers the rest.  Y == X is allowed: every lane
// reads its elements before writing them.
#include <hip/hip_runtime.h>

#include "rep_math.h"
#include "repops_internal.h"
#include "stream_store.h"

#pragma clang fp contract(off)

namespace repops {
namespace {

struct CopyOp {  // no arithmetic: the streaming ceiling of this kernel
  __device__ __forceinline__ float operator()(float x) const { return x; }
};
struct ExpOp {
  __device__ __forceinline__ float operator()(float x) const { return rep_exp(x); }
};
struct GeluOp {
  __device__ __forceinline__ float operator()(float x) const { return rep_gelu(x); }
};
struct ErfOp {
  __device__ __forceinline__ float operator()(float x) const { return rep_erf(x); }
};
struct GeluErfOp {
  __device__ __forceinline__ float operator()(float x) const { return rep_gelu_erf(x); }
};

template <class Op>
__global__ __launch_bounds__(1024) void elementwise_kernel(int64_t n, const float* __restrict__ x,
                                                           float* y, int vec) {
  const Op op;
  const int64_t tid = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
  int64_t done = 0;
  if (vec) {
    const int64_t n4 = n / 4;
    const float4* x4 = reinterpret_cast<const float4*>(x);
    float4* y4 = reinterpret_cast<float4*>(y);
    for (int64_t i = tid; i < n4; i += stride) {
      const float4 v = x4[i];
      float4 o;
      o.x = op(v.x);
      o.y = op(v.y);
      o.z = op(v.z);
      o.w = op(v.w);
      st_stream(y4 + i, o);
    }
    done = n4 * 4;
  }
  for (int64_t i = done + tid; i < n; i += stride) st_stream(y + i, op(x[i]));
}

template <class Op>
hipError_t launch(int64_t n, const float* x, float* y, int threads, int max_blocks, hipStream_t s) {
  const bool vec = (reinterpret_cast<uintptr_t>(x) % 16 == 0) &&
                   (reinterpret_cast<uintptr_t>(y) % 16 == 0);
  const int64_t items = vec ? (n + 3) / 4 : n;
  int64_t blocks = (items + threads - 1) / threads;
  if (max_blocks > 0 && blocks > max_blocks) blocks = max_blocks;
  const int64_t cap = int64_t(1) << 30;
  if (blocks > cap) blocks = cap;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(elementwise_kernel<Op>, dim3(static_cast<unsigned>(blocks)), dim3(threads), 0,
                     s, n, x, y, vec ? 1 : 0);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gelu(int64_t n, const float* x, float* y, int threads, int max_blocks,
                       hipStream_t s) {
  return launch<GeluOp>(n, x, y, threads, max_blocks, s);
}

hipError_t launch_copy(int64_t n, const float* x, float* y, int threads, int max_blocks,
                       hipStream_t s) {
  return launch<CopyOp>(n, x, y, threads, max_blocks, s);
}

hipError_t launch_exp(int64_t n, const float* x, float* y, int threads, int max_blocks,
                      hipStream_t s) {
  return launch<ExpOp>(n, x, y, threads, max_blocks, s);
}

hipError_t launch_erf(int64_t n, const float* x, float* y, int threads, int max_blocks,
                      hipStream_t s) {
  return launch<ErfOp>(n, x, y, threads, max_blocks, s);
}

hipError_t launch_gelu_erf(int64_t n, const float* x, float* y, int threads, int max_blocks,
                           hipStream_t s) {
  return launch<GeluErfOp>(n, x, y, threads, max_blocks, s);
}

}  // namespace repops
