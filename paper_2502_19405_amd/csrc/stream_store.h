// Stores of streamed results.  The row, elementwise and optimizer kernels
// write each output element once and never read it back in the same launch,
// so their stores carry the nontemporal hint: the written lines are not kept
// in the caches at the expense of inputs still to be read.  The hint changes
// cache policy only, never the values written.
#pragma once

#include <hip/hip_runtime.h>

namespace repops {

__device__ __forceinline__ void st_stream(float* p, float v) { __builtin_nontemporal_store(v, p); }

__device__ __forceinline__ void st_stream(float4* p, const float4& v) {
  typedef float v4f __attribute__((ext_vector_type(4)));
  const v4f q = {v.x, v.y, v.z, v.w};
  __builtin_nontemporal_store(q, reinterpret_cast<v4f*>(p));
}

}  // namespace repops
