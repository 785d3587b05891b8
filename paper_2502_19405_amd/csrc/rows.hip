// Reproducible row softmax and row LayerNorm for gfx950.
//
// Row sums follow the order descriptor, a function of the row length n and
// the row width W only (the Verde paper fixes no row-reduction order; Section
// 3.2 asks only that the order-critical dimension follow one fixed order):
//   strided tree: W partials q[l], x_j added to q[j mod W] in ascending j, then
//       q[l] = q[l] + q[l+s] for s = W/2, ..., 1 (l < s); result q[0];
//   blocked left-to-right: partials of W consecutive elements added left to
//       right.
//
// The wave kernels map the strided tree with W = 64 onto one 64-lane wave:
// lane l owns q[l] and reads x[l], x[l+64], ... (every load instruction covers
// 256 contiguous bytes), and the halving tree is six cross-lane steps.  The
// generic kernels take any W and either combine, one wave per row, with the
// partials in LDS.
#include <hip/hip_runtime.h>

#include "rep_math.h"
#include "repops_internal.h"
#include "row_reduce.h"

#pragma clang fp contract(off)

namespace repops {
namespace {

template <int T>
__global__ __launch_bounds__(512) void softmax_wave_kernel(RowArgs a, int wpb) {
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t row = static_cast<int64_t>(blockIdx.x) * wpb + (threadIdx.x >> 6);
  if (row >= a.rows) return;
  const float* x = a.X + row * a.ldx;
  float* y = a.Y + row * a.ldy;
  int64_t valid = a.cols;
  if (a.period > 0) {
    const int64_t v = row % a.period + 1;
    valid = v < valid ? v : valid;
  }
  const float ninf = -__builtin_huge_valf();
  // Segments of 64 columns wholly past the mask are neither read nor
  // exponentiated (a uniform test); their outputs are +0.
  const int64_t live = (valid + kWave - 1) / kWave;
  float v[T];
  float m = ninf;
#pragma unroll
  for (int t = 0; t < T; ++t) {
    const int64_t j = lane + kWave * t;
    v[t] = ninf;
    if (t < live) v[t] = (j < valid) ? x[j] : ninf;  // masked entries are never read
    m = v[t] > m ? v[t] : m;
  }
  m = wave_max(m);
  float q = 0.0f;
#pragma unroll
  for (int t = 0; t < T; ++t) {
    const int64_t j = lane + kWave * t;
    float e = 0.0f;
    if (t < live) e = (j < valid) ? rep_exp(v[t] - m) : 0.0f;
    v[t] = e;
    q = q + e;  // masked terms are +0 and leave q unchanged
  }
  const float s = wave_tree_sum(q);
  const float r = 1.0f / s;
  if (a.cols == kWave * T) {  // full-width row: unconditional stores
#pragma unroll
    for (int t = 0; t < T; ++t) y[lane + kWave * t] = v[t] * r;
  } else {
#pragma unroll
    for (int t = 0; t < T; ++t) {
      const int64_t j = lane + kWave * t;
      if (j < a.cols) y[j] = v[t] * r;
    }
  }
}

template <int T>
__global__ __launch_bounds__(512) void layernorm_wave_kernel(RowArgs a, int wpb) {
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t row = static_cast<int64_t>(blockIdx.x) * wpb + (threadIdx.x >> 6);
  if (row >= a.rows) return;
  const float* x = a.X + row * a.ldx;
  float* y = a.Y + row * a.ldy;
  float v[T];
  float q = 0.0f;
#pragma unroll
  for (int t = 0; t < T; ++t) {
    const int64_t j = lane + kWave * t;
    v[t] = (j < a.cols) ? x[j] : 0.0f;
    q = q + v[t];
  }
  const float n = static_cast<float>(a.cols);
  const float mean = wave_tree_sum(q) / n;
  float q2 = 0.0f;
#pragma unroll
  for (int t = 0; t < T; ++t) {
    const int64_t j = lane + kWave * t;
    v[t] = (j < a.cols) ? v[t] - mean : 0.0f;
    q2 = __builtin_fmaf(v[t], v[t], q2);
  }
  const float var = wave_tree_sum(q2) / n;
  const float rstd = 1.0f / __builtin_sqrtf(var + a.eps);
  auto out = [&](int t, int64_t j) {
    const float tv = v[t] * rstd;
    float o;
    if (a.gamma && a.beta) o = __builtin_fmaf(tv, a.gamma[j], a.beta[j]);
    else if (a.gamma) o = tv * a.gamma[j];
    else if (a.beta) o = tv + a.beta[j];
    else o = tv;
    y[j] = o;
  };
  if (a.cols == kWave * T) {  // full-width row: unconditional stores
#pragma unroll
    for (int t = 0; t < T; ++t) out(t, lane + kWave * t);
  } else {
#pragma unroll
    for (int t = 0; t < T; ++t) {
      const int64_t j = lane + kWave * t;
      if (j < a.cols) out(t, j);
    }
  }
  if (lane == 0) {
    if (a.mean_out) a.mean_out[row] = mean;
    if (a.rstd_out) a.rstd_out[row] = rstd;
  }
}

// ---------------------------------------------------------------------------
// Generic path: one 64-lane workgroup per row, any W and combine mode.
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(64) void softmax_generic_kernel(RowArgs a) {
  __shared__ float qs[1024];
  const int lane = threadIdx.x;
  for (int64_t row = blockIdx.x; row < a.rows; row += gridDim.x) {
    const float* x = a.X + row * a.ldx;
    float* y = a.Y + row * a.ldy;
    int64_t valid = a.cols;
    if (a.period > 0) {
      const int64_t v = row % a.period + 1;
      valid = v < valid ? v : valid;
    }
    float m = -__builtin_huge_valf();
    for (int64_t j = lane; j < valid; j += kWave) m = x[j] > m ? x[j] : m;
    m = wave_max(m);
    auto term = [&](float q, int64_t j) {
      return j < valid ? q + rep_exp(x[j] - m) : q;  // masked terms are +0
    };
    const float s = generic_row_sum(a.cols, a.W, a.blocked, term, qs);
    const float r = 1.0f / s;
    for (int64_t j = lane; j < a.cols; j += kWave) {
      const float e = j < valid ? rep_exp(x[j] - m) : 0.0f;
      y[j] = e * r;  // X may alias Y: x[j] is read before y[j] is written
    }
    __syncthreads();
  }
}

__global__ __launch_bounds__(64) void layernorm_generic_kernel(RowArgs a) {
  __shared__ float qs[1024];
  const int lane = threadIdx.x;
  const float n = static_cast<float>(a.cols);
  for (int64_t row = blockIdx.x; row < a.rows; row += gridDim.x) {
    const float* x = a.X + row * a.ldx;
    float* y = a.Y + row * a.ldy;
    auto sum_term = [&](float q, int64_t j) { return q + x[j]; };
    const float mean = generic_row_sum(a.cols, a.W, a.blocked, sum_term, qs) / n;
    auto sq_term = [&](float q, int64_t j) {
      const float d = x[j] - mean;
      return __builtin_fmaf(d, d, q);
    };
    const float var = generic_row_sum(a.cols, a.W, a.blocked, sq_term, qs) / n;
    const float rstd = 1.0f / __builtin_sqrtf(var + a.eps);
    for (int64_t j = lane; j < a.cols; j += kWave) {
      const float tv = (x[j] - mean) * rstd;
      float o;
      if (a.gamma && a.beta) o = __builtin_fmaf(tv, a.gamma[j], a.beta[j]);
      else if (a.gamma) o = tv * a.gamma[j];
      else if (a.beta) o = tv + a.beta[j];
      else o = tv;
      y[j] = o;
    }
    if (lane == 0) {
      if (a.mean_out) a.mean_out[row] = mean;
      if (a.rstd_out) a.rstd_out[row] = rstd;
    }
    __syncthreads();
  }
}

using WaveKernel = void (*)(RowArgs, int);

WaveKernel pick_softmax(int64_t cols) {
  if (cols <= kWave * 1) return softmax_wave_kernel<1>;
  if (cols <= kWave * 2) return softmax_wave_kernel<2>;
  if (cols <= kWave * 4) return softmax_wave_kernel<4>;
  if (cols <= kWave * 8) return softmax_wave_kernel<8>;
  if (cols <= kWave * 16) return softmax_wave_kernel<16>;
  if (cols <= kWave * 32) return softmax_wave_kernel<32>;
  return softmax_wave_kernel<64>;
}

WaveKernel pick_layernorm(int64_t cols) {
  if (cols <= kWave * 1) return layernorm_wave_kernel<1>;
  if (cols <= kWave * 2) return layernorm_wave_kernel<2>;
  if (cols <= kWave * 4) return layernorm_wave_kernel<4>;
  if (cols <= kWave * 8) return layernorm_wave_kernel<8>;
  if (cols <= kWave * 12) return layernorm_wave_kernel<12>;
  if (cols <= kWave * 16) return layernorm_wave_kernel<16>;
  if (cols <= kWave * 32) return layernorm_wave_kernel<32>;
  return layernorm_wave_kernel<64>;
}

unsigned generic_grid(int64_t rows) {
  const int64_t cap = int64_t(1) << 30;
  return static_cast<unsigned>(rows < cap ? rows : cap);
}

}  // namespace

int64_t rows_wave_max_cols() { return int64_t(kWave) * kMaxPerLane; }

hipError_t launch_softmax_wave(const RowArgs& a, int wpb, hipStream_t s) {
  const int64_t blocks = (a.rows + wpb - 1) / wpb;
  hipLaunchKernelGGL(pick_softmax(a.cols), dim3(static_cast<unsigned>(blocks)), dim3(kWave * wpb),
                     0, s, a, wpb);
  return hipGetLastError();
}

hipError_t launch_layernorm_wave(const RowArgs& a, int wpb, hipStream_t s) {
  const int64_t blocks = (a.rows + wpb - 1) / wpb;
  hipLaunchKernelGGL(pick_layernorm(a.cols), dim3(static_cast<unsigned>(blocks)),
                     dim3(kWave * wpb), 0, s, a, wpb);
  return hipGetLastError();
}

hipError_t launch_softmax_generic(const RowArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(softmax_generic_kernel, dim3(generic_grid(a.rows)), dim3(kWave), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_layernorm_generic(const RowArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(layernorm_generic_kernel, dim3(generic_grid(a.rows)), dim3(kWave), 0, s, a);
  return hipGetLastError();
}

}  // namespace repops
