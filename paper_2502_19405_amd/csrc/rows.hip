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

#pragma clang fp contract(off)

namespace repops {
namespace {

constexpr int kWave = 64;
constexpr int kMaxPerLane = 32;  // register-resident rows: cols <= 64 * 32

// Halving tree over the 64 lane partials: after the step with distance s, lane
// l < s holds q[l] + q[l+s].  Lanes >= s keep stale values that no later step
// reads.  Every lane returns q[0].
__device__ __forceinline__ float wave_tree_sum(float q) {
#pragma unroll
  for (int s = kWave / 2; s >= 1; s >>= 1) {
    const float other = __shfl_down(q, s, kWave);
    q = q + other;
  }
  return __shfl(q, 0, kWave);
}

// Maximum over the wave (order-free up to the sign of a zero maximum, which
// cannot change any softmax output: x - (+0) and x - (-0) differ only for
// x = -0, and exp_rep(+0) = exp_rep(-0) = 1).
__device__ __forceinline__ float wave_max(float m) {
#pragma unroll
  for (int s = kWave / 2; s >= 1; s >>= 1) {
    const float other = __shfl_xor(m, s, kWave);
    m = other > m ? other : m;
  }
  return m;
}

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

// Sum of term(j), j in [0, n), in the descriptor's order.  qs is LDS holding at
// least 1024 floats.  Every lane returns the sum.
template <class Term>
__device__ float generic_row_sum(int64_t n, int W, int blocked, Term term, float* qs) {
  const int lane = threadIdx.x;
  if (!blocked) {
    for (int l = lane; l < W; l += kWave) {
      float q = 0.0f;
      for (int64_t j = l; j < n; j += W) q = term(q, j);
      qs[l] = q;
    }
    __syncthreads();
    for (int s = W / 2; s >= 1; s >>= 1) {
      for (int l = lane; l < s; l += kWave) qs[l] = qs[l] + qs[l + s];
      __syncthreads();
    }
    const float r = qs[0];
    __syncthreads();
    return r;
  }
  // Blocked: block partials are formed 64 at a time in parallel, then added
  // left to right by lane 0.
  const int64_t nblk = (n + W - 1) / W;
  float acc = 0.0f;
  for (int64_t b0 = 0; b0 < nblk; b0 += kWave) {
    const int64_t b = b0 + lane;
    if (b < nblk) {
      float p = 0.0f;
      const int64_t j1 = (b + 1) * W < n ? (b + 1) * W : n;
      for (int64_t j = b * W; j < j1; ++j) p = term(p, j);
      qs[lane] = p;
    }
    __syncthreads();
    if (lane == 0) {
      const int64_t cnt = nblk - b0 < kWave ? nblk - b0 : kWave;
      for (int64_t c = 0; c < cnt; ++c) acc = acc + qs[c];
    }
    __syncthreads();
  }
  if (lane == 0) qs[0] = acc;
  __syncthreads();
  const float r = qs[0];
  __syncthreads();
  return r;
}

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
  return softmax_wave_kernel<32>;
}

WaveKernel pick_layernorm(int64_t cols) {
  if (cols <= kWave * 1) return layernorm_wave_kernel<1>;
  if (cols <= kWave * 2) return layernorm_wave_kernel<2>;
  if (cols <= kWave * 4) return layernorm_wave_kernel<4>;
  if (cols <= kWave * 8) return layernorm_wave_kernel<8>;
  if (cols <= kWave * 12) return layernorm_wave_kernel<12>;
  if (cols <= kWave * 16) return layernorm_wave_kernel<16>;
  return layernorm_wave_kernel<32>;
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
