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
#include "rows_internal.h"
#include "stream_store.h"

#pragma clang fp contract(off)

namespace repops {
namespace {

template <int T>
__global__ __launch_bounds__(512) void softmax_wave_kernel(RowArgs a, int wpb) {
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t row = static_cast<int64_t>(blockIdx.x) * wpb + wave_id();
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
    for (int t = 0; t < T; ++t) st_stream(y + lane + kWave * t, v[t] * r);
  } else {
#pragma unroll
    for (int t = 0; t < T; ++t) {
      const int64_t j = lane + kWave * t;
      if (j < a.cols) st_stream(y + j, v[t] * r);
    }
  }
}

template <int T>
__global__ __launch_bounds__(512) void layernorm_wave_kernel(RowArgs a, int wpb) {
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t row = static_cast<int64_t>(blockIdx.x) * wpb + wave_id();
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
  // gamma and beta join the row's loads when a lane holds few values
  constexpr bool kPre = T <= 16;
  float gv[kPre ? T : 1], bv[kPre ? T : 1];
  if constexpr (kPre) {
#pragma unroll
    for (int t = 0; t < T; ++t) {
      const int64_t j = lane + kWave * t;
      gv[t] = (a.gamma && j < a.cols) ? a.gamma[j] : 0.0f;
      bv[t] = (a.beta && j < a.cols) ? a.beta[j] : 0.0f;
    }
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
    float gj, bj;
    if constexpr (kPre) {
      gj = gv[t];
      bj = bv[t];
    } else {
      gj = a.gamma ? a.gamma[j] : 0.0f;
      bj = a.beta ? a.beta[j] : 0.0f;
    }
    float o;
    if (a.gamma && a.beta) o = __builtin_fmaf(tv, gj, bj);
    else if (a.gamma) o = tv * gj;
    else if (a.beta) o = tv + bj;
    else o = tv;
    st_stream(y + j, o);
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
// Wide rows: one row per workgroup of S waves.  Wave w holds the columns
// j = lane + 64 * (w * T + t), t < T; the lane chains run through the waves in
// order (chain_across_waves), so every lane sees its terms in exactly the
// order of the one-wave kernels above and the results are the same bits.
// ---------------------------------------------------------------------------

template <int T>
__global__ __launch_bounds__(512) void softmax_split_kernel(RowArgs a) {
  __shared__ float chain[kWave];
  __shared__ float wave_maxima[8];
  const int lane = threadIdx.x & (kWave - 1);
  const int w = wave_id();
  const int S = static_cast<int>(blockDim.x >> 6);
  const float ninf = -__builtin_huge_valf();
  for (int64_t row = blockIdx.x; row < a.rows; row += gridDim.x) {
    const float* x = a.X + row * a.ldx;
    float* y = a.Y + row * a.ldy;
    int64_t valid = a.cols;
    if (a.period > 0) {
      const int64_t v = row % a.period + 1;
      valid = v < valid ? v : valid;
    }
    const int64_t live = (valid + kWave - 1) / kWave;  // segments holding unmasked entries
    const int64_t s0 = int64_t(T) * w;                 // this wave's first segment
    float v[T];
    float m = ninf;
#pragma unroll
    for (int t = 0; t < T; ++t) {
      const int64_t j = lane + kWave * (s0 + t);
      v[t] = ninf;
      if (s0 + t < live) v[t] = (j < valid) ? x[j] : ninf;  // masked entries are never read
      m = v[t] > m ? v[t] : m;
    }
    // The maximum is a value of the row whatever the order of comparison (see
    // wave_max), so the waves' maxima may be combined in any order.
    m = wave_max(m);
    if (lane == 0) wave_maxima[w] = m;
    __syncthreads();
    m = wave_maxima[0];
    for (int k = 1; k < S; ++k) m = wave_maxima[k] > m ? wave_maxima[k] : m;
#pragma unroll
    for (int t = 0; t < T; ++t) {
      const int64_t j = lane + kWave * (s0 + t);
      float e = 0.0f;
      if (s0 + t < live) e = (j < valid) ? rep_exp(v[t] - m) : 0.0f;
      v[t] = e;
    }
    const float q = chain_across_waves(chain, lane, w, S, [&](float c) {
#pragma unroll
      for (int t = 0; t < T; ++t) c = c + v[t];  // masked terms are +0
      return c;
    });
    const float r = 1.0f / wave_tree_sum(q);
#pragma unroll
    for (int t = 0; t < T; ++t) {
      const int64_t j = lane + kWave * (s0 + t);
      if (j < a.cols) st_stream(y + j, v[t] * r);
    }
    __syncthreads();  // chains and maxima read before the next row
  }
}

template <int T>
__global__ __launch_bounds__(512) void layernorm_split_kernel(RowArgs a) {
  __shared__ float chain_sum[kWave];
  __shared__ float chain_sq[kWave];
  const int lane = threadIdx.x & (kWave - 1);
  const int w = wave_id();
  const int S = static_cast<int>(blockDim.x >> 6);
  const float n = static_cast<float>(a.cols);
  for (int64_t row = blockIdx.x; row < a.rows; row += gridDim.x) {
    const float* x = a.X + row * a.ldx;
    float* y = a.Y + row * a.ldy;
    const int64_t j0 = lane + int64_t(kWave) * T * w;
    float v[T];
#pragma unroll
    for (int t = 0; t < T; ++t) {
      const int64_t j = j0 + kWave * t;
      v[t] = (j < a.cols) ? x[j] : 0.0f;
    }
    constexpr bool kPre = T <= 16;  // gamma and beta join the row's loads
    float gv[kPre ? T : 1], bv[kPre ? T : 1];
    if constexpr (kPre) {
#pragma unroll
      for (int t = 0; t < T; ++t) {
        const int64_t j = j0 + kWave * t;
        gv[t] = (a.gamma && j < a.cols) ? a.gamma[j] : 0.0f;
        bv[t] = (a.beta && j < a.cols) ? a.beta[j] : 0.0f;
      }
    }
    const float q = chain_across_waves(chain_sum, lane, w, S, [&](float c) {
#pragma unroll
      for (int t = 0; t < T; ++t) c = c + v[t];
      return c;
    });
    const float mean = wave_tree_sum(q) / n;
#pragma unroll
    for (int t = 0; t < T; ++t) {
      const int64_t j = j0 + kWave * t;
      v[t] = (j < a.cols) ? v[t] - mean : 0.0f;
    }
    const float q2 = chain_across_waves(chain_sq, lane, w, S, [&](float c) {
#pragma unroll
      for (int t = 0; t < T; ++t) c = __builtin_fmaf(v[t], v[t], c);
      return c;
    });
    const float var = wave_tree_sum(q2) / n;
    const float rstd = 1.0f / __builtin_sqrtf(var + a.eps);
#pragma unroll
    for (int t = 0; t < T; ++t) {
      const int64_t j = j0 + kWave * t;
      if (j < a.cols) {
        const float tv = v[t] * rstd;
        float gj, bj;
        if constexpr (kPre) {
          gj = gv[t];
          bj = bv[t];
        } else {
          gj = a.gamma ? a.gamma[j] : 0.0f;
          bj = a.beta ? a.beta[j] : 0.0f;
        }
        float o;
        if (a.gamma && a.beta) o = __builtin_fmaf(tv, gj, bj);
        else if (a.gamma) o = tv * gj;
        else if (a.beta) o = tv + bj;
        else o = tv;
        st_stream(y + j, o);
      }
    }
    if (w == 0 && lane == 0) {
      if (a.mean_out) a.mean_out[row] = mean;
      if (a.rstd_out) a.rstd_out[row] = rstd;
    }
    __syncthreads();  // chains read before the next row
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
      st_stream(y + j, e * r);  // X may alias Y: x[j] is read before y[j] is written
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
      st_stream(y + j, o);
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
int64_t rows_split_max_cols(int S) { return split_max_cols(S); }

namespace {
using SplitKernel = void (*)(RowArgs);
template <template <int> class K>
SplitKernel pick_split(int64_t cols, int S) {
  const int64_t per_lane = (cols + int64_t(kWave) * S - 1) / (int64_t(kWave) * S);
  if (per_lane <= 1) return K<1>::fn;
  if (per_lane <= 2) return K<2>::fn;
  if (per_lane <= 4) return K<4>::fn;
  if (per_lane <= 8) return K<8>::fn;
  if (per_lane <= 16) return K<16>::fn;
  if (per_lane <= 32) return K<32>::fn;
  return nullptr;
}
template <int T> struct SoftmaxSplit { static constexpr SplitKernel fn = softmax_split_kernel<T>; };
template <int T> struct LayernormSplit { static constexpr SplitKernel fn = layernorm_split_kernel<T>; };

hipError_t launch_split(SplitKernel k, const RowArgs& a, int S, hipStream_t s) {
  if (!k) return hipErrorInvalidValue;
  const int64_t cap = int64_t(1) << 30;
  hipLaunchKernelGGL(k, dim3(static_cast<unsigned>(a.rows < cap ? a.rows : cap)),
                     dim3(kWave * S), 0, s, a);
  return hipGetLastError();
}
}  // namespace

hipError_t launch_softmax_split(const RowArgs& a, int S, hipStream_t s) {
  return launch_split(pick_split<SoftmaxSplit>(a.cols, S), a, S, s);
}

hipError_t launch_layernorm_split(const RowArgs& a, int S, hipStream_t s) {
  return launch_split(pick_split<LayernormSplit>(a.cols, S), a, S, s);
}

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
