// Reproducible Llama-block operators for gfx950: sin/cos, the rotary position
// embedding, RMSNorm, SiLU and the SiLU-gated unit (forward and backward).
//
// The Llama programs of the Verde paper's evaluation (Section 4.2) use these
// beside the operators of the DistilBERT block; Section 3.1 lists the math
// functions that RepOps rebuilds with a controlled order.  Every output is one
// fixed sequence of binary32 operations; row sums take the order descriptor's
// row order.
//
// Rotary embedding: one 64-lane wave per row; lane i computes the angle and
// its sin/cos once and applies them to the pair (i, i + d/2) of every head, so
// the transcendental work is amortised over the heads and the kernel streams
// the row once (8 B per element).
#include <hip/hip_runtime.h>

#include "llama_internal.h"
#include "rep_math.h"
#include "row_reduce.h"
#include "rows_internal.h"
#include "stream_store.h"

#pragma clang fp contract(off)

namespace repops {
namespace {

// ---------------------------------------------------------------------------
// sin / cos (elementwise test export)
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(1024) void sincos_kernel(int64_t n, const float* x, float* s,
                                                      float* c) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n;
       i += stride) {
    float sv, cv;
    rep_sincos(x[i], sv, cv);
    if (s) s[i] = sv;
    if (c) c[i] = cv;
  }
}

// ---------------------------------------------------------------------------
// rotary embedding (rotate-half pairing)
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(512) void rope_kernel(RopeArgs a, int wpb) {
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t row = static_cast<int64_t>(blockIdx.x) * wpb + wave_id();
  if (row >= a.rows) return;
  const int64_t pos = (a.period > 0 ? row % a.period : row) + a.offset;
  const float pf = static_cast<float>(pos);  // exact: pos < 2^24
  const float* x = a.X + row * a.ldx;
  float* y = a.Y + row * a.ldy;
  const int64_t half = a.head_dim / 2;
  for (int64_t i = lane; i < half; i += kWave) {
    const float angle = pf * a.inv_freq[i];
    float sv, cv;
    rep_sincos(angle, sv, cv);
#pragma unroll 4
    for (int64_t h = 0; h < a.heads; ++h) {
      const int64_t j = h * a.head_dim + i;
      const float x1 = x[j], x2 = x[j + half];
      const float p1 = x1 * cv, p2 = x2 * sv, p3 = x2 * cv, p4 = x1 * sv;
      // Y may equal X: both elements of the pair are read before either is written
      st_stream(y + j, a.inverse ? p1 + p2 : p1 - p2);
      st_stream(y + j + half, a.inverse ? p3 - p4 : p3 + p4);
    }
  }
}

// ---------------------------------------------------------------------------
// RMSNorm forward: ms = rowsum(fma(x, x, .)) / n; rstd = 1 / sqrt(ms + eps);
// y = (x * rstd) * gamma.
// ---------------------------------------------------------------------------

template <int T>
__global__ __launch_bounds__(512) void rmsnorm_wave_kernel(RmsArgs a, int wpb) {
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
    q = __builtin_fmaf(v[t], v[t], q);  // terms past the row: fma(0, 0, q) = q
  }
  constexpr bool kPre = T <= 16;  // gamma joins the row's loads when a lane holds few values
  float gv[kPre ? T : 1];
  if constexpr (kPre) {
#pragma unroll
    for (int t = 0; t < T; ++t) {
      const int64_t j = lane + kWave * t;
      gv[t] = (a.gamma && j < a.cols) ? a.gamma[j] : 0.0f;
    }
  }
  const float n = static_cast<float>(a.cols);
  const float ms = wave_tree_sum(q) / n;
  const float rstd = 1.0f / __builtin_sqrtf(ms + a.eps);
  auto out = [&](int t, int64_t j) {
    const float tv = v[t] * rstd;
    if constexpr (kPre) return a.gamma ? tv * gv[t] : tv;
    else return a.gamma ? tv * a.gamma[j] : tv;
  };
  if (a.cols == kWave * T) {
#pragma unroll
    for (int t = 0; t < T; ++t) st_stream(y + lane + kWave * t, out(t, lane + kWave * t));
  } else {
#pragma unroll
    for (int t = 0; t < T; ++t) {
      const int64_t j = lane + kWave * t;
      if (j < a.cols) st_stream(y + j, out(t, j));
    }
  }
  if (lane == 0 && a.rstd_out) a.rstd_out[row] = rstd;
}

// Wide rows: one row per workgroup of S waves.  Wave w holds the values
// j = lane + 64 * (w * T + t), t < T; the lane's chain passes from wave to
// wave in order through LDS (wave w continues where wave w - 1 stopped), so
// every lane sees its values in exactly the order of the one-wave kernel.
// After the last wave's turn every wave reduces the finished chains itself.
template <int T>
__global__ __launch_bounds__(512) void rmsnorm_split_kernel(RmsArgs a) {
  __shared__ float chain[kWave];
  const int lane = threadIdx.x & (kWave - 1);
  const int w = wave_id();
  const int S = static_cast<int>(blockDim.x >> 6);
  const float n = static_cast<float>(a.cols);
  for (int64_t row = blockIdx.x; row < a.rows; row += gridDim.x) {
    const float* x = a.X + row * a.ldx;
    float* y = a.Y + row * a.ldy;
    const int64_t j0 = lane + int64_t(kWave) * T * w;  // this wave's first column
    float v[T];
#pragma unroll
    for (int t = 0; t < T; ++t) {
      const int64_t j = j0 + kWave * t;
      v[t] = (j < a.cols) ? x[j] : 0.0f;
    }
    constexpr bool kPre = T <= 16;  // gamma joins the row's loads
    float gv[kPre ? T : 1];
    if constexpr (kPre) {
#pragma unroll
      for (int t = 0; t < T; ++t) {
        const int64_t j = j0 + kWave * t;
        gv[t] = (a.gamma && j < a.cols) ? a.gamma[j] : 0.0f;
      }
    }
    const float q = chain_across_waves(chain, lane, w, S, [&](float c) {
#pragma unroll
      for (int t = 0; t < T; ++t) c = __builtin_fmaf(v[t], v[t], c);  // past the row: c
      return c;
    });
    const float ms = wave_tree_sum(q) / n;
    const float rstd = 1.0f / __builtin_sqrtf(ms + a.eps);
#pragma unroll
    for (int t = 0; t < T; ++t) {
      const int64_t j = j0 + kWave * t;
      if (j < a.cols) {
        const float tv = v[t] * rstd;
        if constexpr (kPre) st_stream(y + j, a.gamma ? tv * gv[t] : tv);
        else st_stream(y + j, a.gamma ? tv * a.gamma[j] : tv);
      }
    }
    if (w == 0 && lane == 0 && a.rstd_out) a.rstd_out[row] = rstd;
    __syncthreads();  // every wave has read the chains before the next row
  }
}

__global__ __launch_bounds__(64) void rmsnorm_generic_kernel(RmsArgs a) {
  __shared__ float qs[1024];
  const int lane = threadIdx.x;
  const float n = static_cast<float>(a.cols);
  for (int64_t row = blockIdx.x; row < a.rows; row += gridDim.x) {
    const float* x = a.X + row * a.ldx;
    float* y = a.Y + row * a.ldy;
    auto sq_term = [&](float q, int64_t j) { return __builtin_fmaf(x[j], x[j], q); };
    const float ms = generic_row_sum(a.cols, a.W, a.blocked, sq_term, qs) / n;
    const float rstd = 1.0f / __builtin_sqrtf(ms + a.eps);
    for (int64_t j = lane; j < a.cols; j += kWave) {
      const float tv = x[j] * rstd;
      st_stream(y + j, a.gamma ? tv * a.gamma[j] : tv);  // Y may equal X: x[j] is read first
    }
    if (lane == 0 && a.rstd_out) a.rstd_out[row] = rstd;
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// SiLU and the SiLU-gated unit: elementwise, 16-byte accesses when aligned.
// ---------------------------------------------------------------------------

struct SiluOp {
  __device__ __forceinline__ float operator()(float g, float) const { return rep_silu(g); }
};
struct SwigluOp {
  __device__ __forceinline__ float operator()(float g, float u) const { return rep_silu(g) * u; }
};

template <class Op, bool TWO>
__global__ __launch_bounds__(1024) void gated_kernel(int64_t n, const float* g, const float* u,
                                                     float* y, int vec) {
  const Op op;
  const int64_t tid = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
  int64_t done = 0;
  if (vec) {
    const int64_t n4 = n / 4;
    const float4* g4 = reinterpret_cast<const float4*>(g);
    const float4* u4 = reinterpret_cast<const float4*>(u);
    float4* y4 = reinterpret_cast<float4*>(y);
    for (int64_t i = tid; i < n4; i += stride) {
      const float4 gv = g4[i];
      float4 uv = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
      if (TWO) uv = u4[i];
      float4 o;
      o.x = op(gv.x, uv.x);
      o.y = op(gv.y, uv.y);
      o.z = op(gv.z, uv.z);
      o.w = op(gv.w, uv.w);
      st_stream(y4 + i, o);
    }
    done = n4 * 4;
  }
  for (int64_t i = done + tid; i < n; i += stride) st_stream(y + i, op(g[i], TWO ? u[i] : 0.0f));
}

// dgate = (dy * u) * silu'(g); dup = dy * silu(g).
__device__ __forceinline__ void swiglu_bwd_one(float g, float u, float dy, float& dg, float& du) {
  const float dyu = dy * u;
  dg = dyu * rep_silu_grad(g);
  du = dy * rep_silu(g);
}

__global__ __launch_bounds__(1024) void swiglu_bwd_kernel(int64_t n, const float* g, const float* u,
                                                          const float* dy, float* dg, float* du,
                                                          int vec) {
  const int64_t tid = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
  int64_t done = 0;
  if (vec) {
    const int64_t n4 = n / 4;
    const float4* g4 = reinterpret_cast<const float4*>(g);
    const float4* u4 = reinterpret_cast<const float4*>(u);
    const float4* d4 = reinterpret_cast<const float4*>(dy);
    float4* dg4 = reinterpret_cast<float4*>(dg);
    float4* du4 = reinterpret_cast<float4*>(du);
    for (int64_t i = tid; i < n4; i += stride) {
      const float4 gv = g4[i], uv = u4[i], dv = d4[i];
      float4 a, b;
      swiglu_bwd_one(gv.x, uv.x, dv.x, a.x, b.x);
      swiglu_bwd_one(gv.y, uv.y, dv.y, a.y, b.y);
      swiglu_bwd_one(gv.z, uv.z, dv.z, a.z, b.z);
      swiglu_bwd_one(gv.w, uv.w, dv.w, a.w, b.w);
      st_stream(dg4 + i, a);
      st_stream(du4 + i, b);
    }
    done = n4 * 4;
  }
  for (int64_t i = done + tid; i < n; i += stride) {
    float a, b;
    swiglu_bwd_one(g[i], u[i], dy[i], a, b);
    st_stream(dg + i, a);
    st_stream(du + i, b);
  }
}

using RmsWaveKernel = void (*)(RmsArgs, int);

RmsWaveKernel pick_rmsnorm(int64_t cols) {
  if (cols <= kWave * 1) return rmsnorm_wave_kernel<1>;
  if (cols <= kWave * 2) return rmsnorm_wave_kernel<2>;
  if (cols <= kWave * 4) return rmsnorm_wave_kernel<4>;
  if (cols <= kWave * 8) return rmsnorm_wave_kernel<8>;
  if (cols <= kWave * 12) return rmsnorm_wave_kernel<12>;
  if (cols <= kWave * 16) return rmsnorm_wave_kernel<16>;
  if (cols <= kWave * 32) return rmsnorm_wave_kernel<32>;
  return rmsnorm_wave_kernel<64>;
}

bool aligned16(const void* p) { return reinterpret_cast<uintptr_t>(p) % 16 == 0; }

int64_t ew_grid(int64_t items, int threads, int max_blocks) {
  int64_t blocks = (items + threads - 1) / threads;
  if (max_blocks > 0 && blocks > max_blocks) blocks = max_blocks;
  const int64_t cap = int64_t(1) << 30;
  if (blocks > cap) blocks = cap;
  if (blocks < 1) blocks = 1;
  return blocks;
}

}  // namespace

// RMSNorm rows stay in registers up to 64 values per lane (Llama's 4096).
int64_t rmsnorm_wave_max_cols() { return int64_t(kWave) * kMaxPerLane; }
int64_t rmsnorm_split_max_cols(int S) { return split_max_cols(S); }

hipError_t launch_sincos(int64_t n, const float* x, float* s, float* c, int threads,
                         int max_blocks, hipStream_t st) {
  hipLaunchKernelGGL(sincos_kernel, dim3(static_cast<unsigned>(ew_grid(n, threads, max_blocks))),
                     dim3(threads), 0, st, n, x, s, c);
  return hipGetLastError();
}

hipError_t launch_rope(const RopeArgs& a, int wpb, hipStream_t s) {
  const int64_t blocks = (a.rows + wpb - 1) / wpb;
  hipLaunchKernelGGL(rope_kernel, dim3(static_cast<unsigned>(blocks)), dim3(kWave * wpb), 0, s, a,
                     wpb);
  return hipGetLastError();
}

hipError_t launch_rmsnorm_wave(const RmsArgs& a, int wpb, hipStream_t s) {
  const int64_t blocks = (a.rows + wpb - 1) / wpb;
  hipLaunchKernelGGL(pick_rmsnorm(a.cols), dim3(static_cast<unsigned>(blocks)), dim3(kWave * wpb),
                     0, s, a, wpb);
  return hipGetLastError();
}

hipError_t launch_rmsnorm_split(const RmsArgs& a, int S, hipStream_t s) {
  const int64_t per_wave = (a.cols + int64_t(kWave) * S - 1) / (int64_t(kWave) * S);
  void (*k)(RmsArgs) = nullptr;
  if (per_wave <= 1) k = rmsnorm_split_kernel<1>;
  else if (per_wave <= 2) k = rmsnorm_split_kernel<2>;
  else if (per_wave <= 4) k = rmsnorm_split_kernel<4>;
  else if (per_wave <= 8) k = rmsnorm_split_kernel<8>;
  else if (per_wave <= 16) k = rmsnorm_split_kernel<16>;
  else if (per_wave <= 32) k = rmsnorm_split_kernel<32>;
  else return hipErrorInvalidValue;
  const int64_t cap = int64_t(1) << 30;
  hipLaunchKernelGGL(k, dim3(static_cast<unsigned>(a.rows < cap ? a.rows : cap)),
                     dim3(kWave * S), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_rmsnorm_generic(const RmsArgs& a, hipStream_t s) {
  const int64_t cap = int64_t(1) << 30;
  hipLaunchKernelGGL(rmsnorm_generic_kernel, dim3(static_cast<unsigned>(a.rows < cap ? a.rows : cap)),
                     dim3(kWave), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_silu(int64_t n, const float* x, float* y, int threads, int max_blocks,
                       hipStream_t s) {
  const bool vec = aligned16(x) && aligned16(y);
  const int64_t blocks = ew_grid(vec ? (n + 3) / 4 : n, threads, max_blocks);
  hipLaunchKernelGGL((gated_kernel<SiluOp, false>), dim3(static_cast<unsigned>(blocks)),
                     dim3(threads), 0, s, n, x, static_cast<const float*>(nullptr), y, vec ? 1 : 0);
  return hipGetLastError();
}

hipError_t launch_swiglu(int64_t n, const float* g, const float* u, float* y, int threads,
                         int max_blocks, hipStream_t s) {
  const bool vec = aligned16(g) && aligned16(u) && aligned16(y);
  const int64_t blocks = ew_grid(vec ? (n + 3) / 4 : n, threads, max_blocks);
  hipLaunchKernelGGL((gated_kernel<SwigluOp, true>), dim3(static_cast<unsigned>(blocks)),
                     dim3(threads), 0, s, n, g, u, y, vec ? 1 : 0);
  return hipGetLastError();
}

hipError_t launch_swiglu_bwd(int64_t n, const float* g, const float* u, const float* dy, float* dg,
                             float* du, int threads, int max_blocks, hipStream_t s) {
  const bool vec = aligned16(g) && aligned16(u) && aligned16(dy) && aligned16(dg) && aligned16(du);
  const int64_t blocks = ew_grid(vec ? (n + 3) / 4 : n, threads, max_blocks);
  hipLaunchKernelGGL(swiglu_bwd_kernel, dim3(static_cast<unsigned>(blocks)), dim3(threads), 0, s, n,
                     g, u, dy, dg, du, vec ? 1 : 0);
  return hipGetLastError();
}

}  // namespace repops
