// Row-reduction building blocks shared by the forward and backward row
// kernels: the strided tree with W = 64 on one 64-lane wave, the order-free
// wave maximum, and the LDS-based reduction for any row width and combine
// mode.  The orders are those of the order descriptor (strided tree: x_j into
// partial q[j mod W] in ascending j, then a halving tree; blocked: partials of
// W consecutive terms added left to right).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#pragma clang fp contract(off)

namespace repops {

constexpr int kWave = 64;
constexpr int kMaxPerLane = 64;  // register-resident rows: cols <= 64 * 64

// This thread's wave within the workgroup, as a value the compiler knows to be
// uniform over the wave: per-row scalars indexed by it are then read with
// scalar loads, which the vector-load counter does not wait for.
__device__ __forceinline__ int wave_id() {
  return __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x >> 6));
}

// Cross-lane reads done in registers.  After lane_hi32(v), lane l < 32 holds
// v[l + 32]; after lane_hi16(v), lane l of lanes 0..15 (and 32..47) holds
// v[l + 16] (the gfx950 permute-swaps exchange the upper half of one operand
// with the lower half of the other).  lane_down<D>(v), D in {1, 2, 4, 8},
// gives lane l the value of lane l + D within its row of 16 lanes (a DPP row
// shift; lanes whose source leaves the row read +0).  Unlike __shfl these
// never go through the LDS crossbar.  The wave must have all 64 lanes active.
__device__ __forceinline__ float lane_hi32(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v),
                                                  false, false);
  return __uint_as_float(r[1]);
}
__device__ __forceinline__ float lane_hi16(float v) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v),
                                                  false, false);
  return __uint_as_float(r[1]);
}
template <int D>
__device__ __forceinline__ float lane_down(float v) {
  static_assert(D == 1 || D == 2 || D == 4 || D == 8, "row shift of 1, 2, 4 or 8 lanes");
  // DPP control 0x100 + D: row_shl by D; all rows and banks written.
  return __int_as_float(
      __builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x100 + D, 0xf, 0xf, false));
}
__device__ __forceinline__ float wave_broadcast0(float v) {
  return __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(v)));
}

// Halving tree over the 64 lane partials: after the step with distance s, lane
// l < s holds q[l] + q[l+s].  Lanes >= s keep values that no later step reads.
// Every lane returns q[0].  (An IEEE sum is commutative, so the compiler may
// place the moved operand first.)  Called with all 64 lanes active.
__device__ __forceinline__ float wave_tree_sum(float q) {
  q = q + lane_hi32(q);
  q = q + lane_hi16(q);
  q = q + lane_down<8>(q);
  q = q + lane_down<4>(q);
  q = q + lane_down<2>(q);
  q = q + lane_down<1>(q);
  return wave_broadcast0(q);
}

// Maximum over the wave (order-free up to the sign of a zero maximum, which
// cannot change any softmax output: x - (+0) and x - (-0) differ only for
// x = -0, and exp_rep(+0) = exp_rep(-0) = 1).  Same data movement as the tree
// sum, so lane 0 ends with the maximum of all 64 lanes; every lane returns it.
// Called with all 64 lanes active.
__device__ __forceinline__ float wave_max(float m) {
  auto mx = [](float a, float b) { return b > a ? b : a; };
  m = mx(m, lane_hi32(m));
  m = mx(m, lane_hi16(m));
  m = mx(m, lane_down<8>(m));
  m = mx(m, lane_down<4>(m));
  m = mx(m, lane_down<2>(m));
  m = mx(m, lane_down<1>(m));
  return wave_broadcast0(m);
}

// Per-lane chains continued across the S waves of a workgroup, in wave order:
// wave k starts from what wave k - 1 left in chain[lane] (+0 for wave 0),
// folds its own terms in with `step`, and leaves the result there.  Every
// wave returns the finished chains.  All waves of the workgroup must call it
// (it holds S barriers); a following use of the same array needs a barrier
// first, since waves read the finished chains after the last one.
template <class Step>
__device__ __forceinline__ float chain_across_waves(float* chain, int lane, int w, int S,
                                                    Step step) {
  for (int k = 0; k < S; ++k) {
    if (w == k) chain[lane] = step(k > 0 ? chain[lane] : 0.0f);
    __syncthreads();
  }
  return chain[lane];
}

// Workgroup barrier that waits for this wave's LDS operations only: global
// loads issued before it stay in flight (__syncthreads would also wait for
// them).  The memory clobber keeps LDS accesses on their side of the barrier.
__device__ __forceinline__ void lds_only_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

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

}  // namespace repops
