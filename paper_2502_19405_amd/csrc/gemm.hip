// Reproducible fp32 GEMM / batched GEMM for gfx950 (vector-ALU paths).
//
// Every output C[i][j] is one fixed sequence of binary32 operations, the
// blocked left-to-right contraction of the Verde paper's matrix-multiplication
// listing (Section 3.2) with block length k_block:
//     acc = +0
//     for each block of k_block consecutive k (ascending):
//         P = +0;  for k ascending in the block:  P = fma(A[i][k], B[k][j], P)
//         acc = acc + P
//     C = acc (* alpha) (+ bias[j])
// The output indices are spread over lanes, waves and workgroups freely; the
// k walk of one output always stays inside one lane, in ascending order, so
// tile sizes, launch shapes and operand layout cannot change a bit.  Zero
// padding past K adds fma(0, 0, P), which is P except for the sign of a zero:
// a block partial can be -0 (fma(a, b, +0) with a negative product below half
// the smallest subnormal rounds to -0), and fma(0, 0, -0) = +0.  The output
// cannot see that sign: every block partial is added into an accumulator that
// starts at +0, acc + (+0) and acc + (-0) are both acc when acc != 0, and
// +0 + (-0) = +0 under round-to-nearest, so acc is never -0 and takes the same
// bits whichever sign the zero partial had.
#include <hip/hip_runtime.h>

#include "gemm_store.h"
#include "repops_internal.h"

#pragma clang fp contract(off)

namespace repops {
namespace {

template <bool FUSED>
__device__ __forceinline__ float kstep(float a, float b, float p) {
  if constexpr (FUSED) {
    return __builtin_fmaf(a, b, p);
  } else {
    const float prod = a * b;
    return p + prod;
  }
}

// ---------------------------------------------------------------------------
// SIMPLE: one output per thread, operands straight from global memory.  Any
// block length; the reference-shaped GPU path.
// ---------------------------------------------------------------------------
template <bool FUSED>
__global__ __launch_bounds__(256) void gemm_simple_kernel(GemmArgs g, int64_t tiles_m,
                                                         int64_t tiles_n, int64_t ntiles) {
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  const int64_t blk = g.k_block > 0 ? g.k_block : g.k;
  for (int64_t t = blockIdx.x; t < ntiles; t += gridDim.x) {
    const int64_t tn = t % tiles_n;
    const int64_t tm = (t / tiles_n) % tiles_m;
    const int64_t bz = t / (tiles_n * tiles_m);
    const int64_t b1 = bz % g.batch1, b0 = bz / g.batch1;
    const int64_t i = tm * 16 + ty, j = tn * 16 + tx;
    if (i >= g.m || j >= g.n) continue;
    const float* A = g.A + b0 * g.sa0 + b1 * g.sa1;
    const float* B = g.B + b0 * g.sb0 + b1 * g.sb1;
    const float* a = g.ta ? A + i : A + i * g.lda;
    const int64_t ia = g.ta ? g.lda : 1;
    const float* b = g.tb ? B + j * g.ldb : B + j;
    const int64_t ib = g.tb ? 1 : g.ldb;
    float acc = 0.0f;
    for (int64_t k0 = 0; k0 < g.k; k0 += blk) {
      const int64_t k1 = (k0 + blk < g.k) ? k0 + blk : g.k;
      float p = 0.0f;
      for (int64_t kk = k0; kk < k1; ++kk) p = kstep<FUSED>(a[kk * ia], b[kk * ib], p);
      acc = acc + p;
    }
    const int64_t co = b0 * g.sc0 + b1 * g.sc1;
    gemm_store(g, g.C + co, g.G ? g.G + co : nullptr, g.gelu_in ? g.gelu_in + co : nullptr, i, j,
               acc);
  }
}

// ---------------------------------------------------------------------------
// TILED: BM x BN output tile per workgroup, BK-deep k slices staged through
// LDS (double buffered), TM x TN outputs per lane.  Needs k_block % BK == 0
// (or k_block == 0) so that block boundaries fall on slice boundaries.
// ---------------------------------------------------------------------------
template <int BM, int BN, int BK, int TM, int TN, bool FUSED>
__global__ __launch_bounds__((BM / TM) * (BN / TN)) void gemm_tiled_kernel(GemmArgs g,
                                                                        int64_t tiles_m,
                                                                        int64_t tiles_n,
                                                                        int64_t ntiles) {
  constexpr int NT = (BM / TM) * (BN / TN);
  constexpr int A_PER = BM * BK / NT;
  constexpr int B_PER = BK * BN / NT;
  static_assert(BM * BK % NT == 0 && BK * BN % NT == 0, "tile not divisible by threads");
  constexpr int PAD = 4;
  __shared__ float As[2][BK][BM + PAD];
  __shared__ float Bs[2][BK][BN + PAD];

  const int tid = threadIdx.x;
  const int tx = tid % (BN / TN), ty = tid / (BN / TN);
  const int64_t K = g.k;
  const int64_t nkt = (K + BK - 1) / BK;
  const int64_t slices_per_block = g.k_block > 0 ? g.k_block / BK : (nkt > 0 ? nkt : 1);

  for (int64_t t = blockIdx.x; t < ntiles; t += gridDim.x) {
    const int64_t tn = t % tiles_n;
    const int64_t tm = (t / tiles_n) % tiles_m;
    const int64_t bz = t / (tiles_n * tiles_m);
    const int64_t b1 = bz % g.batch1, b0 = bz / g.batch1;
    const int64_t m0 = tm * BM, n0 = tn * BN;
    const float* A = g.A + b0 * g.sa0 + b1 * g.sa1;
    const float* B = g.B + b0 * g.sb0 + b1 * g.sb1;

    float ra[A_PER], rb[B_PER];
    auto load = [&](int64_t k0) {
#pragma unroll
      for (int q = 0; q < A_PER; ++q) {
        const int e = tid + q * NT;
        int i, kk;
        if (g.ta) { kk = e / BM; i = e % BM; } else { i = e / BK; kk = e % BK; }
        const int64_t gi = m0 + i, gk = k0 + kk;
        float v = 0.0f;
        if (gi < g.m && gk < K) v = g.ta ? A[gk * g.lda + gi] : A[gi * g.lda + gk];
        ra[q] = v;
      }
#pragma unroll
      for (int q = 0; q < B_PER; ++q) {
        const int e = tid + q * NT;
        int j, kk;
        if (g.tb) { j = e / BK; kk = e % BK; } else { kk = e / BN; j = e % BN; }
        const int64_t gj = n0 + j, gk = k0 + kk;
        float v = 0.0f;
        if (gj < g.n && gk < K) v = g.tb ? B[gj * g.ldb + gk] : B[gk * g.ldb + gj];
        rb[q] = v;
      }
    };
    auto store = [&](int buf) {
#pragma unroll
      for (int q = 0; q < A_PER; ++q) {
        const int e = tid + q * NT;
        int i, kk;
        if (g.ta) { kk = e / BM; i = e % BM; } else { i = e / BK; kk = e % BK; }
        As[buf][kk][i] = ra[q];
      }
#pragma unroll
      for (int q = 0; q < B_PER; ++q) {
        const int e = tid + q * NT;
        int j, kk;
        if (g.tb) { j = e / BK; kk = e % BK; } else { kk = e / BN; j = e % BN; }
        Bs[buf][kk][j] = rb[q];
      }
    };

    float P[TM][TN], acc[TM][TN];
#pragma unroll
    for (int r = 0; r < TM; ++r)
#pragma unroll
      for (int c = 0; c < TN; ++c) { P[r][c] = 0.0f; acc[r][c] = 0.0f; }

    if (nkt > 0) {
      load(0);
      store(0);
    }
    __syncthreads();
    for (int64_t s = 0; s < nkt; ++s) {
      const int cur = static_cast<int>(s & 1);
      if (s + 1 < nkt) load((s + 1) * BK);
#pragma unroll
      for (int kk = 0; kk < BK; ++kk) {
        float a[TM], b[TN];
#pragma unroll
        for (int r = 0; r < TM; ++r) a[r] = As[cur][kk][ty * TM + r];
#pragma unroll
        for (int c = 0; c < TN; ++c) b[c] = Bs[cur][kk][tx * TN + c];
#pragma unroll
        for (int r = 0; r < TM; ++r)
#pragma unroll
          for (int c = 0; c < TN; ++c) P[r][c] = kstep<FUSED>(a[r], b[c], P[r][c]);
      }
      if (s + 1 < nkt) store(cur ^ 1);
      __syncthreads();
      if ((s + 1) % slices_per_block == 0 || s + 1 == nkt) {
#pragma unroll
        for (int r = 0; r < TM; ++r)
#pragma unroll
          for (int c = 0; c < TN; ++c) { acc[r][c] = acc[r][c] + P[r][c]; P[r][c] = 0.0f; }
      }
    }

    float* C = g.C + b0 * g.sc0 + b1 * g.sc1;
    float* G = g.G ? g.G + b0 * g.sc0 + b1 * g.sc1 : nullptr;
    const float* X = g.gelu_in ? g.gelu_in + b0 * g.sc0 + b1 * g.sc1 : nullptr;
#pragma unroll
    for (int r = 0; r < TM; ++r) {
      const int64_t i = m0 + ty * TM + r;
      if (i >= g.m) continue;
#pragma unroll
      for (int c = 0; c < TN; ++c) {
        const int64_t j = n0 + tx * TN + c;
        if (j < g.n) gemm_store(g, C, G, X, i, j, acc[r][c]);
      }
    }
  }
}

struct TiledEntry {
  GemmConfig cfg;
  int threads;
  void (*fused)(GemmArgs, int64_t, int64_t, int64_t);
  void (*unfused)(GemmArgs, int64_t, int64_t, int64_t);
};

#define REPOPS_TILED(BM, BN, BK, TM, TN)                                               \
  {{#BM "x" #BN "x" #BK "/" #TM "x" #TN, BM, BN, BK},                                  \
   (BM / TM) * (BN / TN),                                                              \
   gemm_tiled_kernel<BM, BN, BK, TM, TN, true>,                                        \
   gemm_tiled_kernel<BM, BN, BK, TM, TN, false>}

const TiledEntry kTiled[] = {
    REPOPS_TILED(64, 64, 16, 4, 4),
    REPOPS_TILED(128, 128, 16, 8, 8),
    REPOPS_TILED(128, 64, 32, 8, 4),
};
constexpr int kTiledCount = sizeof(kTiled) / sizeof(kTiled[0]);

int64_t grid_for(int64_t ntiles) {
  // Enough workgroups to cover every tile once, capped at what the hardware
  // grid allows; the kernels loop over the rest.
  const int64_t cap = int64_t(1) << 30;
  return ntiles < cap ? ntiles : cap;
}

}  // namespace

int gemm_tiled_count() { return kTiledCount; }
const GemmConfig* gemm_tiled_config(int index) {
  return (index >= 0 && index < kTiledCount) ? &kTiled[index].cfg : nullptr;
}

hipError_t launch_gemm_simple(const GemmArgs& g, hipStream_t s) {
  const int64_t tiles_m = (g.m + 15) / 16, tiles_n = (g.n + 15) / 16;
  const int64_t ntiles = tiles_m * tiles_n * g.batch0 * g.batch1;
  const dim3 grid(static_cast<unsigned>(grid_for(ntiles)));
  if (g.fused)
    hipLaunchKernelGGL(gemm_simple_kernel<true>, grid, dim3(256), 0, s, g, tiles_m, tiles_n, ntiles);
  else
    hipLaunchKernelGGL(gemm_simple_kernel<false>, grid, dim3(256), 0, s, g, tiles_m, tiles_n, ntiles);
  return hipGetLastError();
}

hipError_t launch_gemm_tiled(const GemmArgs& g, int index, hipStream_t s) {
  const TiledEntry& e = kTiled[index];
  const int64_t tiles_m = (g.m + e.cfg.bm - 1) / e.cfg.bm;
  const int64_t tiles_n = (g.n + e.cfg.bn - 1) / e.cfg.bn;
  const int64_t ntiles = tiles_m * tiles_n * g.batch0 * g.batch1;
  const dim3 grid(static_cast<unsigned>(grid_for(ntiles)));
  hipLaunchKernelGGL(g.fused ? e.fused : e.unfused, grid, dim3(e.threads), 0, s, g, tiles_m,
                     tiles_n, ntiles);
  return hipGetLastError();
}

}  // namespace repops

