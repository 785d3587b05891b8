// Reproducible fp32 GEMM on the gfx950 matrix cores.
//
// v_mfma_f32_32x32x1_2b_f32 adds ONE product to each of its 2 x 32 x 32
// accumulators: D[i][j] = C[i][j] + A[i] * B[j], rounded once.  A chain of
// these instructions over ascending k is therefore exactly the fused
// multiply-add chain P = fma(a_k, b_k, P) of the canonical contraction
// (Verde, Section 3.2 listing, with the blocked left-to-right reading): each
// output still sees its k terms one at a time, in order, in one lane.  The
// equality with the vector fma chain -- including subnormal products and
// operands, overflow, signed zeros and the fused-versus-unfused case -- is
// checked by the GPU tests through this kernel against the CPU oracle.  The
// multi-term variants (K > 1 per instruction) sum several products inside
// the unit and are never used.
//
// Tiling: a workgroup of WM x WN waves owns a BM x BN output tile; each wave
// owns (BM/WM) x (BN/WN) outputs as instruction tiles of 64 rows x 32
// columns (the instruction's two 32 x 32 blocks stacked along rows, both
// reading the same 32 B columns).  k advances in BK-deep slices staged
// through double-buffered LDS.  Every k_block steps the block partials P are
// added into the accumulators (acc = acc + P, vector adds) and the next
// block starts from +0.
#include <hip/hip_runtime.h>

#include "repops_internal.h"

#pragma clang fp contract(off)

namespace repops {
namespace {

typedef float v32f __attribute__((ext_vector_type(32)));

__device__ __forceinline__ float epilogue(const GemmArgs& g, float acc, int64_t j) {
  float v = acc;
  if (g.has_alpha) v = v * g.alpha;
  if (g.bias) v = v + g.bias[j];
  return v;
}

// Map the launch-order tile index so that the tiles one XCD receives (the
// hardware deals workgroups round-robin over 8 XCDs) form a compact panel of
// GROUP_M tile rows, which share A and B slices in that XCD's L2.
__device__ __forceinline__ void tile_coords(int64_t t, int64_t ntiles, int64_t tiles_m,
                                            int64_t tiles_n, int64_t* bz, int64_t* tm,
                                            int64_t* tn) {
  constexpr int64_t kXcd = 8, kGroupM = 4;
  if (ntiles % kXcd == 0) t = (t % kXcd) * (ntiles / kXcd) + t / kXcd;
  const int64_t per_batch = tiles_m * tiles_n;
  *bz = t / per_batch;
  const int64_t r = t % per_batch;
  const int64_t group = r / (kGroupM * tiles_n);
  const int64_t first_m = group * kGroupM;
  const int64_t gsize = (tiles_m - first_m) < kGroupM ? (tiles_m - first_m) : kGroupM;
  const int64_t in_group = r % (kGroupM * tiles_n);
  *tm = first_m + in_group % gsize;
  *tn = in_group / gsize;
}

template <int BM, int BN, int BK, int WM, int WN>
__global__ __launch_bounds__(64 * WM * WN) void gemm_mfma_kernel(GemmArgs g, int64_t tiles_m,
                                                                 int64_t tiles_n, int64_t ntiles,
                                                                 int a_vec, int b_vec) {
  constexpr int NT = 64 * WM * WN;
  constexpr int TWM = BM / WM, TWN = BN / WN;  // wave tile
  constexpr int IM = TWM / 64, IN = TWN / 32;  // instruction tiles per wave
  static_assert(TWM % 64 == 0 && TWN % 32 == 0, "wave tile must hold whole instruction tiles");
  static_assert(BK % 4 == 0, "k slice must hold whole float4 groups");
  constexpr int PAD = 4;
  constexpr int AV = BM * BK / 4 / NT;  // float4 groups per thread and slice
  constexpr int BV = BK * BN / 4 / NT;
  static_assert(AV * NT * 4 == BM * BK && BV * NT * 4 == BK * BN, "slice not divisible");
  __shared__ float As[2][BK][BM + PAD];
  __shared__ float Bs[2][BK][BN + PAD];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm0 = (wave / WN) * TWM;
  const int wn0 = (wave % WN) * TWN;
  const int64_t K = g.k;
  const int64_t nslices = (K + BK - 1) / BK;
  const int64_t slices_per_block = g.k_block > 0 ? g.k_block / BK : (nslices > 0 ? nslices : 1);

  for (int64_t t = blockIdx.x; t < ntiles; t += gridDim.x) {
    int64_t bz, tm, tn;
    tile_coords(t, ntiles, tiles_m, tiles_n, &bz, &tm, &tn);
    const int64_t b1 = bz % g.batch1, b0 = bz / g.batch1;
    const int64_t m0 = tm * BM, n0 = tn * BN;
    const float* A = g.A + b0 * g.sa0 + b1 * g.sa1;
    const float* B = g.B + b0 * g.sb0 + b1 * g.sb1;

    float4 ra[AV], rb[BV];
    // Global -> registers for slice k0.  Element (row, k) of the logical A
    // lands in As[k][row]; element (k, col) of B in Bs[k][col].  Groups of 4
    // run along the stored contiguous dimension.
    auto load = [&](int64_t k0) {
#pragma unroll
      for (int q = 0; q < AV; ++q) {
        const int e = tid + q * NT;
        float v[4];
        if (!g.ta) {  // A row-major: groups along k
          const int i = e / (BK / 4), kq = (e % (BK / 4)) * 4;
          const int64_t gi = m0 + i, gk = k0 + kq;
          const float* p = A + gi * g.lda + gk;
          if (a_vec && gi < g.m && gk + 4 <= K) {
            const float4 f = *reinterpret_cast<const float4*>(p);
            v[0] = f.x; v[1] = f.y; v[2] = f.z; v[3] = f.w;
          } else {
#pragma unroll
            for (int c = 0; c < 4; ++c) v[c] = (gi < g.m && gk + c < K) ? p[c] : 0.0f;
          }
        } else {  // A stored k x m: groups along m
          const int kk = e / (BM / 4), i = (e % (BM / 4)) * 4;
          const int64_t gi = m0 + i, gk = k0 + kk;
          const float* p = A + gk * g.lda + gi;
          if (a_vec && gk < K && gi + 4 <= g.m) {
            const float4 f = *reinterpret_cast<const float4*>(p);
            v[0] = f.x; v[1] = f.y; v[2] = f.z; v[3] = f.w;
          } else {
#pragma unroll
            for (int c = 0; c < 4; ++c) v[c] = (gk < K && gi + c < g.m) ? p[c] : 0.0f;
          }
        }
        ra[q] = make_float4(v[0], v[1], v[2], v[3]);
      }
#pragma unroll
      for (int q = 0; q < BV; ++q) {
        const int e = tid + q * NT;
        float v[4];
        if (!g.tb) {  // B row-major: groups along n
          const int kk = e / (BN / 4), j = (e % (BN / 4)) * 4;
          const int64_t gj = n0 + j, gk = k0 + kk;
          const float* p = B + gk * g.ldb + gj;
          if (b_vec && gk < K && gj + 4 <= g.n) {
            const float4 f = *reinterpret_cast<const float4*>(p);
            v[0] = f.x; v[1] = f.y; v[2] = f.z; v[3] = f.w;
          } else {
#pragma unroll
            for (int c = 0; c < 4; ++c) v[c] = (gk < K && gj + c < g.n) ? p[c] : 0.0f;
          }
        } else {  // B stored n x k: groups along k
          const int j = e / (BK / 4), kq = (e % (BK / 4)) * 4;
          const int64_t gj = n0 + j, gk = k0 + kq;
          const float* p = B + gj * g.ldb + gk;
          if (b_vec && gj < g.n && gk + 4 <= K) {
            const float4 f = *reinterpret_cast<const float4*>(p);
            v[0] = f.x; v[1] = f.y; v[2] = f.z; v[3] = f.w;
          } else {
#pragma unroll
            for (int c = 0; c < 4; ++c) v[c] = (gj < g.n && gk + c < K) ? p[c] : 0.0f;
          }
        }
        rb[q] = make_float4(v[0], v[1], v[2], v[3]);
      }
    };
    auto store = [&](int buf) {
#pragma unroll
      for (int q = 0; q < AV; ++q) {
        const int e = tid + q * NT;
        if (!g.ta) {
          const int i = e / (BK / 4), kq = (e % (BK / 4)) * 4;
          As[buf][kq + 0][i] = ra[q].x;
          As[buf][kq + 1][i] = ra[q].y;
          As[buf][kq + 2][i] = ra[q].z;
          As[buf][kq + 3][i] = ra[q].w;
        } else {
          const int kk = e / (BM / 4), i = (e % (BM / 4)) * 4;
          *reinterpret_cast<float4*>(&As[buf][kk][i]) = ra[q];
        }
      }
#pragma unroll
      for (int q = 0; q < BV; ++q) {
        const int e = tid + q * NT;
        if (!g.tb) {
          const int kk = e / (BN / 4), j = (e % (BN / 4)) * 4;
          *reinterpret_cast<float4*>(&Bs[buf][kk][j]) = rb[q];
        } else {
          const int j = e / (BK / 4), kq = (e % (BK / 4)) * 4;
          Bs[buf][kq + 0][j] = rb[q].x;
          Bs[buf][kq + 1][j] = rb[q].y;
          Bs[buf][kq + 2][j] = rb[q].z;
          Bs[buf][kq + 3][j] = rb[q].w;
        }
      }
    };

    v32f P[IM][IN], acc[IM][IN];
#pragma unroll
    for (int a = 0; a < IM; ++a)
#pragma unroll
      for (int b = 0; b < IN; ++b) {
        P[a][b] = v32f{};
        acc[a][b] = v32f{};
      }

    if (nslices > 0) {
      load(0);
      store(0);
    }
    __syncthreads();
    for (int64_t s = 0; s < nslices; ++s) {
      const int cur = static_cast<int>(s & 1);
      if (s + 1 < nslices) load((s + 1) * BK);
#pragma unroll
      for (int kk = 0; kk < BK; ++kk) {
        float av[IM], bv[IN];
#pragma unroll
        for (int a = 0; a < IM; ++a) av[a] = As[cur][kk][wm0 + a * 64 + lane];
#pragma unroll
        for (int b = 0; b < IN; ++b) bv[b] = Bs[cur][kk][wn0 + b * 32 + (lane & 31)];
#pragma unroll
        for (int a = 0; a < IM; ++a)
#pragma unroll
          for (int b = 0; b < IN; ++b)
            P[a][b] = __builtin_amdgcn_mfma_f32_32x32x1f32(av[a], bv[b], P[a][b], 0, 0, 0);
      }
      if (s + 1 < nslices) store(cur ^ 1);
      __syncthreads();
      if ((s + 1) % slices_per_block == 0 || s + 1 == nslices) {
#pragma unroll
        for (int a = 0; a < IM; ++a)
#pragma unroll
          for (int b = 0; b < IN; ++b) {
            acc[a][b] = acc[a][b] + P[a][b];
            P[a][b] = v32f{};
          }
      }
    }

    // Accumulator layout of the instruction (lane l, register r): block
    // r / 16 covers rows 32*(r/16) + [0, 32); inside it row
    // 8*((r%16)/4) + 4*(l/32) + r%4 and column l % 32.
    float* C = g.C + b0 * g.sc0 + b1 * g.sc1;
#pragma unroll
    for (int a = 0; a < IM; ++a)
#pragma unroll
      for (int b = 0; b < IN; ++b) {
        const int64_t j = n0 + wn0 + b * 32 + (lane & 31);
#pragma unroll
        for (int r = 0; r < 32; ++r) {
          const int row = 32 * (r / 16) + 8 * ((r % 16) / 4) + 4 * (lane / 32) + (r % 4);
          const int64_t i = m0 + wm0 + a * 64 + row;
          if (i < g.m && j < g.n) C[i * g.ldc + j] = epilogue(g, acc[a][b][r], j);
        }
      }
  }
}

struct MfmaEntry {
  GemmConfig cfg;
  int threads;
  void (*kernel)(GemmArgs, int64_t, int64_t, int64_t, int, int);
};

#define REPOPS_MFMA(BM, BN, BK, WM, WN)                                                       \
  {{#BM "x" #BN "x" #BK "/w" #WM "x" #WN, BM, BN, BK}, 64 * WM * WN,                          \
   gemm_mfma_kernel<BM, BN, BK, WM, WN>}

const MfmaEntry kMfma[] = {
    REPOPS_MFMA(128, 128, 16, 2, 2),
    REPOPS_MFMA(128, 64, 16, 2, 2),
    REPOPS_MFMA(256, 128, 16, 4, 2),
    REPOPS_MFMA(64, 64, 16, 1, 2),
};
constexpr int kMfmaCount = sizeof(kMfma) / sizeof(kMfma[0]);

bool aligned16(const void* p) { return reinterpret_cast<uintptr_t>(p) % 16 == 0; }

}  // namespace

int gemm_mfma_count() { return kMfmaCount; }
const GemmConfig* gemm_mfma_config(int index) {
  return (index >= 0 && index < kMfmaCount) ? &kMfma[index].cfg : nullptr;
}

hipError_t launch_gemm_mfma(const GemmArgs& g, int index, hipStream_t s) {
  const MfmaEntry& e = kMfma[index];
  const int64_t tiles_m = (g.m + e.cfg.bm - 1) / e.cfg.bm;
  const int64_t tiles_n = (g.n + e.cfg.bn - 1) / e.cfg.bn;
  const int64_t ntiles = tiles_m * tiles_n * g.batch0 * g.batch1;
  const int64_t cap = int64_t(1) << 30;
  const unsigned grid = static_cast<unsigned>(ntiles < cap ? ntiles : cap);
  // float4 loads need 16-byte aligned rows and batch origins
  const int a_vec = aligned16(g.A) && g.lda % 4 == 0 && g.sa0 % 4 == 0 && g.sa1 % 4 == 0;
  const int b_vec = aligned16(g.B) && g.ldb % 4 == 0 && g.sb0 % 4 == 0 && g.sb1 % 4 == 0;
  hipLaunchKernelGGL(e.kernel, dim3(grid), dim3(e.threads), 0, s, g, tiles_m, tiles_n, ntiles,
                     a_vec, b_vec);
  return hipGetLastError();
}

}  // namespace repops
