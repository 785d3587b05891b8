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

#include "gemm_store.h"
#include "repops_internal.h"

#pragma clang fp contract(off)

namespace repops {
namespace {

typedef float v32f __attribute__((ext_vector_type(32)));

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

// Causal products (per batch element, row i, column j, contraction index kk).
// causal == 1: only outputs with j <= i are wanted, so a tile whose first
// column lies past its last row is skipped (its outputs are left unwritten).
// causal == 2: A is zero at kk > i, so a row tile starting at m0 needs k only
// up to the end of the k block holding row m0 + bm - 1's diagonal; every later
// block is a chain of zero products, whose partial is +0 and leaves acc
// unchanged (acc + (+0) = acc; acc is never -0), so skipping it keeps the bits.
__device__ __forceinline__ bool tile_above_diagonal(const GemmArgs& g, int64_t m0, int bm,
                                                    int64_t n0) {
  return g.causal == 1 && n0 > m0 + bm - 1;
}

__device__ __forceinline__ int64_t k_extent(const GemmArgs& g, int64_t m0, int bm) {
  if (g.causal != 2 || g.k_block <= 0) return g.k;
  const int64_t end = (m0 + bm + g.k_block - 1) / g.k_block * g.k_block;
  return end < g.k ? end : g.k;
}

// With causal == 1, square tiles and at least as many tile columns as rows,
// the launch covers only the tiles at or below each batch element's diagonal
// (tn <= tm): tile r of a batch element is the r-th of the lower triangle in
// row order.
__device__ __host__ __forceinline__ bool causal_triangle(int causal, int bm, int bn,
                                                         int64_t tiles_m, int64_t tiles_n) {
  return causal == 1 && bm == bn && tiles_n >= tiles_m;
}

// Tile of launch index t for any product: the lower triangle's tiles only (see
// causal_triangle), or every tile with tile_coords -- row tiles in reverse order
// when A is zero above its diagonal (causal == 2), so that the row tiles with
// the longest contraction start first.
__device__ __forceinline__ void tile_of(const GemmArgs& g, int bm, int bn, int64_t t,
                                        int64_t ntiles, int64_t tiles_m, int64_t tiles_n,
                                        int64_t* bz, int64_t* tm, int64_t* tn) {
  if (causal_triangle(g.causal, bm, bn, tiles_m, tiles_n)) {
    constexpr int64_t kXcd = 8;
    if (ntiles % kXcd == 0) t = (t % kXcd) * (ntiles / kXcd) + t / kXcd;
    const int64_t per = tiles_m * (tiles_m + 1) / 2;
    *bz = t / per;
    const int64_t r = t % per;
    // the last row tile whose triangle starts at or before r (integer
    // bisection; r < per, so it lies below tiles_m)
    int64_t row = 0, hi = tiles_m - 1;
    while (row < hi) {
      const int64_t mid = (row + hi + 1) / 2;
      if (mid * (mid + 1) / 2 <= r) row = mid; else hi = mid - 1;
    }
    *tm = row;
    *tn = r - row * (row + 1) / 2;
    return;
  }
  tile_coords(t, ntiles, tiles_m, tiles_n, bz, tm, tn);
  if (g.causal == 2) *tm = tiles_m - 1 - *tm;
}

template <int BM, int BN, int BK, int WM, int WN, bool TA, bool TB>
struct MfmaTile {
  static constexpr int NT = 64 * WM * WN;
  static constexpr int TWM = BM / WM, TWN = BN / WN;  // wave tile
  static constexpr int IM = TWM / 64, IN = TWN / 32;  // instruction tiles per wave
  static_assert(TWM % 64 == 0 && TWN % 32 == 0, "wave tile must hold whole instruction tiles");
  static_assert(BK % 4 == 0, "k slice must hold whole float4 groups");
  static constexpr int PAD = 4;
  static constexpr int AV = BM * BK / 4 / NT;  // float4 groups per thread and slice
  static constexpr int BV = BK * BN / 4 / NT;
  static_assert(AV * NT * 4 == BM * BK && BV * NT * 4 == BK * BN, "slice not divisible");

  struct Smem {
    float a[2][BK][BM + PAD];
    float b[2][BK][BN + PAD];
  };

  // Coordinates of float4 group q of this thread inside the A / B slice.
  // Groups run along the stored contiguous dimension: k for row-major A and
  // for transposed B, m for transposed A, n for row-major B.
  __device__ static void a_group(int e, int* row, int* kk) {
    if constexpr (!TA) { *row = e / (BK / 4); *kk = (e % (BK / 4)) * 4; }
    else { *kk = e / (BM / 4); *row = (e % (BM / 4)) * 4; }
  }
  __device__ static void b_group(int e, int* col, int* kk) {
    if constexpr (!TB) { *kk = e / (BN / 4); *col = (e % (BN / 4)) * 4; }
    else { *col = e / (BK / 4); *kk = (e % (BK / 4)) * 4; }
  }

  template <bool EDGE>
  __device__ static float4 fetch4(const float* p, bool in0, int valid) {
    // valid: how many of the 4 consecutive elements exist (EDGE only)
    if constexpr (!EDGE) {
      return *reinterpret_cast<const float4*>(p);
    } else {
      float v[4];
#pragma unroll
      for (int c = 0; c < 4; ++c) v[c] = (in0 && c < valid) ? p[c] : 0.0f;
      return make_float4(v[0], v[1], v[2], v[3]);
    }
  }

  template <bool EDGE>
  __device__ static void load(const GemmArgs& g, const float* A, const float* B, int64_t m0,
                              int64_t n0, int64_t k0, int tid, float4* ra, float4* rb) {
#pragma unroll
    for (int q = 0; q < AV; ++q) {
      int row, kk;
      a_group(tid + q * NT, &row, &kk);
      const int64_t gi = m0 + row, gk = k0 + kk;
      if constexpr (!TA) {
        ra[q] = fetch4<EDGE>(A + gi * g.lda + gk, gi < g.m, static_cast<int>(g.k - gk));
      } else {
        ra[q] = fetch4<EDGE>(A + gk * g.lda + gi, gk < g.k, static_cast<int>(g.m - gi));
      }
    }
#pragma unroll
    for (int q = 0; q < BV; ++q) {
      int col, kk;
      b_group(tid + q * NT, &col, &kk);
      const int64_t gj = n0 + col, gk = k0 + kk;
      if constexpr (!TB) {
        rb[q] = fetch4<EDGE>(B + gk * g.ldb + gj, gk < g.k, static_cast<int>(g.n - gj));
      } else {
        rb[q] = fetch4<EDGE>(B + gj * g.ldb + gk, gj < g.n, static_cast<int>(g.k - gk));
      }
    }
  }

  __device__ static void store(Smem& sm, int buf, int tid, const float4* ra, const float4* rb) {
#pragma unroll
    for (int q = 0; q < AV; ++q) {
      int row, kk;
      a_group(tid + q * NT, &row, &kk);
      if constexpr (!TA) {
        sm.a[buf][kk + 0][row] = ra[q].x;
        sm.a[buf][kk + 1][row] = ra[q].y;
        sm.a[buf][kk + 2][row] = ra[q].z;
        sm.a[buf][kk + 3][row] = ra[q].w;
      } else {
        *reinterpret_cast<float4*>(&sm.a[buf][kk][row]) = ra[q];
      }
    }
#pragma unroll
    for (int q = 0; q < BV; ++q) {
      int col, kk;
      b_group(tid + q * NT, &col, &kk);
      if constexpr (!TB) {
        *reinterpret_cast<float4*>(&sm.b[buf][kk][col]) = rb[q];
      } else {
        sm.b[buf][kk + 0][col] = rb[q].x;
        sm.b[buf][kk + 1][col] = rb[q].y;
        sm.b[buf][kk + 2][col] = rb[q].z;
        sm.b[buf][kk + 3][col] = rb[q].w;
      }
    }
  }

  // One BK-deep slice of single-term updates.  FIRST: the slice opens a new
  // k block, so its first update starts the block partial from +0.
  template <bool FIRST>
  __device__ static void slice(const Smem& sm, int buf, int lane, int wm0, int wn0,
                               v32f (&P)[IM][IN]) {
    const v32f zero = {};
#pragma unroll
    for (int kk = 0; kk < BK; ++kk) {
      float av[IM], bv[IN];
#pragma unroll
      for (int a = 0; a < IM; ++a) av[a] = sm.a[buf][kk][wm0 + a * 64 + lane];
#pragma unroll
      for (int b = 0; b < IN; ++b) bv[b] = sm.b[buf][kk][wn0 + b * 32 + (lane & 31)];
#pragma unroll
      for (int a = 0; a < IM; ++a)
#pragma unroll
        for (int b = 0; b < IN; ++b)
          P[a][b] = __builtin_amdgcn_mfma_f32_32x32x1f32(
              av[a], bv[b], (FIRST && kk == 0) ? zero : P[a][b], 0, 0, 0);
    }
  }

  template <bool EDGE>
  __device__ static void run(const GemmArgs& g, Smem& sm, int64_t b0, int64_t b1, int64_t m0,
                             int64_t n0) {
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm0 = (wave / WN) * TWM;
    const int wn0 = (wave % WN) * TWN;
    const int64_t K = k_extent(g, m0, BM);
    const int64_t nslices = (K + BK - 1) / BK;
    const int64_t spb = g.k_block > 0 ? g.k_block / BK : (nslices > 0 ? nslices : 1);
    const float* A = g.A + b0 * g.sa0 + b1 * g.sa1;
    const float* B = g.B + b0 * g.sb0 + b1 * g.sb1;

    v32f P[IM][IN], acc[IM][IN];
#pragma unroll
    for (int a = 0; a < IM; ++a)
#pragma unroll
      for (int b = 0; b < IN; ++b) {
        P[a][b] = v32f{};
        acc[a][b] = v32f{};
      }
    float4 ra[AV], rb[BV];
    if (nslices > 0) {
      load<EDGE>(g, A, B, m0, n0, 0, tid, ra, rb);
      store(sm, 0, tid, ra, rb);
    }
    __syncthreads();
    for (int64_t s = 0; s < nslices; ++s) {
      const int cur = static_cast<int>(s & 1);
      if (s + 1 < nslices) load<EDGE>(g, A, B, m0, n0, (s + 1) * BK, tid, ra, rb);
      if (s % spb == 0) slice<true>(sm, cur, lane, wm0, wn0, P);
      else slice<false>(sm, cur, lane, wm0, wn0, P);
      if (s + 1 < nslices) store(sm, cur ^ 1, tid, ra, rb);
      if ((s + 1) % spb == 0 || s + 1 == nslices) {
#pragma unroll
        for (int a = 0; a < IM; ++a)
#pragma unroll
          for (int b = 0; b < IN; ++b) acc[a][b] = acc[a][b] + P[a][b];
      }
      __syncthreads();
    }

    // Accumulator layout of the instruction (lane l, register r): block
    // r / 16 covers rows 32*(r/16) + [0, 32); inside it row
    // 8*((r%16)/4) + 4*(l/32) + r%4 and column l % 32.
    float* C = g.C + b0 * g.sc0 + b1 * g.sc1;
    float* G = g.G ? g.G + b0 * g.sc0 + b1 * g.sc1 : nullptr;
    const float* X = g.gelu_in ? g.gelu_in + b0 * g.sc0 + b1 * g.sc1 : nullptr;
#pragma unroll
    for (int a = 0; a < IM; ++a)
#pragma unroll
      for (int b = 0; b < IN; ++b) {
        const int64_t j = n0 + wn0 + b * 32 + (lane & 31);
#pragma unroll
        for (int r = 0; r < 32; ++r) {
          const int row = 32 * (r / 16) + 8 * ((r % 16) / 4) + 4 * (lane / 32) + (r % 4);
          const int64_t i = m0 + wm0 + a * 64 + row;
          if (!EDGE || (i < g.m && j < g.n)) gemm_store(g, C, G, X, i, j, acc[a][b][r]);
        }
      }
  }
};

template <int BM, int BN, int BK, int WM, int WN, int MINW, bool TA, bool TB>
__global__ __launch_bounds__(64 * WM * WN, MINW) void gemm_mfma_kernel(GemmArgs g, int64_t tiles_m,
                                                                 int64_t tiles_n, int64_t ntiles,
                                                                 int vec_ok) {
  using T = MfmaTile<BM, BN, BK, WM, WN, TA, TB>;
  __shared__ typename T::Smem sm;
  for (int64_t t = blockIdx.x; t < ntiles; t += gridDim.x) {
    int64_t bz, tm, tn;
    tile_of(g, BM, BN, t, ntiles, tiles_m, tiles_n, &bz, &tm, &tn);
    const int64_t b1 = bz % g.batch1, b0 = bz / g.batch1;
    const int64_t m0 = tm * BM, n0 = tn * BN;
    if (tile_above_diagonal(g, m0, BM, n0)) continue;  // uniform over the workgroup
    // Interior tiles (whole tile inside C, whole k slices, aligned rows) take
    // the path without per-element checks; the choice is uniform per tile.
    const bool interior = vec_ok && m0 + BM <= g.m && n0 + BN <= g.n && g.k % BK == 0;
    if (interior) T::template run<false>(g, sm, b0, b1, m0, n0);
    else T::template run<true>(g, sm, b0, b1, m0, n0);
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// Staged variant: operands go from global memory straight into LDS
// (global_load_lds_dwordx4: each lane's 16 bytes land at base + lane * 16),
// through an NS-deep ring of 16-deep k slices, so several slices are in
// flight without holding them in registers.  Instruction tiles are 32 rows x
// 64 columns here (the instruction's two 32 x 32 blocks side by side along
// columns, both reading the same 32 A rows).
//
// LDS forms of one slice (16 k values):
//   k-packed: [4 groups of 4 k][rows][4]: a lane reads its row's 4 k values
//     with one 16-byte LDS read (row-major A; transposed B);
//   k-major:  [16 k][rows]: a lane reads one value per k (transposed A;
//     row-major B), two k at once with a paired read.
// Rows past M (columns past N) are loaded from the last valid row (column):
// they only feed outputs that are never stored.  K must be a multiple of BK,
// rows 16-byte aligned and the k-major operand's row count (N of row-major B,
// M of transposed A) a multiple of 4; otherwise the register-staged kernel of
// the same tile shape runs.
//
// Pipelining (a wave may be the only one on its SIMD, so whatever it does
// between two matrix steps idles the matrix unit unless it fits inside the
// 16 passes of the step before): each group of 4 k issues the LDS reads of
// the next group right after its own first step; one workgroup barrier per
// slice, placed inside the slice's last group, publishes the next slice and
// frees the slot just read for the slice NS ahead; slot and block positions
// are counters, not divisions.  With the default 64-deep k blocks the loop
// body is one turn of the ring, unrolled, with no branches (see slice<>).
// ---------------------------------------------------------------------------
typedef float v4f __attribute__((ext_vector_type(4)));

// s_waitcnt with only the vector-memory counter bounded (gfx9 encoding:
// vmcnt in bits 3:0 and 15:14, expcnt 6:4 and lgkmcnt 11:8 left at maximum).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}
typedef __attribute__((address_space(3))) void* lds_void_ptr;
typedef __attribute__((address_space(1))) void* global_void_ptr;

// Workgroup barrier that waits for this wave's LDS reads and writes only.
// Unlike __syncthreads() it does not wait for outstanding global-to-LDS
// loads (later slices stay in flight); the slice about to be read is waited
// for explicitly with wait_vmcnt before it.  The memory clobber keeps the
// compiler from moving memory accesses across it.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// DUAL: a second set of block partials, so that each 64-deep block's adds into
// acc are spread over the next block's matrix steps (the staged kernel uses it
// where a wave owns one instruction tile).
// GELU_OUT: the epilogue can write the GELU of the output (repops_matmul_gelu);
// the grouped kernel, which never does, leaves that path out (with both GELU
// paths its four tile forms together spilled registers).
// EPI: interior tiles take the specialised stores (store_plain); without it every
// output goes through the checked loop -- the form kept for products with no
// scale, bias or GELU array, whose kernels the added store code would otherwise
// change (register assignment and the schedule of the matrix loop).
template <int BM, int BN, int BK, int WM, int WN, int NS, bool TA, bool TB, bool DUAL,
          bool GELU_OUT = true, bool RING = false, bool EPI = true>
struct StagedTile {
  static_assert(BK % 16 == 0, "k slices hold whole 16-step groups");
  static constexpr int NW = WM * WN;
  static constexpr int TWM = BM / WM, TWN = BN / WN;
  static constexpr int IM = TWM / 32, IN = TWN / 64;
  static_assert(TWM % 32 == 0 && TWN % 64 == 0, "wave tile must hold whole instruction tiles");
  static constexpr int A_FLOATS = BM * BK, B_FLOATS = BN * BK;
  static constexpr int A_LOADS = A_FLOATS / 256, B_LOADS = B_FLOATS / 256;  // wave loads per slice
  static_assert(A_LOADS % NW == 0 && B_LOADS % NW == 0, "slice loads must split evenly over waves");
  static_assert(BM % 64 == 0 && BN % 64 == 0, "tile edges must hold whole wave loads");

  struct Smem {
    float a[NS][A_FLOATS];
    float b[NS][B_FLOATS];
  };

  // Sources of this wave's direct loads at k = 0, and how far (in floats)
  // each moves per unit of k.  k-packed chunk q of an operand with R rows:
  // [q][R][4]; wave load t covers rows 64t' .. 64t'+63 of chunk t / (R/64).
  // k-major with R rows: wave load t covers floats [256t, 256t+256) = k rows
  // 256t/R ...
  static constexpr int AU = A_LOADS / NW, BU = B_LOADS / NW;  // wave loads per slice
  struct Src {
    const float* a[AU];
    const float* b[BU];
    int64_t astep, bstep;
  };

  template <bool KPACKED, int R>
  __device__ static const float* src_at_k0(const float* base, int64_t ld, int64_t r0,
                                           int64_t rmax, int t, int lane) {
    if constexpr (KPACKED) {
      const int q = t / (R / 64);                 // k group of 4
      const int row = (t % (R / 64)) * 64 + lane;
      int64_t gr = r0 + row;
      gr = gr < rmax ? gr : rmax - 1;
      return base + gr * ld + 4 * q;
    } else {
      const int flat = t * 256 + lane * 4;        // = k * R + row
      const int kk = flat / R, row = flat % R;
      // rmax is a multiple of 4 here, so a group is either wholly inside
      // or wholly past the edge (then it re-reads the last group)
      int64_t gr = r0 + row;
      gr = gr < rmax ? gr : rmax - 4;
      return base + kk * ld + gr;
    }
  }

  __device__ static Src sources(const GemmArgs& g, const float* A, const float* B, int64_t m0,
                                int64_t n0, int wave, int lane) {
    Src src;
#pragma unroll
    for (int u = 0; u < AU; ++u)
      src.a[u] = src_at_k0<!TA, BM>(A, g.lda, m0, g.m, wave + u * NW, lane);
#pragma unroll
    for (int u = 0; u < BU; ++u)
      src.b[u] = src_at_k0<TB, BN>(B, g.ldb, n0, g.n, wave + u * NW, lane);
    src.astep = TA ? g.lda : 1;
    src.bstep = TB ? 1 : g.ldb;
    return src;
  }

  // Issue this wave's share of the direct loads of slice s into ring slot.
  __device__ static void issue_slice(Smem& sm, const Src& src, int s, int slot, int wave) {
    const int64_t k0 = static_cast<int64_t>(s) * BK;
    const int64_t ao = k0 * src.astep, bo = k0 * src.bstep;
#pragma unroll
    for (int u = 0; u < AU; ++u)
      __builtin_amdgcn_global_load_lds((global_void_ptr)(src.a[u] + ao),
                                       (lds_void_ptr)(sm.a[slot] + (wave + u * NW) * 256), 16, 0,
                                       0);
#pragma unroll
    for (int u = 0; u < BU; ++u)
      __builtin_amdgcn_global_load_lds((global_void_ptr)(src.b[u] + bo),
                                       (lds_void_ptr)(sm.b[slot] + (wave + u * NW) * 256), 16, 0,
                                       0);
  }

  struct Pack {
    v4f a[IM];
    v4f b[IN];
  };

  // LDS reads of one group of 4 k (a lane's operands for 4 matrix steps).
  __device__ static void read_pack(const float* sa, const float* sb, int lane, int wm0, int wn0,
                                   int q, Pack& pk) {
#pragma unroll
    for (int i = 0; i < IM; ++i) {
      const int row = wm0 + i * 32 + (lane & 31);
      if constexpr (!TA) {
        pk.a[i] = *reinterpret_cast<const v4f*>(sa + (q * BM + row) * 4);
      } else {
#pragma unroll
        for (int c = 0; c < 4; ++c) pk.a[i][c] = sa[(4 * q + c) * BM + row];
      }
    }
#pragma unroll
    for (int j = 0; j < IN; ++j) {
      const int col = wn0 + j * 64 + lane;
      if constexpr (TB) {
        pk.b[j] = *reinterpret_cast<const v4f*>(sb + (q * BN + col) * 4);
      } else {
#pragma unroll
        for (int c = 0; c < 4; ++c) pk.b[j][c] = sb[(4 * q + c) * BN + col];
      }
    }
  }

  // Matrix steps [LO, HI) of one group of 4 k, in the order (c, i, j); step
  // c of every tile comes before step c + 1.  OPEN: step c = 0 starts the
  // block partials from +0.
  template <bool OPEN, int LO, int HI>
  __device__ static void mfma_steps(const Pack& pk, v32f (&P)[IM][IN]) {
    const v32f zero = {};
#pragma unroll
    for (int t = LO; t < HI; ++t) {
      const int c = t / (IM * IN), i = (t / IN) % IM, j = t % IN;
      P[i][j] = __builtin_amdgcn_mfma_f32_32x32x1f32(pk.a[i][c], pk.b[j][c],
                                                     (OPEN && c == 0) ? zero : P[i][j], 0, 0, 0);
    }
  }

  // Matrix step t (in the order of mfma_steps); t and open fold to constants.
  __device__ static __forceinline__ void mfma_step(const Pack& pk, v32f (&P)[IM][IN], int t,
                                                   bool open) {
    const v32f zero = {};
    const int c = t / (IM * IN), i = (t / IN) % IM, j = t % IN;
    P[i][j] = __builtin_amdgcn_mfma_f32_32x32x1f32(pk.a[i][c], pk.b[j][c],
                                                   (open && c == 0) ? zero : P[i][j], 0, 0, 0);
  }

  // Waits until this wave's loads of a slice have landed, given how many
  // later slices of this wave were issued after it (at most MAXL).
  template <int MAXL>
  __device__ static void wait_landed(int later) {
    constexpr int PER = (A_LOADS + B_LOADS) / NW;  // wave loads per slice
    static_assert(PER * MAXL < 64, "vmcnt range");
    if constexpr (MAXL == 0) {
      wait_vmcnt<0>();
    } else {
      if (later >= MAXL) wait_vmcnt<MAXL * PER>();
      else wait_landed<MAXL - 1>(later);
    }
  }

  // Slice s from ring slot `slot`; pk[0] already holds its first group of 4 k.
  // Each group's matrix steps are split after the first one: the LDS reads
  // of the next group go out there, so the remaining steps (each occupying
  // the matrix unit for 16 passes) cover their latency.  (While global-to-LDS
  // loads are in flight the compiler only waits for all LDS reads at once,
  // so the reads must be issued early rather than waited for selectively.)
  // In the last group the next slice is published at that point instead:
  // this wave waits for its share of slice s + 1; the barrier (every wave has
  // read all of slot `slot`, every share of slice s + 1 has landed) lets the
  // slot be refilled with slice s + NS; then the next slice's first group is
  // read.  OPEN: the slice opens a k block.
  //
  // FAST: every slice keeps the ring full -- past the last slice it re-loads
  // the last slice into the freed slot (in bounds; never read as data) -- so
  // every slice waits for the same load count and takes no branch; plain
  // ALU work may then be scheduled between the matrix steps.
  //
  // ADD: acc = acc + done (the previous k block's partials, held in a second
  // register set) is spread in small shares between this slice's matrix
  // steps, where it costs no matrix-unit time.
  template <bool OPEN, bool FAST, bool ADD = false>
  __device__ static void slice(Smem& sm, const Src& src, const Src& nsrc, int nlim, int s,
                               int nslices, int slot, int nslot, int lane, int wave, int wm0,
                               int wn0, Pack (&pk)[2], v32f (&P)[IM][IN], v32f (&acc)[IM][IN],
                               const v32f (&done)[IM][IN]) {
    constexpr int QN = BK / 4;
    constexpr int STEPS = 4 * IM * IN;
    constexpr int PER = (A_LOADS + B_LOADS) / NW;
    constexpr int CROSS = FAST ? 0x2 : 0;  // sched_barrier mask: plain VALU work may cross
    static_assert(QN % 2 == 0, "the next slice's first group must land in pk[0]");
#pragma unroll
    for (int q = 0; q < QN; ++q) {
      if (OPEN && q == 0) mfma_steps<true, 0, 1>(pk[0], P);
      else mfma_steps<false, 0, 1>(pk[q & 1], P);
      __builtin_amdgcn_sched_barrier(CROSS);
      if (q + 1 < QN) {
        read_pack(sm.a[slot], sm.b[slot], lane, wm0, wn0, q + 1, pk[(q + 1) & 1]);
      } else if (FAST) {
        wait_vmcnt<(NS - 2) * PER>();
        lds_barrier();
        if constexpr (RING) {
          // Past this tile's last slice the freed slot takes slice
          // s + NS - nslices (at most nlim) of the tile nsrc describes: the
          // next tile's first slices, or this tile's again (loads never read
          // as data).
          const bool here = s + NS < nslices;
          const int past = s + NS - nslices < nlim ? s + NS - nslices : nlim;
          Src pick;
#pragma unroll
          for (int u = 0; u < AU; ++u) pick.a[u] = here ? src.a[u] : nsrc.a[u];
#pragma unroll
          for (int u = 0; u < BU; ++u) pick.b[u] = here ? src.b[u] : nsrc.b[u];
          pick.astep = src.astep;
          pick.bstep = src.bstep;
          issue_slice(sm, pick, here ? s + NS : past, slot, wave);
        } else {
          issue_slice(sm, src, s + NS < nslices ? s + NS : nslices - 1, slot, wave);
        }
        read_pack(sm.a[nslot], sm.b[nslot], lane, wm0, wn0, 0, pk[0]);
      } else if (s + 1 < nslices) {
        const int later = nslices - 2 - s;  // slices after s + 1, capped by the ring
        wait_landed<NS - 2>(later < NS - 2 ? later : NS - 2);
        lds_barrier();
        if (s + NS < nslices) issue_slice(sm, src, s + NS, slot, wave);
        read_pack(sm.a[nslot], sm.b[nslot], lane, wm0, wn0, 0, pk[0]);
      }
      __builtin_amdgcn_sched_barrier(CROSS);
      if constexpr (ADD) {
        constexpr int NCH = QN * (STEPS - 1), TOT = IM * IN * 32;
#pragma unroll
        for (int t = 1; t < STEPS; ++t) {
          mfma_step(pk[q & 1], P, t, OPEN && q == 0);
          __builtin_amdgcn_sched_barrier(0);
          const int ch = q * (STEPS - 1) + t - 1;
#pragma unroll
          for (int f = TOT * ch / NCH; f < TOT * (ch + 1) / NCH; ++f) {
            const int u = f / 32, r = f % 32;
            acc[u / IN][u % IN][r] = acc[u / IN][u % IN][r] + done[u / IN][u % IN][r];
          }
          __builtin_amdgcn_sched_barrier(0);
        }
      } else {
        if (OPEN && q == 0) mfma_steps<true, 1, STEPS>(pk[0], P);
        else mfma_steps<false, 1, STEPS>(pk[q & 1], P);
      }
      __builtin_amdgcn_sched_barrier(CROSS);
    }
  }

  // One turn of the ring (NS slices, one k block) of the fast path,
  // accumulating the block in X while the previous block's partials in Y join
  // acc during the first slice.
  __device__ static void turn(Smem& sm, const Src& src, const Src& nsrc, int nlim, int s0,
                              int nslices, int lane, int wave, int wm0, int wn0, Pack (&pk)[2],
                              v32f (&X)[IM][IN], v32f (&acc)[IM][IN], const v32f (&Y)[IM][IN]) {
#pragma unroll
    for (int t = 0; t < NS; ++t) {
      if (t == 0)
        slice<true, true, true>(sm, src, nsrc, nlim, s0, nslices, 0, 1 % NS, lane, wave, wm0,
                                wn0, pk, X, acc, Y);
      else
        slice<false, true>(sm, src, nsrc, nlim, s0 + t, nslices, t, (t + 1) % NS, lane, wave,
                           wm0, wn0, pk, X, acc, Y);
    }
  }

  // The fast path with the second partial set over one tile's nslices slices
  // (a whole number of ring turns, one k block each): the ring holds slices
  // 0 .. NS - 1 and pk[0] the first group of slice 0.  acc receives the tile's
  // accumulators; past the last slice the ring is refilled from nsrc (see
  // slice), and pk[0] then holds the first group of that tile's slice 0.
  __device__ static void dual_fast(Smem& sm, const Src& src, const Src& nsrc, int nlim,
                                   int nslices, int lane, int wave, int wm0, int wn0,
                                   Pack (&pk)[2], v32f (&acc)[IM][IN]) {
    // Q starts at +0, so the first block adds +0 to +0.
    v32f P[IM][IN], Q[IM][IN];
#pragma unroll
    for (int i = 0; i < IM; ++i)
#pragma unroll
      for (int j = 0; j < IN; ++j) {
        P[i][j] = v32f{};
        Q[i][j] = v32f{};
        acc[i][j] = v32f{};
      }
    int s0 = 0;
    for (; s0 + 2 * NS <= nslices; s0 += 2 * NS) {
      turn(sm, src, nsrc, nlim, s0, nslices, lane, wave, wm0, wn0, pk, P, acc, Q);
      turn(sm, src, nsrc, nlim, s0 + NS, nslices, lane, wave, wm0, wn0, pk, Q, acc, P);
    }
    if (s0 < nslices) {
      turn(sm, src, nsrc, nlim, s0, nslices, lane, wave, wm0, wn0, pk, P, acc, Q);
#pragma unroll
      for (int i = 0; i < IM; ++i)
#pragma unroll
        for (int j = 0; j < IN; ++j) acc[i][j] = acc[i][j] + P[i][j];
    } else {
#pragma unroll
      for (int i = 0; i < IM; ++i)
#pragma unroll
        for (int j = 0; j < IN; ++j) acc[i][j] = acc[i][j] + Q[i][j];
    }
  }

  // Accumulator layout (lane l, register r): block r / 16 holds columns
  // 32*(r/16) + (l % 32), row 8*((r%16)/4) + 4*(l/32) + r%4.
  // An interior tile's stores: the scale, the bias and the GELU arrays resolved
  // once per tile (a lane's bias values read once), one address per output row
  // and array, no bounds checks; the operations are gemm_store's, in its order.
  template <bool ALPHA, bool BIAS, bool GOUT, bool XIN>
  __device__ static void store_plain(const GemmArgs& g, float* C, float* G, const float* X,
                                     int64_t m0, int64_t n0, int lane, int wm0, int wn0,
                                     const v32f (&acc)[IM][IN]) {
    const int64_t r0 = m0 + wm0 + 4 * (lane / 32);
    const int64_t c0 = n0 + wn0 + (lane & 31);
    float bj[IN][2];
#pragma unroll
    for (int j = 0; j < IN; ++j)
#pragma unroll
      for (int h = 0; h < 2; ++h) bj[j][h] = BIAS ? g.bias[c0 + j * 64 + 32 * h] : 0.0f;
    // The GELU inputs of all the lane's outputs are loaded before any store:
    // the compiler cannot see that X and C do not overlap (the host rejects
    // overlap), so loads written after earlier rows' stores would stay after
    // them, and each row would wait out a memory round trip.
    float xv[XIN ? IM : 1][4][4][IN][2];
    if constexpr (XIN) {
#pragma unroll
      for (int i = 0; i < IM; ++i)
#pragma unroll
        for (int q = 0; q < 4; ++q)
#pragma unroll
          for (int r4 = 0; r4 < 4; ++r4) {
            const float* px = X + (r0 + i * 32 + 8 * q + r4) * g.ld_gelu_in + c0;
#pragma unroll
            for (int j = 0; j < IN; ++j)
#pragma unroll
              for (int h = 0; h < 2; ++h) xv[i][q][r4][j][h] = px[j * 64 + 32 * h];
          }
    }
#pragma unroll
    for (int i = 0; i < IM; ++i)
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4) {
          const int64_t row = r0 + i * 32 + 8 * q + r4;
          float* pc = C + row * g.ldc + c0;
          float* pg = GOUT ? G + row * g.ldg + c0 : nullptr;
#pragma unroll
          for (int j = 0; j < IN; ++j)
#pragma unroll
            for (int h = 0; h < 2; ++h) {
              const int o = j * 64 + 32 * h;
              float v = gemm_scale_bias<ALPHA, BIAS>(acc[i][j][16 * h + 4 * q + r4], g.alpha,
                                                     bj[j][h]);
              if constexpr (XIN) v = v * rep_gelu_grad(xv[i][q][r4][j][h]);
              if constexpr (RING) {  // streamed: see run_ring
                __builtin_nontemporal_store(v, pc + o);
                if constexpr (GOUT) __builtin_nontemporal_store(rep_gelu(v), pg + o);
              } else {
                pc[o] = v;
                if constexpr (GOUT) pg[o] = rep_gelu(v);
              }
            }
        }
  }

  __device__ static void store_tile(const GemmArgs& g, int64_t b0, int64_t b1, int64_t m0,
                                    int64_t n0, int lane, int wm0, int wn0,
                                    const v32f (&acc)[IM][IN]) {
    float* C = g.C + b0 * g.sc0 + b1 * g.sc1;
    float* G = (GELU_OUT && g.G) ? g.G + b0 * g.sc0 + b1 * g.sc1 : nullptr;
    const float* X = g.gelu_in ? g.gelu_in + b0 * g.sc0 + b1 * g.sc1 : nullptr;
    // interior tile (uniform over the workgroup)
    if (EPI && m0 + BM <= g.m && n0 + BN <= g.n) {
      if (!G && !X) {
        if (g.has_alpha) {
          if (g.bias)
            store_plain<true, true, false, false>(g, C, G, X, m0, n0, lane, wm0, wn0, acc);
          else
            store_plain<true, false, false, false>(g, C, G, X, m0, n0, lane, wm0, wn0, acc);
        } else {
          if (g.bias)
            store_plain<false, true, false, false>(g, C, G, X, m0, n0, lane, wm0, wn0, acc);
          else
            store_plain<false, false, false, false>(g, C, G, X, m0, n0, lane, wm0, wn0, acc);
        }
        return;
      }
      if constexpr (GELU_OUT) {  // the forward product's GELU (no scale)
        if (G && !X && !g.has_alpha) {
          if (g.bias)
            store_plain<false, true, true, false>(g, C, G, X, m0, n0, lane, wm0, wn0, acc);
          else
            store_plain<false, false, true, false>(g, C, G, X, m0, n0, lane, wm0, wn0, acc);
          return;
        }
      }
      if (X && !G && !g.has_alpha && !g.bias) {  // the GELU backward's product
        store_plain<false, false, false, true>(g, C, G, X, m0, n0, lane, wm0, wn0, acc);
        return;
      }
    }
#pragma unroll
    for (int i = 0; i < IM; ++i)
#pragma unroll
      for (int j = 0; j < IN; ++j)
#pragma unroll
        for (int r = 0; r < 32; ++r) {
          const int64_t row = m0 + wm0 + i * 32 + 8 * ((r % 16) / 4) + 4 * (lane / 32) + (r % 4);
          const int64_t col = n0 + wn0 + j * 64 + 32 * (r / 16) + (lane & 31);
          if (row < g.m && col < g.n) gemm_store(g, C, G, X, row, col, acc[i][j][r]);
        }
  }

  __device__ static void run(const GemmArgs& g, Smem& sm, int64_t b0, int64_t b1, int64_t m0,
                             int64_t n0) {
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform in the wave
    const int wm0 = (wave / WN) * TWM;
    const int wn0 = (wave % WN) * TWN;
    // the host guarantees K / BK and k_block / BK fit in int
    const int nslices = static_cast<int>(k_extent(g, m0, BM) / BK);
    const int spb = g.k_block > 0 ? static_cast<int>(g.k_block / BK) : (nslices > 0 ? nslices : 1);
    const Src src = sources(g, g.A + b0 * g.sa0 + b1 * g.sa1, g.B + b0 * g.sb0 + b1 * g.sb1, m0,
                            n0, wave, lane);

    v32f P[IM][IN], acc[IM][IN];
#pragma unroll
    for (int i = 0; i < IM; ++i)
#pragma unroll
      for (int j = 0; j < IN; ++j) {
        P[i][j] = v32f{};
        acc[i][j] = v32f{};
      }
    // Prologue: the ring's NS slots filled with slices 0 .. NS - 1; slice 0
    // published and its first group read.
    Pack pk[2];
#pragma unroll
    for (int s = 0; s < NS; ++s)
      if (s < nslices) issue_slice(sm, src, s, s, wave);
    if (nslices > 0) {
      wait_landed<NS - 1>(nslices - 1 < NS - 1 ? nslices - 1 : NS - 1);
      lds_barrier();
      read_pack(sm.a[0], sm.b[0], lane, wm0, wn0, 0, pk[0]);
    }
    // Fast path: 64-deep k blocks (FSPB slices each) that tile the ring, and a
    // whole number of ring turns: one loop iteration is one turn, with the
    // ring slots and the block boundaries known at compile time.
    constexpr int FSPB = BK <= 64 ? 64 / BK : 0;
    if (FSPB > 0 && NS % FSPB == 0 && spb == FSPB && nslices % NS == 0) {
      if constexpr (DUAL && FSPB == NS) {
        // The second partial set: one ring turn is one k block, alternating
        // between P and Q, and each block's partials join acc during the next
        // block's first slice.
        dual_fast(sm, src, src, nslices - 1, nslices, lane, wave, wm0, wn0, pk, acc);
      } else {
        for (int s0 = 0; s0 < nslices; s0 += NS) {
#pragma unroll
          for (int t = 0; t < NS; ++t) {
            if (t % FSPB == 0)
              slice<true, true>(sm, src, src, nslices - 1, s0 + t, nslices, t, (t + 1) % NS,
                                lane, wave, wm0, wn0, pk, P, acc, P);
            else
              slice<false, true>(sm, src, src, nslices - 1, s0 + t, nslices, t, (t + 1) % NS,
                                 lane, wave, wm0, wn0, pk, P, acc, P);
            if (t % FSPB == FSPB - 1) {
#pragma unroll
              for (int i = 0; i < IM; ++i)
#pragma unroll
                for (int j = 0; j < IN; ++j) acc[i][j] = acc[i][j] + P[i][j];
            }
          }
        }
      }
      wait_vmcnt<0>();  // the re-loads past the end
    } else {
      int slot = 0, pos = 0;  // ring slot of slice s; s's place inside its k block
      for (int s = 0; s < nslices; ++s) {
        const int nslot = slot + 1 == NS ? 0 : slot + 1;
        if (pos == 0)
          slice<true, false>(sm, src, src, 0, s, nslices, slot, nslot, lane, wave, wm0, wn0, pk,
                             P, acc, P);
        else
          slice<false, false>(sm, src, src, 0, s, nslices, slot, nslot, lane, wave, wm0, wn0, pk,
                              P, acc, P);
        if (++pos == spb || s + 1 == nslices) {
          pos = 0;
#pragma unroll
          for (int i = 0; i < IM; ++i)
#pragma unroll
            for (int j = 0; j < IN; ++j) acc[i][j] = acc[i][j] + P[i][j];
        }
        slot = nslot;
      }
    }
    __syncthreads();
    store_tile(g, b0, b1, m0, n0, lane, wm0, wn0, acc);
  }

  // Launch index t's batch element and tile origin.
  __device__ static void locate(const GemmArgs& g, int64_t t, int64_t ntiles, int64_t tiles_m,
                                int64_t tiles_n, int64_t* b0, int64_t* b1, int64_t* m0,
                                int64_t* n0) {
    int64_t bz, tm, tn;
    tile_of(g, BM, BN, t, ntiles, tiles_m, tiles_n, &bz, &tm, &tn);
    *b1 = bz % g.batch1;
    *b0 = bz / g.batch1;
    *m0 = tm * BM;
    *n0 = tn * BN;
  }

  __device__ static Src sources_of(const GemmArgs& g, int64_t b0, int64_t b1, int64_t m0,
                                   int64_t n0, int wave, int lane) {
    return sources(g, g.A + b0 * g.sa0 + b1 * g.sa1, g.B + b0 * g.sb0 + b1 * g.sb1, m0, n0, wave,
                   lane);
  }

  // Launch indices blockIdx.x, + gridDim.x, ... in one workgroup, the ring
  // running on from each tile into the next: the last ring turn of a tile
  // loads the next tile's first NS slices into the slots it frees and its last
  // slice publishes the next tile's first one, so the next tile starts on
  // operands already in LDS while this tile's stores drain.  (The next tile's
  // first waits then also cover those stores: vector-memory operations
  // complete in issue order.)  An interior tile's stores are non-temporal:
  // with short contractions (the attention scores) a round of tiles writes
  // about as much as it reads, and cached output lines would push out of L2
  // the operand panels that the neighbouring tiles are reading.  Every tile
  // takes the fast path with the second partial set and the same slice count:
  // K and k_block make whole ring turns of one k block each, and no tile is
  // skipped or cut short (the host checks).
  __device__ static void run_ring(const GemmArgs& g, Smem& sm, int64_t tiles_m, int64_t tiles_n,
                                  int64_t ntiles) {
    static_assert(DUAL && RING, "the ring form runs the fast path with the second partial set");
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm0 = (wave / WN) * TWM;
    const int wn0 = (wave % WN) * TWN;
    const int nslices = static_cast<int>(g.k / BK);
    int64_t t = blockIdx.x;
    int64_t b0, b1, m0, n0;
    locate(g, t, ntiles, tiles_m, tiles_n, &b0, &b1, &m0, &n0);
    Src src = sources_of(g, b0, b1, m0, n0, wave, lane);
    // the first tile's prologue, as in run()
    Pack pk[2];
#pragma unroll
    for (int s = 0; s < NS; ++s) issue_slice(sm, src, s, s, wave);
    wait_landed<NS - 1>(NS - 1);
    lds_barrier();
    read_pack(sm.a[0], sm.b[0], lane, wm0, wn0, 0, pk[0]);
    for (;;) {
      const int64_t tn = t + gridDim.x;
      const bool more = tn < ntiles;  // uniform over the workgroup
      int64_t nb0 = b0, nb1 = b1, nm0 = m0, nn0 = n0;
      if (more) locate(g, tn, ntiles, tiles_m, tiles_n, &nb0, &nb1, &nm0, &nn0);
      const Src nsrc = more ? sources_of(g, nb0, nb1, nm0, nn0, wave, lane) : src;
      v32f acc[IM][IN];
      dual_fast(sm, src, nsrc, nslices - 1, nslices, lane, wave, wm0, wn0, pk, acc);
      store_tile(g, b0, b1, m0, n0, lane, wm0, wn0, acc);
      if (!more) break;
      t = tn;
      b0 = nb0;
      b1 = nb1;
      m0 = nm0;
      n0 = nn0;
      src = nsrc;
    }
    wait_vmcnt<0>();  // the re-loads past the last tile
  }
};

template <int BM, int BN, int BK, int WM, int WN, int NS, int MINW, bool TA, bool TB, bool EPI>
__global__ __launch_bounds__(64 * WM * WN, MINW) void gemm_mfma_staged_kernel(
    GemmArgs g, int64_t tiles_m, int64_t tiles_n, int64_t ntiles, int) {
  // one instruction tile per wave leaves registers for the second partial set
  using T = StagedTile<BM, BN, BK, WM, WN, NS, TA, TB, (BM / WM / 32) * (BN / WN / 64) == 1,
                       true, false, EPI>;
  __shared__ typename T::Smem sm;
  for (int64_t t = blockIdx.x; t < ntiles; t += gridDim.x) {
    int64_t bz, tm, tn;
    tile_of(g, BM, BN, t, ntiles, tiles_m, tiles_n, &bz, &tm, &tn);
    const int64_t b1 = bz % g.batch1, b0 = bz / g.batch1;
    if (tile_above_diagonal(g, tm * BM, BM, tn * BN)) continue;  // uniform over the workgroup
    T::run(g, sm, b0, b1, tm * BM, tn * BN);
  }
}

// The persistent form of a staged tile (StagedTile::run_ring); the host
// launches about one workgroup per compute unit.
template <int BM, int BN, int BK, int WM, int WN, int NS, int MINW, bool TA, bool TB>
__global__ __launch_bounds__(64 * WM * WN, MINW) void gemm_mfma_ring_kernel(
    GemmArgs g, int64_t tiles_m, int64_t tiles_n, int64_t ntiles, int) {
  using T = StagedTile<BM, BN, BK, WM, WN, NS, TA, TB, true, true, true>;
  __shared__ typename T::Smem sm;
  T::run_ring(g, sm, tiles_m, tiles_n, ntiles);
}

// Several products in one launch with table entry 0's tile: workgroup t
// finds its product p (first[p] <= t < first[p + 1]) and runs that product's
// tile with the transposes it needs.  The four layouts' LDS forms have the
// same size, so one allocation serves them all.  Every tile is the same
// computation as in a launch of its own product, so the bits are the same.
template <int BM, int BN, int BK, int WM, int WN, int NS, int MINW, bool DUAL>
__global__ __launch_bounds__(64 * WM * WN, MINW) void gemm_mfma_grouped_kernel(GroupArgs ga) {
  using T00 = StagedTile<BM, BN, BK, WM, WN, NS, false, false, DUAL, false>;
  using T01 = StagedTile<BM, BN, BK, WM, WN, NS, false, true, DUAL, false>;
  using T10 = StagedTile<BM, BN, BK, WM, WN, NS, true, false, DUAL, false>;
  using T11 = StagedTile<BM, BN, BK, WM, WN, NS, true, true, DUAL, false>;
  static_assert(sizeof(typename T00::Smem) == sizeof(typename T11::Smem), "one LDS form size");
  __shared__ typename T00::Smem sm;
  const int64_t t = blockIdx.x;
  int p = 0;
  while (p + 1 < ga.count && t >= ga.first[p + 1]) ++p;
  const GemmArgs& g = ga.g[p];
  const int64_t ntiles = ga.first[p + 1] - ga.first[p];
  int64_t bz, tm, tn;
  tile_coords(t - ga.first[p], ntiles, ga.tiles_m[p], ga.tiles_n[p], &bz, &tm, &tn);
  const int64_t m0 = tm * BM, n0 = tn * BN;
  if (!g.ta && !g.tb) T00::run(g, sm, 0, 0, m0, n0);
  else if (!g.ta) T01::run(g, *reinterpret_cast<typename T01::Smem*>(&sm), 0, 0, m0, n0);
  else if (!g.tb) T10::run(g, *reinterpret_cast<typename T10::Smem*>(&sm), 0, 0, m0, n0);
  else T11::run(g, *reinterpret_cast<typename T11::Smem*>(&sm), 0, 0, m0, n0);
}

struct MfmaEntry {
  GemmConfig cfg;
  int threads;
  void (*kernel[4])(GemmArgs, int64_t, int64_t, int64_t, int);  // [ta * 2 + tb]
  // staged variant of the same tile shape (nullptr: none); needs K % 16 == 0
  // and 16-byte aligned rows.  [0]: for products with no scale, bias or GELU
  // array; [1]: for the others (the specialised interior stores)
  void (*staged[2][4])(GemmArgs, int64_t, int64_t, int64_t, int);
  // persistent form of the staged tile with the ring running across tiles
  // (nullptr: none); taken where every tile makes whole ring turns
  void (*ring[4])(GemmArgs, int64_t, int64_t, int64_t, int);
};

// MINW: waves per SIMD the register allocation must leave room for.
#define REPOPS_MFMA(BM, BN, BK, WM, WN, MINW)                                                 \
  {{#BM "x" #BN "x" #BK "/w" #WM "x" #WN "/o" #MINW, BM, BN, BK},                             \
   64 * WM * WN,                                                                              \
   {gemm_mfma_kernel<BM, BN, BK, WM, WN, MINW, false, false>,                                 \
    gemm_mfma_kernel<BM, BN, BK, WM, WN, MINW, false, true>,                                  \
    gemm_mfma_kernel<BM, BN, BK, WM, WN, MINW, true, false>,                                  \
    gemm_mfma_kernel<BM, BN, BK, WM, WN, MINW, true, true>},                                  \
   {{nullptr, nullptr, nullptr, nullptr}, {nullptr, nullptr, nullptr, nullptr}},              \
   {nullptr, nullptr, nullptr, nullptr}}

// The staged kernels of a tile: [1] with the specialised interior stores; [0]
// with EPI = EPI0 -- false keeps a form whose every output takes the checked
// loop, true makes [0] the same kernels as [1].
#define REPOPS_STAGED_KERNELS(BM, BN, BK, WM, WN, NS, MINW, EPI0)                            \
  {{gemm_mfma_staged_kernel<BM, BN, BK, WM, WN, NS, MINW, false, false, EPI0>,               \
    gemm_mfma_staged_kernel<BM, BN, BK, WM, WN, NS, MINW, false, true, EPI0>,                \
    gemm_mfma_staged_kernel<BM, BN, BK, WM, WN, NS, MINW, true, false, EPI0>,                \
    gemm_mfma_staged_kernel<BM, BN, BK, WM, WN, NS, MINW, true, true, EPI0>},                \
   {gemm_mfma_staged_kernel<BM, BN, BK, WM, WN, NS, MINW, false, false, true>,               \
    gemm_mfma_staged_kernel<BM, BN, BK, WM, WN, NS, MINW, false, true, true>,                \
    gemm_mfma_staged_kernel<BM, BN, BK, WM, WN, NS, MINW, true, false, true>,                \
    gemm_mfma_staged_kernel<BM, BN, BK, WM, WN, NS, MINW, true, true, true>}}

// MINW: waves per SIMD the register allocation must leave room for; FWM x FWN:
// the wave grid of the register-staged fallback of the same tile (as many
// waves, each owning whole 64 x 32 instruction tiles).
#define REPOPS_STAGED(BM, BN, BK, WM, WN, NS, MINW, FWM, FWN, EPI0)                          \
  {{#BM "x" #BN "x" #BK "/w" #WM "x" #WN "/o" #MINW "/s" #NS, BM, BN, BK},                    \
   64 * WM * WN,                                                                              \
   {gemm_mfma_kernel<BM, BN, BK, FWM, FWN, MINW, false, false>,                               \
    gemm_mfma_kernel<BM, BN, BK, FWM, FWN, MINW, false, true>,                                \
    gemm_mfma_kernel<BM, BN, BK, FWM, FWN, MINW, true, false>,                                \
    gemm_mfma_kernel<BM, BN, BK, FWM, FWN, MINW, true, true>},                                \
   REPOPS_STAGED_KERNELS(BM, BN, BK, WM, WN, NS, MINW, EPI0),                                 \
   {nullptr, nullptr, nullptr, nullptr}}

// A staged tile with its persistent ring form as well (one instruction tile
// per wave: the second partial set).
#define REPOPS_RING(BM, BN, BK, WM, WN, NS, MINW, FWM, FWN)                                  \
  {{#BM "x" #BN "x" #BK "/w" #WM "x" #WN "/o" #MINW "/s" #NS "/ring", BM, BN, BK},            \
   64 * WM * WN,                                                                              \
   {gemm_mfma_kernel<BM, BN, BK, FWM, FWN, MINW, false, false>,                               \
    gemm_mfma_kernel<BM, BN, BK, FWM, FWN, MINW, false, true>,                                \
    gemm_mfma_kernel<BM, BN, BK, FWM, FWN, MINW, true, false>,                                \
    gemm_mfma_kernel<BM, BN, BK, FWM, FWN, MINW, true, true>},                                \
   REPOPS_STAGED_KERNELS(BM, BN, BK, WM, WN, NS, MINW, false),                                \
   {gemm_mfma_ring_kernel<BM, BN, BK, WM, WN, NS, MINW, false, false>,                        \
    gemm_mfma_ring_kernel<BM, BN, BK, WM, WN, NS, MINW, false, true>,                         \
    gemm_mfma_ring_kernel<BM, BN, BK, WM, WN, NS, MINW, true, false>,                         \
    gemm_mfma_ring_kernel<BM, BN, BK, WM, WN, NS, MINW, true, true>}}

const MfmaEntry kMfma[] = {
    REPOPS_STAGED(128, 128, 16, 4, 2, 4, 2, 2, 4, false),  // 0: default for large outputs
    REPOPS_STAGED(128, 128, 16, 2, 2, 4, 2, 2, 2, true),   // 1: one wave per SIMD
    REPOPS_MFMA(128, 128, 16, 2, 2, 2),                    // 2: short k, few tiles
    REPOPS_STAGED(128, 128, 32, 2, 2, 4, 1, 2, 2, true),   // 3
    REPOPS_STAGED(256, 128, 16, 4, 2, 3, 1, 4, 2, true),   // 4
    REPOPS_MFMA(64, 64, 32, 1, 2, 2),                      // 5: small outputs
    REPOPS_STAGED(128, 128, 32, 4, 2, 4, 2, 2, 4, true),   // 6
    REPOPS_STAGED(256, 128, 16, 4, 2, 4, 2, 4, 2, true),   // 7
    // 8: products whose A is zero above its diagonal (causal probabilities x
    // values): 64-row tiles end their contraction closer to their diagonal, and
    // three workgroups per CU overlap one tile's loads and stores with another's
    REPOPS_STAGED(64, 128, 16, 2, 2, 4, 3, 1, 4, true),
    // 9: entry 0's tile, persistent, its ring running on into the next tile
    REPOPS_RING(128, 128, 16, 4, 2, 4, 2, 2, 4),
};
constexpr int kMfmaCount = sizeof(kMfma) / sizeof(kMfma[0]);

bool aligned16(const void* p) { return reinterpret_cast<uintptr_t>(p) % 16 == 0; }

}  // namespace

int gemm_mfma_count() { return kMfmaCount; }
const GemmConfig* gemm_mfma_config(int index) {
  return (index >= 0 && index < kMfmaCount) ? &kMfma[index].cfg : nullptr;
}

bool gemm_mfma_staged_ok(const GemmArgs& g, int index) {
  const MfmaEntry& e = kMfma[index];
  const bool vec_ok = aligned16(g.A) && g.lda % 4 == 0 && g.sa0 % 4 == 0 && g.sa1 % 4 == 0 &&
                      aligned16(g.B) && g.ldb % 4 == 0 && g.sb0 % 4 == 0 && g.sb1 % 4 == 0;
  return e.staged[1][0] && vec_ok && g.k % e.cfg.bk == 0 && g.k / e.cfg.bk <= INT32_MAX &&
         g.k_block / e.cfg.bk <= INT32_MAX && (!g.ta || g.m % 4 == 0) && (g.tb || g.n % 4 == 0);
}

// Tiles of a launch that the ring form of entry `index` can take, else 0: every
// tile makes whole ring turns of one 64-deep k block each (16-deep slices,
// four slots) over the same K, the staged kernel's layout rules hold, and no
// tile is skipped or cut short.  *cus receives the device's compute units; the
// launch takes the ring form when the tiles outnumber them.
int64_t gemm_mfma_ring_tiles(const GemmArgs& g, int index, int* cus) {
  const MfmaEntry& e = kMfma[index];
  *cus = 0;
  if (!e.ring[0] || e.cfg.bk != 16 || g.k <= 0 || g.k_block != 64 || g.k % 64 != 0 ||
      !gemm_mfma_staged_ok(g, index))
    return 0;
  const int64_t tiles_m = (g.m + e.cfg.bm - 1) / e.cfg.bm;
  const int64_t tiles_n = (g.n + e.cfg.bn - 1) / e.cfg.bn;
  const bool tri = causal_triangle(g.causal, e.cfg.bm, e.cfg.bn, tiles_m, tiles_n);
  if (g.causal != 0 && !tri) return 0;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      *cus <= 0) {
    *cus = 0;
    return 0;
  }
  const int64_t per_batch = tri ? tiles_m * (tiles_m + 1) / 2 : tiles_m * tiles_n;
  return per_batch * g.batch0 * g.batch1;
}

void gemm_mfma_tile(int index, int* bm, int* bn) {
  *bm = kMfma[index].cfg.bm;
  *bn = kMfma[index].cfg.bn;
}

hipError_t launch_gemm_mfma_grouped(const GroupArgs& ga, hipStream_t s) {
  // table entry 0: 128 x 128 tiles, 8 waves, a 4-slot ring of 16-deep slices
  const int64_t total = ga.first[ga.count];
  hipLaunchKernelGGL((gemm_mfma_grouped_kernel<128, 128, 16, 4, 2, 4, 2, true>),
                     dim3(static_cast<unsigned>(total)), dim3(512), 0, s, ga);
  return hipGetLastError();
}

hipError_t launch_gemm_mfma(const GemmArgs& g, int index, hipStream_t s) {
  const MfmaEntry& e = kMfma[index];
  const int64_t tiles_m = (g.m + e.cfg.bm - 1) / e.cfg.bm;
  const int64_t tiles_n = (g.n + e.cfg.bn - 1) / e.cfg.bn;
  const int64_t per_batch = causal_triangle(g.causal, e.cfg.bm, e.cfg.bn, tiles_m, tiles_n)
                                ? tiles_m * (tiles_m + 1) / 2
                                : tiles_m * tiles_n;
  const int64_t ntiles = per_batch * g.batch0 * g.batch1;
  const int64_t cap = int64_t(1) << 30;
  const unsigned grid = static_cast<unsigned>(ntiles < cap ? ntiles : cap);
  // float4 loads need 16-byte aligned rows and batch origins
  const int vec_ok = aligned16(g.A) && g.lda % 4 == 0 && g.sa0 % 4 == 0 && g.sa1 % 4 == 0 &&
                     aligned16(g.B) && g.ldb % 4 == 0 && g.sb0 % 4 == 0 && g.sb1 % 4 == 0;
  auto kernel = e.kernel[g.ta * 2 + g.tb];
  // the staged kernel takes whole slices only: K a multiple of its depth
  // (and slice counts that fit in int)
  const bool staged_ok = vec_ok && g.k % e.cfg.bk == 0 && g.k / e.cfg.bk <= INT32_MAX &&
                         g.k_block / e.cfg.bk <= INT32_MAX && (!g.ta || g.m % 4 == 0) &&
                         (g.tb || g.n % 4 == 0);
  unsigned blocks = grid;
  // the specialised stores where the product has a scale, a bias or a GELU array
  const int epi = (g.has_alpha || g.bias || g.G || g.gelu_in) ? 1 : 0;
  if (e.staged[1][0] && staged_ok) kernel = e.staged[epi][g.ta * 2 + g.tb];
  int cus = 0;
  if (gemm_mfma_ring_tiles(g, index, &cus) > cus) {
    kernel = e.ring[g.ta * 2 + g.tb];
    blocks = static_cast<unsigned>(cus);
  }
  hipLaunchKernelGGL(kernel, dim3(blocks), dim3(e.threads), 0, s, g, tiles_m, tiles_n, ntiles,
                     vec_ok);
  return hipGetLastError();
}

}  // namespace repops
