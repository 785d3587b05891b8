// Reproducible training-step operators for gfx950: softmax, LayerNorm and
// GELU backward, and the Adam / AdamW update.
//
// The training runs of the Verde paper (Section 4.2, Adam optimizer) execute
// the extended graph of Section 2.2: forward nodes, their backward nodes and
// the optimizer update.  Each backward operator below is one fixed sequence of
// binary32 operations per output; its row reductions take the order
// descriptor's row order, and the LayerNorm parameter gradients reduce over
// rows with the contraction's blocked left-to-right rule.
//
// LayerNorm parameter gradients: for column j, dgamma_j = sum over rows i of
// dy_ij * t_ij and dbeta_j = sum of dy_ij, with blocks of k_block consecutive
// rows, each block a sequential chain from +0 (fma for dgamma, add for dbeta),
// block partials added left to right.  The partials are formed in the same
// pass as the input gradient (one workgroup per row block staging rows in
// LDS, or, with few blocks, a block's rows and column slices spread over
// several workgroups), or on their own with one thread per (block, column)
// -- every chain is independent -- and a second kernel adds them left to
// right per column.
// With a single block the first kernel writes the gradients directly as the
// left-to-right sum of that one partial, +0 + P: a fused dgamma chain can end
// at -0 (a negative product below half the smallest subnormal rounds to -0),
// and the accumulator's +0 + (-0) = +0 must still be taken.
#include <hip/hip_runtime.h>

#include <mutex>

#include "rep_math.h"
#include "repops_internal.h"
#include "train_internal.h"
#include "row_reduce.h"
#include "stream_store.h"

#pragma clang fp contract(off)

namespace repops {
namespace {

// ---------------------------------------------------------------------------
// softmax backward: dx_j = y_j * (dy_j - s), s = rowsum of fma(y_j, dy_j, .)
// over the unmasked columns; masked columns get +0.
// ---------------------------------------------------------------------------

// The widest rows (T = 64) keep 128 row values per lane and run at most four
// waves per workgroup, which leaves them a full register file.
template <int T>
__global__ __launch_bounds__(T > 32 ? 256 : 512) void softmax_bwd_wave_kernel(RowBwdArgs a,
                                                                              int wpb) {
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t row = static_cast<int64_t>(blockIdx.x) * wpb + wave_id();
  if (row >= a.rows) return;
  const float* y = a.Y + row * a.ldy;
  const float* dy = a.dY + row * a.lddy;
  float* dx = a.dX + row * a.lddx;
  int64_t valid = a.cols;
  if (a.period > 0) {
    const int64_t v = row % a.period + 1;
    valid = v < valid ? v : valid;
  }
  const int64_t live = (valid + kWave - 1) / kWave;
  float yv[T], dv[T];
  float q = 0.0f;
#pragma unroll
  for (int t = 0; t < T; ++t) {
    const int64_t j = lane + kWave * t;
    yv[t] = 0.0f;
    dv[t] = 0.0f;
    if (t < live && j < valid) {  // masked entries are never read
      yv[t] = y[j];
      dv[t] = dy[j];
    }
    // Masked and absent terms take no operation (as in the oracle's row
    // order): the chain can hold -0 (a negative product below half the
    // smallest subnormal), which fma(+0, +0, -0) = +0 would change.
    if (j < valid) q = __builtin_fmaf(yv[t], dv[t], q);
  }
  const float s = wave_tree_sum(q);
  auto out = [&](int t, int64_t j) {
    const float diff = dv[t] - s;
    return j < valid ? yv[t] * diff : 0.0f;
  };
  if (a.cols == kWave * T) {  // full-width row: unconditional stores
#pragma unroll
    for (int t = 0; t < T; ++t) st_stream(dx + lane + kWave * t, out(t, lane + kWave * t));
  } else {
#pragma unroll
    for (int t = 0; t < T; ++t) {
      const int64_t j = lane + kWave * t;
      if (j < a.cols) st_stream(dx + j, out(t, j));
    }
  }
}

__global__ __launch_bounds__(64) void softmax_bwd_generic_kernel(RowBwdArgs a) {
  __shared__ float qs[1024];
  const int lane = threadIdx.x;
  for (int64_t row = blockIdx.x; row < a.rows; row += gridDim.x) {
    const float* y = a.Y + row * a.ldy;
    const float* dy = a.dY + row * a.lddy;
    float* dx = a.dX + row * a.lddx;
    int64_t valid = a.cols;
    if (a.period > 0) {
      const int64_t v = row % a.period + 1;
      valid = v < valid ? v : valid;
    }
    auto term = [&](float q, int64_t j) { return j < valid ? __builtin_fmaf(y[j], dy[j], q) : q; };
    const float s = generic_row_sum(a.cols, a.W, a.blocked, term, qs);
    for (int64_t j = lane; j < a.cols; j += kWave) {
      float o = 0.0f;
      if (j < valid) {
        const float diff = dy[j] - s;
        o = y[j] * diff;
      }
      st_stream(dx + j, o);  // dX may equal Y or dY: element j is read before it is written
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// LayerNorm backward, input gradient.  With the forward's mean and rstd:
//   t_j = (x_j - mean) * rstd;  g_j = dy_j * gamma_j (dy_j without gamma);
//   a = rowsum(g) / n;  b = rowsum of fma(g_j, t_j, .) / n;
//   dx_j = rstd * ((g_j - a) - t_j * b).
// ---------------------------------------------------------------------------

// t_j = (x_j - mean) * rstd and g_j = dy_j * gamma_j (dy_j without gamma) of
// the columns j0 + 64 t, t < T, +0 past the row.  Every load is issued before
// any arithmetic (a load and its use in one conditional block would wait for
// each element in turn).
template <int T>
__device__ __forceinline__ void ln_bwd_terms(const RowBwdArgs& a, const float* x, const float* dy,
                                             int64_t j0, float mean, float rstd, float (&tv)[T],
                                             float (&gv)[T]) {
  float xv[T], dv[T], gm[T];
#pragma unroll
  for (int t = 0; t < T; ++t) {
    const int64_t j = j0 + kWave * t;
    xv[t] = 0.0f;
    dv[t] = 0.0f;
    if (j < a.cols) {
      xv[t] = x[j];
      dv[t] = dy[j];
    }
  }
  if (a.gamma) {
#pragma unroll
    for (int t = 0; t < T; ++t) {
      const int64_t j = j0 + kWave * t;
      gm[t] = 0.0f;
      if (j < a.cols) gm[t] = a.gamma[j];
    }
  }
#pragma unroll
  for (int t = 0; t < T; ++t) {
    const bool in = j0 + kWave * t < a.cols;
    const float d = xv[t] - mean;
    const float tt = d * rstd;
    const float g = a.gamma ? dv[t] * gm[t] : dv[t];
    tv[t] = in ? tt : 0.0f;
    gv[t] = in ? g : 0.0f;
  }
}

// dX of one row by one wave (row < a.rows, uniform over the wave; all 64
// lanes active).
template <int T>
__device__ __forceinline__ void layernorm_bwd_row(const RowBwdArgs& a, int64_t row, int lane) {
  const float* x = a.Y + row * a.ldy;
  const float* dy = a.dY + row * a.lddy;
  float* dx = a.dX + row * a.lddx;
  const float mean = a.rms ? 0.0f : a.mean[row], rstd = a.rstd[row];
  float tv[T], gv[T];
  ln_bwd_terms<T>(a, x, dy, lane, mean, rstd, tv, gv);
  float q = 0.0f;
#pragma unroll
  for (int t = 0; t < T; ++t) q = q + gv[t];  // terms past the row are +0 and leave q unchanged
  const float n = static_cast<float>(a.cols);
  const float am = a.rms ? 0.0f : wave_tree_sum(q) / n;
  float q2 = 0.0f;
#pragma unroll
  for (int t = 0; t < T; ++t)  // terms past the row take no operation (the chain may hold -0)
    if (lane + kWave * t < a.cols) q2 = __builtin_fmaf(gv[t], tv[t], q2);
  const float bm = wave_tree_sum(q2) / n;
  auto out = [&](int t) {
    const float u = gv[t] - am;
    const float tb = tv[t] * bm;
    const float w = u - tb;
    return rstd * w;
  };
  if (a.cols == kWave * T) {
#pragma unroll
    for (int t = 0; t < T; ++t) st_stream(dx + lane + kWave * t, out(t));
  } else {
#pragma unroll
    for (int t = 0; t < T; ++t) {
      const int64_t j = lane + kWave * t;
      if (j < a.cols) st_stream(dx + j, out(t));
    }
  }
}

template <int T>
__global__ __launch_bounds__(512) void layernorm_bwd_wave_kernel(RowBwdArgs a, int wpb) {
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t row = static_cast<int64_t>(blockIdx.x) * wpb + wave_id();
  if (row >= a.rows) return;
  layernorm_bwd_row<T>(a, row, lane);
}

// ---------------------------------------------------------------------------
// Wide rows: one row per workgroup of S waves (wave w holds the columns
// lane + 64 * (w * T + t)); each lane's chains pass from wave to wave through
// LDS in wave order, so the terms meet in the one-wave kernels' order and the
// results are the same bits.
// ---------------------------------------------------------------------------

template <int T>
__global__ __launch_bounds__(512) void softmax_bwd_split_kernel(RowBwdArgs a) {
  __shared__ float chain[kWave];
  const int lane = threadIdx.x & (kWave - 1);
  const int w = wave_id();
  const int S = static_cast<int>(blockDim.x >> 6);
  for (int64_t row = blockIdx.x; row < a.rows; row += gridDim.x) {
    const float* y = a.Y + row * a.ldy;
    const float* dy = a.dY + row * a.lddy;
    float* dx = a.dX + row * a.lddx;
    int64_t valid = a.cols;
    if (a.period > 0) {
      const int64_t v = row % a.period + 1;
      valid = v < valid ? v : valid;
    }
    const int64_t live = (valid + kWave - 1) / kWave;
    const int64_t s0 = int64_t(T) * w;  // this wave's first segment
    float yv[T], dv[T];
#pragma unroll
    for (int t = 0; t < T; ++t) {
      const int64_t j = lane + kWave * (s0 + t);
      yv[t] = 0.0f;
      dv[t] = 0.0f;
      if (s0 + t < live && j < valid) {  // masked entries are never read
        yv[t] = y[j];
        dv[t] = dy[j];
      }
    }
    const float q = chain_across_waves(chain, lane, w, S, [&](float c) {
#pragma unroll
      for (int t = 0; t < T; ++t)  // masked and absent terms: no operation (c may be -0)
        if (lane + kWave * (s0 + t) < valid) c = __builtin_fmaf(yv[t], dv[t], c);
      return c;
    });
    const float sum = wave_tree_sum(q);
#pragma unroll
    for (int t = 0; t < T; ++t) {
      const int64_t j = lane + kWave * (s0 + t);
      if (j < a.cols) st_stream(dx + j, j < valid ? yv[t] * (dv[t] - sum) : 0.0f);
    }
    __syncthreads();  // chains read before the next row
  }
}

template <int T>
__global__ __launch_bounds__(512) void layernorm_bwd_split_kernel(RowBwdArgs a) {
  __shared__ float chain_g[kWave];
  __shared__ float chain_gt[kWave];
  const int lane = threadIdx.x & (kWave - 1);
  const int w = wave_id();
  const int S = static_cast<int>(blockDim.x >> 6);
  const float n = static_cast<float>(a.cols);
  for (int64_t row = blockIdx.x; row < a.rows; row += gridDim.x) {
    const float* x = a.Y + row * a.ldy;
    const float* dy = a.dY + row * a.lddy;
    float* dx = a.dX + row * a.lddx;
    const float mean = a.rms ? 0.0f : a.mean[row], rstd = a.rstd[row];
    const int64_t j0 = lane + int64_t(kWave) * T * w;
    float tv[T], gv[T];
    ln_bwd_terms<T>(a, x, dy, j0, mean, rstd, tv, gv);
    float am = 0.0f;
    if (!a.rms) {  // uniform over the workgroup
      const float q = chain_across_waves(chain_g, lane, w, S, [&](float c) {
#pragma unroll
        for (int t = 0; t < T; ++t) c = c + gv[t];  // past the row: +0
        return c;
      });
      am = wave_tree_sum(q) / n;
    }
    const float q2 = chain_across_waves(chain_gt, lane, w, S, [&](float c) {
#pragma unroll
      for (int t = 0; t < T; ++t)  // past the row: no operation (c may be -0)
        if (j0 + kWave * t < a.cols) c = __builtin_fmaf(gv[t], tv[t], c);
      return c;
    });
    const float bm = wave_tree_sum(q2) / n;
#pragma unroll
    for (int t = 0; t < T; ++t) {
      const int64_t j = j0 + kWave * t;
      if (j < a.cols) {
        const float u = gv[t] - am;
        const float tb = tv[t] * bm;
        st_stream(dx + j, rstd * (u - tb));
      }
    }
    __syncthreads();  // chains read before the next row
  }
}

__global__ __launch_bounds__(64) void layernorm_bwd_generic_kernel(RowBwdArgs a) {
  __shared__ float qs[1024];
  const int lane = threadIdx.x;
  const float n = static_cast<float>(a.cols);
  for (int64_t row = blockIdx.x; row < a.rows; row += gridDim.x) {
    const float* x = a.Y + row * a.ldy;
    const float* dy = a.dY + row * a.lddy;
    float* dx = a.dX + row * a.lddx;
    const float mean = a.rms ? 0.0f : a.mean[row], rstd = a.rstd[row];
    auto g_at = [&](int64_t j) { return a.gamma ? dy[j] * a.gamma[j] : dy[j]; };
    auto t_at = [&](int64_t j) {
      const float d = x[j] - mean;
      return d * rstd;
    };
    auto sum_g = [&](float q, int64_t j) { return q + g_at(j); };
    const float am = a.rms ? 0.0f : generic_row_sum(a.cols, a.W, a.blocked, sum_g, qs) / n;
    auto sum_gt = [&](float q, int64_t j) { return __builtin_fmaf(g_at(j), t_at(j), q); };
    const float bm = generic_row_sum(a.cols, a.W, a.blocked, sum_gt, qs) / n;
    for (int64_t j = lane; j < a.cols; j += kWave) {
      const float gj = g_at(j), tj = t_at(j);
      const float u = gj - am;
      const float tb = tj * bm;
      const float w = u - tb;
      st_stream(dx + j, rstd * w);  // dX may equal X or dY: element j is read before it is written
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// LayerNorm parameter gradients.
// ---------------------------------------------------------------------------

// Workspace layout of the block partials: for each of the two arrays (dgamma,
// then dbeta), the columns in tiles of kTile (the last one narrower), each
// tile stored block-major ([block][column in tile]).  All partials of one
// tile are one contiguous span, which the combine reads whole; the total is
// 2 * blocks * cols floats.
constexpr int kTile = 16;

__device__ __forceinline__ int64_t ws_index(int arr, int64_t b, int64_t j, int64_t nblk,
                                            int64_t cols) {
  const int64_t t0 = j & ~int64_t(kTile - 1);
  const int64_t tw = cols - t0 < kTile ? cols - t0 : kTile;
  return (arr * cols + t0) * nblk + b * tw + (j - t0);
}

constexpr int kParamThreads = 256;

__global__ __launch_bounds__(kParamThreads) void layernorm_param_partial_kernel(
    LnParamArgs a, int64_t col_groups, int64_t blk, int64_t nblk) {
  const int64_t bid = blockIdx.x;
  const int64_t beta = bid / col_groups;
  const int64_t j = (bid - beta * col_groups) * kParamThreads + threadIdx.x;
  if (j >= a.cols) return;
  const int64_t i0 = beta * blk;
  const int64_t i1 = (i0 + blk < a.rows) ? i0 + blk : a.rows;
  const float* xp = a.X + j;
  const float* dp = a.dY + j;
  float pg = 0.0f, pb = 0.0f;
  int64_t i = i0;
  // Rows in batches whose loads all issue before any arithmetic (one memory
  // round trip per batch); the chains themselves advance one row at a time.
  if (a.sum_only) {  // bias gradient: dY's column chains only, 32 rows a batch
    constexpr int RB = 32;
    for (; i + RB <= i1; i += RB) {
      float dv[RB];
#pragma unroll
      for (int r = 0; r < RB; ++r) dv[r] = dp[(i + r) * a.lddy];
#pragma unroll
      for (int r = 0; r < RB; ++r) pb = pb + dv[r];
    }
    for (; i < i1; ++i) pb = pb + dp[i * a.lddy];
  }
  constexpr int RB = 16;
  for (; i + RB <= i1; i += RB) {
    float xv[RB], dv[RB], mv[RB], rv[RB];
#pragma unroll
    for (int r = 0; r < RB; ++r) {
      xv[r] = xp[(i + r) * a.ldx];
      dv[r] = dp[(i + r) * a.lddy];
      mv[r] = a.rms ? 0.0f : a.mean[i + r];
      rv[r] = a.rstd[i + r];
    }
#pragma unroll
    for (int r = 0; r < RB; ++r) {
      const float d = xv[r] - mv[r];
      const float t = d * rv[r];
      pg = __builtin_fmaf(dv[r], t, pg);
      pb = pb + dv[r];
    }
  }
  for (; i < i1; ++i) {
    const float dv = dp[i * a.lddy];
    const float d = xp[i * a.ldx] - (a.rms ? 0.0f : a.mean[i]);
    const float t = d * a.rstd[i];
    pg = __builtin_fmaf(dv, t, pg);
    pb = pb + dv;
  }
  if (nblk == 1) {
    if (a.dgamma) a.dgamma[j] = 0.0f + pg;  // the accumulator step: -0 becomes +0
    if (a.dbeta) a.dbeta[j] = 0.0f + pb;
  } else {
    a.ws[ws_index(0, beta, j, nblk, a.cols)] = pg;
    a.ws[ws_index(1, beta, j, nblk, a.cols)] = pb;
  }
}

// Left-to-right sum of the block partials, per column.  The chains are long
// (one add per row block) and each add depends on the previous one, so the
// operands must be at hand: a workgroup owns COLS columns of one tile, all
// its threads copy their partials for up to kCombChunk blocks (both arrays)
// into LDS chain-major ([chain][block], rows padded so that 16-byte reads stay
// aligned and spread over the banks), and then one lane per chain reads four
// consecutive partials per LDS read and adds them in block order.  Chains past
// the last block are padded with +0, which leaves a chain that started at +0
// unchanged.  Whole tiles (COLS = kTile) read contiguous spans; with many
// blocks quarter tiles (COLS = 4) put four times as many workgroups on the
// loads, which bound the time there.
constexpr int kCombChunk = 960;  // blocks per LDS pass: a multiple of 64 (pitch = 4 mod 64)

template <int COLS, int NT, int MAXCHUNK>
__global__ __launch_bounds__(NT) void layernorm_param_combine_kernel(LnParamArgs a, int64_t nblk,
                                                                     int pitch) {
  constexpr int kChains = 2 * COLS;  // dgamma and dbeta of each column
  // loads in flight per thread: a pass of MAXCHUNK blocks in one batch
  constexpr int kBatch = (2 * MAXCHUNK * COLS + NT - 1) / NT;
  static_assert(kTile % COLS == 0, "a workgroup's columns lie in one tile");
  extern __shared__ float buf[];  // [kChains][pitch]
  const int tid = threadIdx.x;
  constexpr int kSub = kTile / COLS;
  const int64_t t0 = static_cast<int64_t>(blockIdx.x / kSub) * kTile;
  const int c0 = static_cast<int>(blockIdx.x % kSub) * COLS;  // first column within the tile
  const int tw = static_cast<int>(a.cols - t0 < kTile ? a.cols - t0 : kTile);
  const int chunk = pitch - 4;  // blocks per pass (a multiple of 4)
  float acc = 0.0f;             // thread ch < kChains: chain ch
  const int ch = tid;
  for (int64_t b0 = 0; b0 < nblk; b0 += chunk) {
    const int nb = static_cast<int>(nblk - b0 < chunk ? nblk - b0 : chunk);
    const int nb4 = (nb + 3) & ~3;
    // stage: element e of one array's share is (block e / COLS, column
    // c0 + e % COLS); consecutive threads read consecutive columns.
    const int span = nb * COLS;
    for (int base = 0; base < 2 * span; base += NT * kBatch) {
      float v[kBatch];
#pragma unroll
      for (int r = 0; r < kBatch; ++r) {
        const int e2 = base + r * NT + tid;
        const int arr = e2 >= span;
        const int e = e2 - arr * span;
        const int b = e / COLS, c = c0 + e % COLS;
        v[r] = 0.0f;
        if (e2 < 2 * span && c < tw) v[r] = a.ws[(arr * a.cols + t0) * nblk + (b0 + b) * tw + c];
      }
#pragma unroll
      for (int r = 0; r < kBatch; ++r) {
        const int e2 = base + r * NT + tid;
        if (e2 < 2 * span) {
          const int arr = e2 >= span;
          const int e = e2 - arr * span;
          buf[(arr * COLS + e % COLS) * pitch + e / COLS] = v[r];
        }
      }
    }
    // +0 past the last block of the pass, up to the next multiple of 4
    if (tid < kChains * 4) {
      const int b = nb + (tid & 3);
      if (b < nb4) buf[(tid >> 2) * pitch + b] = 0.0f;
    }
    __syncthreads();
    if (ch < kChains) {
      const float4* row = reinterpret_cast<const float4*>(buf + ch * pitch);
#pragma unroll 8
      for (int q = 0; q < nb4 / 4; ++q) {
        const float4 v = row[q];
        acc = acc + v.x;
        acc = acc + v.y;
        acc = acc + v.z;
        acc = acc + v.w;
      }
    }
    __syncthreads();
  }
  if (ch < kChains) {
    const int arr = ch / COLS, c = c0 + ch % COLS;
    if (c < tw) {
      if (arr == 0) {
        if (a.dgamma) a.dgamma[t0 + c] = acc;
      } else {
        if (a.dbeta) a.dbeta[t0 + c] = acc;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// LayerNorm backward, fused: input gradient and parameter-gradient block
// partials from one read of X and dY.  One workgroup per block of k_block rows
// with R waves.  The block's rows are taken R at a time: wave w computes the
// input gradient of row chunk + w exactly as the wave kernel does and stages
// t_j and dy_j of that row in LDS; then every thread advances the chains of
// its columns through the R staged rows in row order.  At the end of the
// block the partials go to the workspace (or to dgamma / dbeta directly when
// the rows form a single block).
// ---------------------------------------------------------------------------

constexpr int kFusedChains = 4;  // columns per thread in the chain phase

template <int T, int MAXT, bool PF>
__global__ __launch_bounds__(MAXT) void layernorm_bwd_fused_kernel(RowBwdArgs a, LnParamArgs p,
                                                                   int R, int64_t nblk) {
  extern __shared__ float stage[];  // [R][cols] t, then [R][cols] dy
  const int64_t cols = a.cols;
  float* st = stage;
  float* sd = stage + static_cast<int64_t>(R) * cols;
  const int tid = threadIdx.x;
  const int nthr = R * kWave;
  const int lane = tid & (kWave - 1);
  const int w = tid >> 6;  // (a wave-uniform index measured slower here for 2048-wide rows)
  const int64_t beta = blockIdx.x;
  const int64_t blk = nblk == 1 ? a.rows : p.k_block;
  const int64_t r0 = beta * blk;
  const int64_t r1 = (r0 + blk < a.rows) ? r0 + blk : a.rows;
  const float n = static_cast<float>(cols);
  float gam[T];
#pragma unroll
  for (int t = 0; t < T; ++t) {
    const int64_t j = lane + kWave * t;
    gam[t] = (a.gamma && j < cols) ? a.gamma[j] : 1.0f;
  }
  float pg[kFusedChains], pb[kFusedChains];
#pragma unroll
  for (int k = 0; k < kFusedChains; ++k) {
    pg[k] = 0.0f;
    pb[k] = 0.0f;
  }
  // Rows are software-pipelined (PF): the loads of a wave's next row are
  // issued after this row's dX stores, before the barriers and the chain
  // phase.  The widest rows load at the top of each pass instead, to stay in
  // registers.
  float xv[T], dv[T];
  auto load_row = [&](int64_t row) {
    const float* x = a.Y + row * a.ldy;
    const float* dy = a.dY + row * a.lddy;
#pragma unroll
    for (int t = 0; t < T; ++t) {
      const int64_t j = lane + kWave * t;
      xv[t] = 0.0f;
      dv[t] = 0.0f;
      if (j < cols) {
        xv[t] = x[j];
        dv[t] = dy[j];
      }
    }
  };
  if (PF && r0 + w < r1) load_row(r0 + w);
  for (int64_t c0 = r0; c0 < r1; c0 += R) {
    const int64_t row = c0 + w;
    if (row < r1) {
      if (!PF) load_row(row);
      float* dx = a.dX + row * a.lddx;
      const float mean = a.rms ? 0.0f : a.mean[row], rstd = a.rstd[row];
      float tv[T], gv[T];
      float q = 0.0f;
#pragma unroll
      for (int t = 0; t < T; ++t) {
        const int64_t j = lane + kWave * t;
        tv[t] = 0.0f;
        gv[t] = 0.0f;
        if (j < cols) {
          const float d = xv[t] - mean;
          tv[t] = d * rstd;
          gv[t] = a.gamma ? dv[t] * gam[t] : dv[t];
          st[w * cols + j] = tv[t];
          sd[w * cols + j] = dv[t];
        }
        q = q + gv[t];
      }
      const float am = a.rms ? 0.0f : wave_tree_sum(q) / n;
      float q2 = 0.0f;
#pragma unroll
      for (int t = 0; t < T; ++t)  // past the row: no operation (q2 may be -0)
        if (lane + kWave * t < cols) q2 = __builtin_fmaf(gv[t], tv[t], q2);
      const float bm = wave_tree_sum(q2) / n;
#pragma unroll
      for (int t = 0; t < T; ++t) {
        const int64_t j = lane + kWave * t;
        if (j < cols) {
          const float u = gv[t] - am;
          const float tb = tv[t] * bm;
          const float wv = u - tb;
          st_stream(dx + j, rstd * wv);
        }
      }
      if (PF && row + R < r1) load_row(row + R);  // next row in flight through the barriers and chains
    }
    lds_only_barrier();
    const int nr = static_cast<int>(r1 - c0 < R ? r1 - c0 : R);
#pragma unroll
    for (int k = 0; k < kFusedChains; ++k) {
      const int64_t j = tid + static_cast<int64_t>(k) * nthr;
      if (j < cols) {
        for (int rr = 0; rr < nr; ++rr) {
          const float dyv = sd[rr * cols + j];
          pg[k] = __builtin_fmaf(dyv, st[rr * cols + j], pg[k]);
          pb[k] = pb[k] + dyv;
        }
      }
    }
    lds_only_barrier();
  }
#pragma unroll
  for (int k = 0; k < kFusedChains; ++k) {
    const int64_t j = tid + static_cast<int64_t>(k) * nthr;
    if (j < cols) {
      if (nblk == 1) {
        if (p.dgamma) p.dgamma[j] = 0.0f + pg[k];  // the accumulator step: -0 becomes +0
        if (p.dbeta) p.dbeta[j] = 0.0f + pb[k];
      } else {
        p.ws[ws_index(0, beta, j, nblk, cols)] = pg[k];
        p.ws[ws_index(1, beta, j, nblk, cols)] = pb[k];
      }
    }
  }
}

// ---------------------------------------------------------------------------
// LayerNorm backward, fused, for few row blocks or rows too wide for the
// one-workgroup-per-block kernel: the G workgroups of a block share its work.
// Workgroup (beta, g) computes dX for its share of the block's rows (whole
// rows, one wave each as the wave kernel does, or a group of waves each for
// the widest; the rows are dealt to the G workgroups in turn) and the chains
// of its column slice over all of the block's rows: chunks of rows are loaded
// by all waves (t formed on the way) into LDS and one thread per column
// advances its two chains through each chunk in row order, while the next
// chunk's loads are in flight.  Every row is read
// twice (whole for dX, by slices for the chains); the G workgroups of a block
// are placed on one XCD so the second read can find the rows in that XCD's L2
// (with 4096-wide rows a 64-row block is 2 MB, and part of the second read
// comes from further out).  The rows are read by workgroups other than the
// one writing their dX, so dX may not take the place of X or dY here.
// ---------------------------------------------------------------------------

constexpr int kSplitWaves = 8;

// dX of the rows first + k * stride + q (k >= 0, q < P = kSplitWaves / S,
// below end) by the kSplitWaves waves of a workgroup, S waves per row and P
// rows at a time: wave h of a group (h < S) holds the columns
// lane + 64 * (h * T + t), and each lane's chains pass from wave to wave of
// the group in order through LDS, so the terms meet in the one-wave order and
// the results are the same bits.  Every wave takes part in every step (the
// steps hold workgroup barriers); a group past end works on row first and
// stores nothing.
template <int T, int S>
__device__ __forceinline__ void layernorm_bwd_rows_grouped(const RowBwdArgs& a, int64_t first,
                                                           int64_t stride, int64_t end, int lane,
                                                           int w) {
  constexpr int P = kSplitWaves / S;
  __shared__ float chain_g[P * kWave], chain_gt[P * kWave];
  const int h = w % S;
  const int slot = (w / S) * kWave + lane;
  const float n = static_cast<float>(a.cols);
  auto group_chain = [&](float* ch, auto step) {
#pragma unroll
    for (int k = 0; k < S; ++k) {
      if (h == k) ch[slot] = step(k > 0 ? ch[slot] : 0.0f);
      __syncthreads();
    }
    return ch[slot];
  };
  for (int64_t base = first; base < end; base += stride) {
    const int64_t row = base + w / S;
    const bool live = row < end;
    const int64_t rr = live ? row : first;
    const float* x = a.Y + rr * a.ldy;
    const float* dy = a.dY + rr * a.lddy;
    const float mean = a.rms ? 0.0f : a.mean[rr], rstd = a.rstd[rr];
    const int64_t j0 = lane + int64_t(kWave) * T * h;
    float tv[T], gv[T];
    ln_bwd_terms<T>(a, x, dy, j0, mean, rstd, tv, gv);
    float am = 0.0f;
    if (!a.rms) {  // uniform over the workgroup
      const float q = group_chain(chain_g, [&](float c) {
#pragma unroll
        for (int t = 0; t < T; ++t) c = c + gv[t];  // past the row: +0
        return c;
      });
      am = wave_tree_sum(q) / n;
    }
    const float q2 = group_chain(chain_gt, [&](float c) {
#pragma unroll
      for (int t = 0; t < T; ++t)  // past the row: no operation (c may be -0)
        if (j0 + kWave * t < a.cols) c = __builtin_fmaf(gv[t], tv[t], c);
      return c;
    });
    const float bm = wave_tree_sum(q2) / n;
    if (live) {
      float* dx = a.dX + row * a.lddx;
#pragma unroll
      for (int t = 0; t < T; ++t) {
        const int64_t j = j0 + kWave * t;
        if (j < a.cols) {
          const float u = gv[t] - am;
          const float tb = tv[t] * bm;
          st_stream(dx + j, rstd * (u - tb));
        }
      }
    }
    __syncthreads();  // chains read before the next rows
  }
}

// The column-split kernel's dX rows: one wave per row up to 32 values per
// lane; wider rows (up to 64 values per lane) shared by four waves of 16
// values each, which leaves the registers for two workgroups per compute unit
// (measured faster than one wave of 64 or two of 32; for 32 values per lane
// one wave measured faster than two of 16).
constexpr int kColsplitGroupT = 16;

template <int T, int SWU>
__global__ __launch_bounds__(kSplitWaves * kWave) void layernorm_bwd_colsplit_kernel(
    RowBwdArgs a, LnParamArgs p, int G, int slice, int64_t nblk) {
  constexpr int SW = kWave * SWU;            // LDS pitch: slice columns at most
  constexpr int RPW = SWU <= 2 ? 8 : 4;      // chunk rows per wave
  constexpr int RC = kSplitWaves * RPW;      // rows per chunk
  __shared__ float st[RC * SW], sd[RC * SW];
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int w = wave_id();
  int64_t beta;
  int g;
  const int64_t bid = blockIdx.x;
  if ((nblk & 7) == 0) {  // workgroups are dealt to the 8 XCDs in turn
    const int64_t xcd = bid & 7, s = bid >> 3;
    beta = (s / G) * 8 + xcd;
    g = static_cast<int>(s % G);
  } else {
    beta = bid / G;
    g = static_cast<int>(bid % G);
  }
  const int64_t blk = nblk == 1 ? a.rows : p.k_block;
  const int64_t r0 = beta * blk;
  const int64_t r1 = (r0 + blk < a.rows) ? r0 + blk : a.rows;
  const int64_t c0 = static_cast<int64_t>(g) * slice;
  const int sw = static_cast<int>(c0 + slice < a.cols ? slice : a.cols - c0);

  float xr[RPW][SWU], dr[RPW][SWU];
  auto load_chunk = [&](int64_t i0) {
#pragma unroll
    for (int r = 0; r < RPW; ++r) {
      const int64_t i = i0 + w + kSplitWaves * r;
#pragma unroll
      for (int u = 0; u < SWU; ++u) {
        const int c = lane + kWave * u;
        xr[r][u] = 0.0f;
        dr[r][u] = 0.0f;
        if (i < r1 && c < sw) {
          xr[r][u] = p.X[i * p.ldx + c0 + c];
          dr[r][u] = p.dY[i * p.lddy + c0 + c];
        }
      }
    }
  };
  load_chunk(r0);

  // dX of the block's rows, dealt to its G workgroups in turn, P rows to a
  // workgroup at a time (one wave per row, P = kSplitWaves, or for wide rows a
  // group of waves per row): the workgroups go through the rows in the order
  // the chains' chunks read them, so that the second read of a row tends to
  // find it in L2.  (A chunk's dX just before its chains, which brings the
  // two reads together, measured slower: each chunk then waits for its own
  // rows.)
  if constexpr (T > 32) {
    static_assert(T % kColsplitGroupT == 0 && kSplitWaves % (T / kColsplitGroupT) == 0,
                  "row groups must tile the workgroup");
    constexpr int S = T / kColsplitGroupT, P = kSplitWaves / S;
    layernorm_bwd_rows_grouped<kColsplitGroupT, S>(a, r0 + int64_t(g) * P, int64_t(P) * G, r1,
                                                   lane, w);
  } else {
    const int64_t stride = int64_t(kSplitWaves) * G;
    for (int64_t row = r0 + int64_t(g) * kSplitWaves + w; row < r1; row += stride)
      layernorm_bwd_row<T>(a, row, lane);
  }

  float pg = 0.0f, pb = 0.0f;
  for (int64_t i0 = r0; i0 < r1; i0 += RC) {
#pragma unroll
    for (int r = 0; r < RPW; ++r) {
      const int rr = w + kSplitWaves * r;
      const int64_t i = i0 + rr;
      if (i < r1) {
        const float mean = p.rms ? 0.0f : p.mean[i], rstd = p.rstd[i];
#pragma unroll
        for (int u = 0; u < SWU; ++u) {
          const float d = xr[r][u] - mean;
          st[rr * SW + lane + kWave * u] = d * rstd;
          sd[rr * SW + lane + kWave * u] = dr[r][u];
        }
      }
    }
    __syncthreads();
    if (i0 + RC < r1) load_chunk(i0 + RC);
    const int nr = static_cast<int>(r1 - i0 < RC ? r1 - i0 : RC);
    if (tid < sw) {
      for (int rr = 0; rr < nr; ++rr) {
        const float dyv = sd[rr * SW + tid];
        pg = __builtin_fmaf(dyv, st[rr * SW + tid], pg);
        pb = pb + dyv;
      }
    }
    __syncthreads();
  }
  if (tid < sw) {
    const int64_t j = c0 + tid;
    if (nblk == 1) {
      if (p.dgamma) p.dgamma[j] = 0.0f + pg;  // the accumulator step: -0 becomes +0
      if (p.dbeta) p.dbeta[j] = 0.0f + pb;
    } else {
      p.ws[ws_index(0, beta, j, nblk, a.cols)] = pg;
      p.ws[ws_index(1, beta, j, nblk, a.cols)] = pb;
    }
  }
}

// ---------------------------------------------------------------------------
// GELU backward and Adam: elementwise, 16-byte accesses where every operand
// is 16-byte aligned.
// ---------------------------------------------------------------------------

struct GeluTanhGrad {
  __device__ __forceinline__ float operator()(float x) const { return rep_gelu_grad(x); }
};
struct GeluErfGrad {
  __device__ __forceinline__ float operator()(float x) const { return rep_gelu_erf_grad(x); }
};

template <class Grad>
__global__ __launch_bounds__(1024) void gelu_bwd_kernel(int64_t n, const float* x, const float* dy,
                                                        float* dx, int vec) {
  const Grad grad;
  const int64_t tid = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
  int64_t done = 0;
  if (vec) {
    const int64_t n4 = n / 4;
    const float4* x4 = reinterpret_cast<const float4*>(x);
    const float4* d4 = reinterpret_cast<const float4*>(dy);
    float4* o4 = reinterpret_cast<float4*>(dx);
    for (int64_t i = tid; i < n4; i += stride) {
      const float4 xv = x4[i];
      const float4 dv = d4[i];
      float4 o;
      o.x = dv.x * grad(xv.x);
      o.y = dv.y * grad(xv.y);
      o.z = dv.z * grad(xv.z);
      o.w = dv.w * grad(xv.w);
      st_stream(o4 + i, o);
    }
    done = n4 * 4;
  }
  for (int64_t i = done + tid; i < n; i += stride) st_stream(dx + i, dy[i] * grad(x[i]));
}

// One element of the Adam / AdamW update (decay: 0 none, 1 decoupled, 2 coupled).
__device__ __forceinline__ void adam_one(const AdamScalars& s, float& p, float g, float& m,
                                         float& v) {
  if (s.decay == 1) p = p * s.dec;
  if (s.decay == 2) g = __builtin_fmaf(s.wd, p, g);
  const float cg = s.c1 * g;
  m = __builtin_fmaf(s.b1, m, cg);
  const float gg = g * g;
  const float cgg = s.c2 * gg;
  v = __builtin_fmaf(s.b2, v, cgg);
  const float rv = __builtin_sqrtf(v);
  const float q = rv / s.sbc2;
  const float den = q + s.eps;
  const float upd = m / den;
  const float su = s.step * upd;
  p = p - su;
}

__global__ __launch_bounds__(1024) void adam_kernel(int64_t n, float* p, const float* g, float* m,
                                                    float* v, AdamScalars s, int vec) {
  const int64_t tid = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
  int64_t done = 0;
  if (vec) {
    const int64_t n4 = n / 4;
    float4* p4 = reinterpret_cast<float4*>(p);
    const float4* g4 = reinterpret_cast<const float4*>(g);
    float4* m4 = reinterpret_cast<float4*>(m);
    float4* v4 = reinterpret_cast<float4*>(v);
    for (int64_t i = tid; i < n4; i += stride) {
      float4 pv = p4[i], mv = m4[i], vv = v4[i];
      const float4 gv = g4[i];
      adam_one(s, pv.x, gv.x, mv.x, vv.x);
      adam_one(s, pv.y, gv.y, mv.y, vv.y);
      adam_one(s, pv.z, gv.z, mv.z, vv.z);
      adam_one(s, pv.w, gv.w, mv.w, vv.w);
      st_stream(p4 + i, pv);
      st_stream(m4 + i, mv);
      st_stream(v4 + i, vv);
    }
    done = n4 * 4;
  }
  for (int64_t i = done + tid; i < n; i += stride) {
    float pv = p[i], mv = m[i], vv = v[i];
    adam_one(s, pv, g[i], mv, vv);
    st_stream(p + i, pv);
    st_stream(m + i, mv);
    st_stream(v + i, vv);
  }
}

using WaveBwdKernel = void (*)(RowBwdArgs, int);

WaveBwdKernel pick_softmax_bwd(int64_t cols) {
  if (cols <= kWave * 1) return softmax_bwd_wave_kernel<1>;
  if (cols <= kWave * 2) return softmax_bwd_wave_kernel<2>;
  if (cols <= kWave * 4) return softmax_bwd_wave_kernel<4>;
  if (cols <= kWave * 8) return softmax_bwd_wave_kernel<8>;
  if (cols <= kWave * 16) return softmax_bwd_wave_kernel<16>;
  if (cols <= kWave * 32) return softmax_bwd_wave_kernel<32>;
  return softmax_bwd_wave_kernel<64>;
}

WaveBwdKernel pick_layernorm_bwd(int64_t cols) {
  if (cols <= kWave * 1) return layernorm_bwd_wave_kernel<1>;
  if (cols <= kWave * 2) return layernorm_bwd_wave_kernel<2>;
  if (cols <= kWave * 4) return layernorm_bwd_wave_kernel<4>;
  if (cols <= kWave * 8) return layernorm_bwd_wave_kernel<8>;
  if (cols <= kWave * 12) return layernorm_bwd_wave_kernel<12>;
  if (cols <= kWave * 16) return layernorm_bwd_wave_kernel<16>;
  if (cols <= kWave * 32) return layernorm_bwd_wave_kernel<32>;
  return layernorm_bwd_wave_kernel<64>;
}

using SplitBwdKernel = void (*)(RowBwdArgs);

template <template <int> class K>
SplitBwdKernel pick_split_bwd(int64_t cols, int S) {
  const int64_t per_lane = (cols + int64_t(kWave) * S - 1) / (int64_t(kWave) * S);
  if (per_lane <= 1) return K<1>::fn;
  if (per_lane <= 2) return K<2>::fn;
  if (per_lane <= 4) return K<4>::fn;
  if (per_lane <= 8) return K<8>::fn;
  if (per_lane <= 16) return K<16>::fn;
  if (per_lane <= 32) return K<32>::fn;
  return nullptr;
}
template <int T> struct SoftmaxBwdSplit { static constexpr SplitBwdKernel fn = softmax_bwd_split_kernel<T>; };
template <int T> struct LayernormBwdSplit { static constexpr SplitBwdKernel fn = layernorm_bwd_split_kernel<T>; };

hipError_t launch_split_bwd(SplitBwdKernel k, const RowBwdArgs& a, int S, hipStream_t s) {
  if (!k) return hipErrorInvalidValue;
  const int64_t cap = int64_t(1) << 30;
  hipLaunchKernelGGL(k, dim3(static_cast<unsigned>(a.rows < cap ? a.rows : cap)),
                     dim3(kWave * S), 0, s, a);
  return hipGetLastError();
}

using FusedKernel = void (*)(RowBwdArgs, LnParamArgs, int, int64_t);

// Kernels for R <= 8 waves (512 threads); the widest rows (32 values per
// lane) load each row at the top of its pass instead of one pass ahead.
FusedKernel pick_layernorm_fused(int64_t cols) {
  if (cols <= kWave * 1) return layernorm_bwd_fused_kernel<1, 512, true>;
  if (cols <= kWave * 2) return layernorm_bwd_fused_kernel<2, 512, true>;
  if (cols <= kWave * 4) return layernorm_bwd_fused_kernel<4, 512, true>;
  if (cols <= kWave * 8) return layernorm_bwd_fused_kernel<8, 512, true>;
  if (cols <= kWave * 12) return layernorm_bwd_fused_kernel<12, 512, true>;
  if (cols <= kWave * 16) return layernorm_bwd_fused_kernel<16, 512, true>;
  return layernorm_bwd_fused_kernel<32, 512, false>;
}

unsigned row_grid(int64_t rows) {
  const int64_t cap = int64_t(1) << 30;
  return static_cast<unsigned>(rows < cap ? rows : cap);
}

int64_t ew_blocks(int64_t items, int threads, int max_blocks) {
  int64_t blocks = (items + threads - 1) / threads;
  if (max_blocks > 0 && blocks > max_blocks) blocks = max_blocks;
  const int64_t cap = int64_t(1) << 30;
  if (blocks > cap) blocks = cap;
  if (blocks < 1) blocks = 1;
  return blocks;
}

bool aligned16(const void* p) { return reinterpret_cast<uintptr_t>(p) % 16 == 0; }

}  // namespace

hipError_t launch_softmax_bwd_wave(const RowBwdArgs& a, int wpb, hipStream_t s) {
  if (a.cols > kWave * 32 && wpb > 4) wpb = 4;
  const int64_t blocks = (a.rows + wpb - 1) / wpb;
  hipLaunchKernelGGL(pick_softmax_bwd(a.cols), dim3(static_cast<unsigned>(blocks)),
                     dim3(kWave * wpb), 0, s, a, wpb);
  return hipGetLastError();
}

hipError_t launch_softmax_bwd_generic(const RowBwdArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(softmax_bwd_generic_kernel, dim3(row_grid(a.rows)), dim3(kWave), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_layernorm_bwd_wave(const RowBwdArgs& a, int wpb, hipStream_t s) {
  const int64_t blocks = (a.rows + wpb - 1) / wpb;
  hipLaunchKernelGGL(pick_layernorm_bwd(a.cols), dim3(static_cast<unsigned>(blocks)),
                     dim3(kWave * wpb), 0, s, a, wpb);
  return hipGetLastError();
}

hipError_t launch_softmax_bwd_split(const RowBwdArgs& a, int S, hipStream_t s) {
  return launch_split_bwd(pick_split_bwd<SoftmaxBwdSplit>(a.cols, S), a, S, s);
}

hipError_t launch_layernorm_bwd_split(const RowBwdArgs& a, int S, hipStream_t s) {
  return launch_split_bwd(pick_split_bwd<LayernormBwdSplit>(a.cols, S), a, S, s);
}

hipError_t launch_layernorm_bwd_generic(const RowBwdArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(layernorm_bwd_generic_kernel, dim3(row_grid(a.rows)), dim3(kWave), 0, s, a);
  return hipGetLastError();
}

int64_t layernorm_param_blocks(int64_t rows, int64_t k_block) {
  if (k_block <= 0 || k_block >= rows) return 1;  // rows == 0: one empty block, gradients +0
  return (rows + k_block - 1) / k_block;
}

int64_t layernorm_param_grid(int64_t rows, int64_t cols, int64_t k_block) {
  const int64_t groups = (cols + kParamThreads - 1) / kParamThreads;
  return layernorm_param_blocks(rows, k_block) * groups;
}

hipError_t launch_layernorm_param_combine(const LnParamArgs& a, int64_t nblk, hipStream_t s) {
  const int64_t tiles = (a.cols + kTile - 1) / kTile;
  const int64_t chunk = nblk < kCombChunk ? (nblk + 3) & ~int64_t(3) : kCombChunk;
  const int pitch = static_cast<int>(chunk) + 4;
  if (nblk <= 256) {  // whole tiles
    const size_t lds = sizeof(float) * 2 * kTile * static_cast<size_t>(pitch);
    hipLaunchKernelGGL((layernorm_param_combine_kernel<kTile, 512, 256>),
                       dim3(static_cast<unsigned>(tiles)), dim3(512), lds, s, a, nblk, pitch);
  } else {  // quarter tiles
    const size_t lds = sizeof(float) * 2 * 4 * static_cast<size_t>(pitch);
    hipLaunchKernelGGL((layernorm_param_combine_kernel<4, 256, kCombChunk>),
                       dim3(static_cast<unsigned>(tiles * (kTile / 4))), dim3(256), lds, s, a, nblk,
                       pitch);
  }
  return hipGetLastError();
}

hipError_t launch_layernorm_param(const LnParamArgs& a, hipStream_t s) {
  const int64_t nblk = layernorm_param_blocks(a.rows, a.k_block);
  const int64_t blk = nblk == 1 ? a.rows : a.k_block;
  const int64_t groups = (a.cols + kParamThreads - 1) / kParamThreads;
  hipLaunchKernelGGL(layernorm_param_partial_kernel, dim3(static_cast<unsigned>(nblk * groups)),
                     dim3(kParamThreads), 0, s, a, groups, blk, nblk);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || nblk == 1) return e;
  return launch_layernorm_param_combine(a, nblk, s);
}

// Dynamic LDS a workgroup may use on the current device, at most 128 KiB.
int64_t lds_budget_bytes() {
  int dev = 0, v = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess ||
      v <= 0)
    return 64 * 1024;
  return v < 128 * 1024 ? v : 128 * 1024;
}

int layernorm_fused_rows(int64_t rows, int64_t cols, int64_t k_block, int requested) {
  // R rows staged per pass: LDS holds 2 * R * cols floats; the chain phase
  // needs R * 64 * kFusedChains >= cols; R <= 8 (512 threads, which leaves
  // each wave the registers for its row and the next one in flight).
  // Without a request: 8.
  const int64_t c = cols > 0 ? cols : 1;
  const int64_t fit = lds_budget_bytes() / (8 * c);
  const int64_t rmax = 8;
  const int64_t rmin = (c + kWave * kFusedChains - 1) / (kWave * kFusedChains);
  int64_t r = fit < rmax ? fit : rmax;
  if (requested > 0 && requested < r) r = requested;
  if (r < rmin) r = rmin;
  if (r > fit || r > rmax) return 0;  // does not fit: use the unfused kernels
  return static_cast<int>(r);
}

hipError_t launch_layernorm_bwd_fused(const RowBwdArgs& a, const LnParamArgs& p, int R,
                                      hipStream_t s) {
  const int64_t nblk = layernorm_param_blocks(a.rows, p.k_block);
  const size_t lds = sizeof(float) * 2 * static_cast<size_t>(R) * static_cast<size_t>(a.cols);
  hipLaunchKernelGGL(pick_layernorm_fused(a.cols), dim3(static_cast<unsigned>(nblk)),
                     dim3(R * kWave), lds, s, a, p, R, nblk);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || nblk == 1) return e;
  return launch_layernorm_param_combine(p, nblk, s);
}

using ColsplitKernel = void (*)(RowBwdArgs, LnParamArgs, int, int, int64_t);

template <int SWU>
ColsplitKernel pick_colsplit_t(int64_t cols) {
  if (cols <= kWave * 1) return layernorm_bwd_colsplit_kernel<1, SWU>;
  if (cols <= kWave * 2) return layernorm_bwd_colsplit_kernel<2, SWU>;
  if (cols <= kWave * 4) return layernorm_bwd_colsplit_kernel<4, SWU>;
  if (cols <= kWave * 8) return layernorm_bwd_colsplit_kernel<8, SWU>;
  if (cols <= kWave * 12) return layernorm_bwd_colsplit_kernel<12, SWU>;
  if (cols <= kWave * 16) return layernorm_bwd_colsplit_kernel<16, SWU>;
  if (cols <= kWave * 32) return layernorm_bwd_colsplit_kernel<32, SWU>;
  return layernorm_bwd_colsplit_kernel<64, SWU>;
}

bool layernorm_colsplit_plan(int64_t rows, int64_t cols, int64_t k_block, ColsplitPlan* pl) {
  // Rows a wave holds in registers, and few row blocks (fewer than one per
  // compute unit) or rows too wide for the one-workgroup-per-block kernel's
  // LDS stage; about 512 workgroups, slices of 16 to 256 columns.
  if (rows < 1 || cols < 1 || cols > kWave * kMaxPerLane || k_block < 1) return false;
  const int64_t nblk = layernorm_param_blocks(rows, k_block);
  if (nblk >= 256 && layernorm_fused_rows(rows, cols, k_block, 0) >= 1) return false;
  int64_t g0 = (512 + nblk - 1) / nblk;
  const int64_t gcol = (cols + kWave - 1) / kWave;
  if (g0 > gcol) g0 = gcol;
  int64_t slice = (cols + g0 - 1) / g0;
  slice = (slice + 15) & ~int64_t(15);
  if (slice > kWave * 4) slice = kWave * 4;
  pl->slice = static_cast<int>(slice);
  pl->G = static_cast<int>((cols + slice - 1) / slice);
  pl->swu = static_cast<int>((slice + kWave - 1) / kWave);
  return true;
}

hipError_t launch_layernorm_bwd_colsplit(const RowBwdArgs& a, const LnParamArgs& p,
                                         const ColsplitPlan& pl, hipStream_t s) {
  const int64_t nblk = layernorm_param_blocks(a.rows, p.k_block);
  ColsplitKernel k = pl.swu == 1   ? pick_colsplit_t<1>(a.cols)
                     : pl.swu == 2 ? pick_colsplit_t<2>(a.cols)
                     : pl.swu == 3 ? pick_colsplit_t<3>(a.cols)
                                   : pick_colsplit_t<4>(a.cols);
  hipLaunchKernelGGL(k, dim3(static_cast<unsigned>(nblk * pl.G)), dim3(kSplitWaves * kWave), 0,
                     s, a, p, pl.G, pl.slice, nblk);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || nblk == 1) return e;
  return launch_layernorm_param_combine(p, nblk, s);
}

hipError_t launch_gelu_bwd(int64_t n, const float* x, const float* dy, float* dx, int threads,
                           int max_blocks, hipStream_t s, bool erf_form) {
  const bool vec = aligned16(x) && aligned16(dy) && aligned16(dx);
  const int64_t blocks = ew_blocks(vec ? (n + 3) / 4 : n, threads, max_blocks);
  if (erf_form)
    hipLaunchKernelGGL(gelu_bwd_kernel<GeluErfGrad>, dim3(static_cast<unsigned>(blocks)),
                       dim3(threads), 0, s, n, x, dy, dx, vec ? 1 : 0);
  else
    hipLaunchKernelGGL(gelu_bwd_kernel<GeluTanhGrad>, dim3(static_cast<unsigned>(blocks)),
                       dim3(threads), 0, s, n, x, dy, dx, vec ? 1 : 0);
  return hipGetLastError();
}

hipError_t launch_adam(int64_t n, float* p, const float* g, float* m, float* v,
                       const AdamScalars& sc, int threads, int max_blocks, hipStream_t s) {
  const bool vec = aligned16(p) && aligned16(g) && aligned16(m) && aligned16(v);
  const int64_t blocks = ew_blocks(vec ? (n + 3) / 4 : n, threads, max_blocks);
  hipLaunchKernelGGL(adam_kernel, dim3(static_cast<unsigned>(blocks)), dim3(threads), 0, s, n, p, g,
                     m, v, sc, vec ? 1 : 0);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Fixed scratch for the LayerNorm backward entry point that allocates nothing
// (repops_layernorm_backward_rows_noalloc): the block partials of the
// parameter gradients go to this array instead of a caller's workspace.  Each
// device holds its own copy for the life of the process.  In host code the
// array's name only stands in for it, so the device address is looked up once
// per device (with that device current) and kept; calls on one device share
// the array.  Every partial the combine reads is written first in the same
// call, so nothing needs clearing between calls.
// ---------------------------------------------------------------------------
static __device__ __align__(256) float scratch[kNoallocScratchBytes / sizeof(float)];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};
}  // namespace

hipError_t noalloc_scratch(void** ptr) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace repops
