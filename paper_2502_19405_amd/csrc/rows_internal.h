// Split-row launchers of the forward row operations (rows.hip): one row per
// workgroup of S waves (S = 2, 4, 8), at most 32 values per lane.
#pragma once

#include <hip/hip_runtime.h>

#include "repops_internal.h"

namespace repops {

// Waves per row that a wide row is split over when the launch leaves the
// choice open: rows up to `wave_cols` columns stay on one wave (1024; the
// callers pass what measured fastest for their operator: 2048 for the softmax
// and the norm backward's input gradient, 4096 for the softmax backward);
// wider rows get the fewest waves (2, 4, 8) that leave at most `per_lane`
// values per lane (16, or 8 for the softmax backward and the RMSNorm, which
// measured best there), or 8.
// (Measured on 4096- and 8192-wide rows: 16 values per lane is within a few
// percent of 8, 16 waves per row is far slower.)
inline int auto_row_split(int64_t cols, int per_lane = 16, int64_t wave_cols = 1024) {
  if (cols <= wave_cols) return 1;
  int S = 2;
  while (S < 8 && cols > int64_t(64) * per_lane * S) S *= 2;
  return S;
}

// Widest row a split over S waves takes (32 values per lane).
inline int64_t split_max_cols(int S) { return int64_t(64) * 32 * S; }

hipError_t launch_softmax_split(const RowArgs& a, int S, hipStream_t s);
hipError_t launch_layernorm_split(const RowArgs& a, int S, hipStream_t s);
// Widest row a split over S waves takes.
int64_t rows_split_max_cols(int S);

}  // namespace repops
