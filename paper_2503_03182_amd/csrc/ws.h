// Workspace sizing shared by the kernels and the host-only planner.
#pragma once
#include <stdint.h>

namespace tps {

constexpr int kColsumRowsPerPart = 32;  // rows summed per partial in column reductions

// f32 partials of a column reduction over rows x cols (one value per column
// and per part of kColsumRowsPerPart rows).
inline uint64_t colsum_ws_elems(int64_t rows, int64_t cols) {
  const int64_t parts = (rows + kColsumRowsPerPart - 1) / kColsumRowsPerPart;
  return (uint64_t)(parts * cols);
}

}  // namespace tps
