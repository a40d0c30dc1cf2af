// Workspace sizing shared by the kernels and the host-only planner.
#pragma once
#include <stdint.h>

namespace tps {

// Column reductions split the rows into at most 16 segments (a multiple of 32
// rows, at least 64); each segment leaves one f32 partial per column.
inline int64_t colsum_seg_rows(int64_t rows) {
  int64_t s = (rows + 15) / 16;
  s = (s + 31) / 32 * 32;
  return s < 64 ? 64 : s;
}
inline int64_t colsum_segments(int64_t rows) {
  const int64_t s = colsum_seg_rows(rows);
  return rows > 0 ? (rows + s - 1) / s : 1;
}
// f32 partials of a column reduction over rows x cols
inline uint64_t colsum_ws_elems(int64_t rows, int64_t cols) { return (uint64_t)(colsum_segments(rows) * cols); }

}  // namespace tps
