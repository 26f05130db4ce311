// Device-side addressing of the packed checkpoint layout, shared by the kernels that
// read or write it.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace dasc {

// Row offset (in rows) of packed row j of checkpoint slot `slot` in the
// [T, n_slots, slice_rows] layout of Sec. 4.3 (rank r holds packed rows
// [r * slice_rows, (r + 1) * slice_rows)); the flat layout (one slice) needs no division.
__device__ inline int64_t slice_row(int64_t j, int64_t slice_rows, int64_t n_rows,
                                    int64_t n_slots, int64_t slot) {
  const int64_t r = slice_rows >= n_rows ? 0 : int64_t(uint32_t(j) / uint32_t(slice_rows));
  return (r * n_slots + slot) * slice_rows + (j - r * slice_rows);
}

// The packed checkpoint as the fused restore-and-refresh kernels read it.
struct CkptView {
  const float* ckpt;
  int64_t n_slots, slice_rows, n_rows;
  const int32_t* slot;   // checkpoint slot per request
};

// Where a dense row of a head sits in checkpoint slot `cslot`, as a float offset of a
// row of `d` words: kOmitted for an omitted row (inv_row < 0), kNoRow for an index past
// the packed rows (restores as +0.0, as in the plain restore).
constexpr int64_t kOmitted = -1, kNoRow = -2;
__device__ inline int64_t ckpt_row_offset(int64_t p, const CkptView& ck, int64_t cslot, int d) {
  return p < 0 ? kOmitted
       : p >= ck.n_rows ? kNoRow
       : slice_row(p, ck.slice_rows, ck.n_rows, ck.n_slots, cslot) * d;
}

}  // namespace dasc
