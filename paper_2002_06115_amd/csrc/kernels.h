// kernels.h -- launchers of the gfx950 kernels (internal).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace kbf {

// How the columns of a b-wide row are spread over the lanes of a lane group.
struct ColumnTiling {
  int vec;       // floats per lane per access: 4 (b % 4 == 0) or 1
  int lpt;       // lanes per group (power of two, <= 64): one group sums one piece
  int width;     // columns one group covers, lpt * vec
  int n_slices;  // ceil(b / width): grid y dimension
};
ColumnTiling column_tiling(int32_t b);

// Segmented gather-multiply-sum over pieces (every pass of the library):
//   acc = sum over positions p of the piece of  w[p] * A[a[p]] (.) B[b_id[p]]
// with pairs[p] = (a[p], b_id[p]).  The result goes to out row dst (rounded to
// float) or to workspace slot -(dst + 1) (double).  B_rows is the row count of
// B; when b_in_lds is set the block copies B's column slice into LDS first.
struct PiecesArgs {
  const int4 *pieces;
  int64_t n_pieces;
  const int2 *pairs;
  const float *weight;  // nullptr = 1
  const float *A;
  const float *B;
  int64_t B_rows;
  int32_t b;
  float *out;
  double *slots;
};
hipError_t launch_pieces(const PiecesArgs &a, bool b_in_lds, int max_blocks, hipStream_t s);

// Bytes of LDS the pieces kernel needs to hold B's column slice.
size_t pieces_lds_bytes(int32_t b, int64_t B_rows);

// Sums workspace slots in order (one combine level).
hipError_t launch_combine(const int4 *tasks, int64_t n_tasks, double *slots, int32_t b,
                          float *out, hipStream_t s);

// Writes +0.0 to the listed rows of out ([rows][b]).
hipError_t launch_zero_rows(const int32_t *rows, int64_t n_rows, int32_t b, float *out,
                            hipStream_t s);

// Makes the LDS variant of the pieces kernel able to use `bytes` of dynamic LDS.
hipError_t prepare_pieces_lds(int32_t b, size_t bytes);

}  // namespace kbf
