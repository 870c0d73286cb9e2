// kernels.h -- launchers of the gfx950 kernels (internal).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace kbf {

// How the columns of a b-wide row are spread over the lanes of a lane group.
struct ColumnTiling {
  int vec;       // floats per lane per access: 4 (b % 4 == 0) or 1
  int lpt;       // lanes per group (power of two, <= 64): one group walks one chunk
  int width;     // columns one group covers, lpt * vec
  int n_slices;  // ceil(b / width): grid y dimension
};
ColumnTiling column_tiling(int32_t b);

// Segmented gather-multiply-sum over a sorted triple stream (every pass of
// the library).  entries[p] = (a, b_id, flush, weight bits) for position p;
// lane group g walks positions [g * chunk, (g + 1) * chunk) accumulating
//     acc += w[p] * A[a[p]] (.) B[b_id[p]]
// and after position p writes acc to out row flush[p] (rounded to float) or
// to workspace slot -(flush[p] + 1) (double) and restarts from zero, unless
// flush[p] is kNoFlush.  B_rows is the row count of B; with b_in_lds the
// workgroup first copies B's column slice into LDS.
struct StreamArgs {
  const int4 *entries;
  int64_t n;
  int32_t chunk;
  const float *A;
  const float *B;
  int64_t B_rows;
  int32_t b;
  float *out;
  double *slots;
};
hipError_t launch_stream(const StreamArgs &a, bool weighted, bool b_in_lds, int max_blocks,
                         hipStream_t s);

// Bytes of LDS the stream kernel needs to hold B's column slice.
size_t stream_lds_bytes(int32_t b, int64_t B_rows);

// Sums workspace slots in order (one combine level).
hipError_t launch_combine(const int4 *tasks, int64_t n_tasks, double *slots, int32_t b,
                          float *out, hipStream_t s);

// Writes +0.0 to the listed rows of out ([rows][b]).
hipError_t launch_zero_rows(const int32_t *rows, int64_t n_rows, int32_t b, float *out,
                            hipStream_t s);

// Lets the LDS variants of the stream kernel use `bytes` of dynamic LDS.
hipError_t prepare_stream_lds(int32_t b, size_t bytes);

}  // namespace kbf
