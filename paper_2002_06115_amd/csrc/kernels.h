// kernels.h -- launchers of the gfx950 kernels (internal).
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>
#include <string>

namespace kbf {

// How the columns of a b-wide row are spread over the lanes of a lane group.
struct ColumnTiling {
  int vec;       // floats per lane per access: 4 (b % 4 == 0) or 1
  int lpt;       // lanes per group (power of two, <= 32): one group walks one chunk
  int width;     // columns one group covers, lpt * vec
  int n_slices;  // ceil(b / width): grid y dimension
};
ColumnTiling column_tiling(int32_t b);
// The same with lane groups of at most max_lpt lanes (a power of two <= 32).
ColumnTiling column_tiling_max(int32_t b, int max_lpt);

// Chunk lengths must be multiples of this (the kernel's step, kUnroll entries).
constexpr int32_t kChunkQuantum = 8;

// Segmented gather-multiply-sum over one layout's entry stream (every pass
// of the library).  entries[p] = (x, y): a triple x = a | run-start flag,
// y = b_id, or a marker x = -1, y = target (row, -(slot + 1), or INT32_MIN
// for none); n is a multiple of chunk, and chunk of kChunkQuantum.  Lane
// group walks the entries of one chunk at a time ([c * chunk, (c + 1) * chunk)):
//     held = B[b_id]                          at a triple flagged run-start
//     acc += w[p] * A[a] (.) held             for every triple
//     target = acc (float row / double slot), acc = 0   at a marker
// A has A_rows rows and B has B_rows rows of b floats.  With `residual` set
// a marker writing row j writes acc + gamma * Z[j] instead (Z has out_rows
// rows): with Z = A the residual hop follow(X, R) + gamma * X of the
// KB-completion chains and its dX pass (A = dY there); with any other Z the
// accumulating follow, Z = out itself adding into the output in place (each
// row's Z is read by the thread that then writes it).  Raw buffer loads need
// Z = A; another Z takes the plain-load path.
// At most this many chunk lists (one per XCD); see StreamArgs::list_chunk.
constexpr int kMaxChunkLists = 8;

struct StreamArgs {
  const int2 *entries;
  const float *weights;  // per entry, nullptr for a hard KB
  int64_t n;
  int32_t chunk;
  const float *A;
  int64_t A_rows;
  const float *B;
  int64_t B_rows;
  int32_t b;
  float *out;
  int64_t out_rows;
  double *slots;
  int64_t n_slots;
  int32_t residual;
  float gamma;
  const float *Z;  // the rows added at markers when residual is set
  // Chunk lists: workgroups with blockIdx.x % n_lists == x walk chunks
  // [list_chunk[x], list_chunk[x + 1]) (list x is meant for XCD x, which runs
  // those workgroups); n_lists = 1 is one list of every chunk.
  int32_t n_lists;
  int64_t list_chunk[kMaxChunkLists + 1];
};
// Largest B column slice (B_rows * slice width * 4 bytes) the stream kernel
// copies into LDS with two workgroups per CU (two copies fit a CU's 160 KB),
// and with one workgroup per CU (hard KB only).
constexpr size_t kMaxLdsB = 80 * 1024;
constexpr size_t kMaxLdsBig = 160 * 1024;

struct StreamOptions {
  // Forces the plain-load variant (used anyway for tables of 4 GB or more)
  // so it can be tested at small sizes.
  bool plain_loads = false;
  // Stage B in LDS when its slice fits (raw-buffer path only); off keeps B
  // rows in registers, the variant used for larger tables.
  bool b_in_lds = true;
  int n_cu = 1;  // compute units of the device, for the LDS variant's grid
  int max_lpt = 32;  // widest lane group of the register variant (narrower: more column slices)
};
// With start / stop events the kernel is launched with hipExtLaunchKernel,
// which sets them to the kernel's own start and end timestamps (no event
// packets of their own on the stream).
hipError_t launch_stream(const StreamArgs &a, const StreamOptions &o, hipStream_t s,
                         hipEvent_t start = nullptr, hipEvent_t stop = nullptr);
// The kernel launch_stream would launch for `a`, as profilers print it
// ("stream_kernel<4, 8, true, false, false, true>"); "" when nothing would be
// launched.  Likewise for launch_tail and launch_combine.
std::string describe_stream(const StreamArgs &a, const StreamOptions &o);

// Sums workspace slots in order (one combine level).  A final row write adds
// gamma * res[row] when res is not null (residual hop, accumulating follow;
// res may be out itself).
hipError_t launch_combine(const int4 *tasks, int64_t n_tasks, double *slots, int64_t n_slots,
                          int32_t b, float *out, int64_t out_rows, const float *res, float gamma,
                          hipStream_t s);

// One launch for a pass's first combine level (tasks of that level, as for
// launch_combine) and its empty rows: +0.0 to the rows of out in the pieces
// (first row, count), or gamma * res[row] when res is not null (residual
// hop).  combine_blocks is set by the launcher.
struct TailArgs {
  const int4 *tasks;
  int64_t n_tasks;
  double *slots;
  int64_t n_slots;
  const int2 *pieces;
  int64_t n_pieces;
  int32_t b;
  float *out;
  int64_t out_rows;
  const float *res;
  float gamma;
  int64_t combine_blocks;
};
hipError_t launch_tail(const TailArgs &a, hipStream_t s);
std::string describe_tail(const TailArgs &a);
std::string describe_combine(int32_t b);

// The fixed device scratch of kb_follow_noalloc: kStaticScratchBytes per
// device, resolved with that device current (static_scratch.hip).  *ptr is
// the current device's copy; every caller on one device shares it.
constexpr size_t kStaticScratchBytes = size_t(64) << 20;
hipError_t static_scratch(int device, void **ptr);

// Bounds violations counted by a checked build (KBFOLLOW_CHECKED) on the
// current device since the last reset; hipErrorNotSupported otherwise.
hipError_t checked_violations(unsigned long long *count, bool reset);

}  // namespace kbf
