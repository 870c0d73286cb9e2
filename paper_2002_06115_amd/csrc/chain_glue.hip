// chain_glue.hip -- column-wise operations between the hops of a multi-hop
// chain (Sec. 3.2): softmax over relations, L1 normalisation of entity
// weights, softmax cross-entropy of the last hop, and their backwards.
//
// Every operation reduces over the n rows of each column of an [n][b]
// batch-contiguous array.  A workgroup of 1024 threads owns 16 consecutive
// columns: 64 row phases of 16 lanes, lane c on column c of the tile, so a
// wavefront reads four 64-byte row segments per load.  Phase p visits rows
// p, p + 64, p + 128, ... in that order, with the loads of four such rows
// issued before their values are used (the reads of a column pass are then
// four deep in flight per thread, 256 rows per workgroup).  The 64 phase
// partials of a column are combined through LDS by a fixed pairwise tree
// (phase p with p + 32, then p + 16, ...).  Sums and maxima are taken in
// double, in that fixed order, so results are bitwise reproducible.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "kbchain.h"

namespace {

constexpr int kCols = 16;
constexpr int kPhases = 64;
constexpr int kThreads = kCols * kPhases;
constexpr int kDepth = 4;  // rows of one thread whose loads are in flight together

struct Tile {
  int col;     // column of this thread (may be >= b: idle, but joins every barrier)
  int phase;   // row phase
  bool valid;  // col < b
};

__device__ __forceinline__ Tile tile(int32_t b) {
  Tile t;
  t.col = blockIdx.x * kCols + (int)(threadIdx.x % kCols);
  t.phase = (int)(threadIdx.x / kCols);
  t.valid = t.col < b;
  return t;
}

using Lds = double[kPhases][kCols];

// Combines the 64 phase values of each column, pairwise in a fixed tree,
// and returns the result to every thread of the column.  MAX: the maximum,
// a NaN winning; otherwise the sum.
template <bool MAX>
__device__ double combine(double v, Lds &lds) {
  const int c = threadIdx.x % kCols, p = threadIdx.x / kCols;
  __syncthreads();  // earlier readers of lds are done
  lds[p][c] = v;
  __syncthreads();
  for (int h = kPhases / 2; h >= 1; h >>= 1) {
    if (p < h) {
      const double a = lds[p][c], w = lds[p + h][c];
      lds[p][c] = MAX ? ((w > a || w != w) ? w : a) : a + w;
    }
    __syncthreads();
  }
  return lds[0][c];
}

// The thread's part of a column reduction: f(i) over its rows i (phase,
// phase + 64, ...), combined in row order.  The row index handed to f is
// clamped to n - 1 so that the kDepth loads of a round are unconditional;
// rows past the end then contribute the identity.
template <bool MAX, class F>
__device__ double column_part(int64_t n, const Tile &t, F f) {
  double acc = MAX ? -INFINITY : 0.0;
  if (!t.valid) return acc;
  for (int64_t i0 = t.phase; i0 < n; i0 += (int64_t)kPhases * kDepth) {
    double v[kDepth];
#pragma unroll
    for (int k = 0; k < kDepth; ++k) {
      const int64_t i = i0 + (int64_t)k * kPhases;
      v[k] = f(i < n ? i : n - 1);
    }
#pragma unroll
    for (int k = 0; k < kDepth; ++k) {
      if (i0 + (int64_t)k * kPhases >= n) break;
      acc = MAX ? ((v[k] > acc || v[k] != v[k]) ? v[k] : acc) : acc + v[k];
    }
  }
  return acc;
}

// Maximum and sum of exp(z - max) of each column of z.
__device__ void softmax_stats(int64_t n, int32_t b, const float *z, const Tile &t, Lds &lds,
                              double *m_out, double *s_out) {
  const int col = t.col;
  double m = column_part<true>(n, t, [&](int64_t i) { return (double)z[i * b + col]; });
  m = combine<true>(m, lds);
  double s = column_part<false>(n, t, [&](int64_t i) { return exp((double)z[i * b + col] - m); });
  s = combine<false>(s, lds);
  *m_out = m;
  *s_out = s;
}

__global__ __launch_bounds__(kThreads) void softmax_kernel(int64_t n, int32_t b,
                                                           const float *__restrict__ z,
                                                           float *__restrict__ p) {
  __shared__ Lds lds;
  const Tile t = tile(b);
  double m, s;
  softmax_stats(n, b, z, t, lds, &m, &s);
  if (!t.valid) return;  // no barrier below
#pragma unroll 4
  for (int64_t i = t.phase; i < n; i += kPhases)
    p[i * b + t.col] = (float)(exp((double)z[i * b + t.col] - m) / s);
}

__global__ __launch_bounds__(kThreads) void softmax_backward_kernel(int64_t n, int32_t b,
                                                                    const float *__restrict__ p,
                                                                    const float *__restrict__ dp,
                                                                    float *__restrict__ dz) {
  __shared__ Lds lds;
  const Tile t = tile(b);
  const int col = t.col;
  double g = column_part<false>(
      n, t, [&](int64_t i) { return (double)dp[i * b + col] * (double)p[i * b + col]; });
  g = combine<false>(g, lds);
  if (!t.valid) return;  // no barrier below
#pragma unroll 4
  for (int64_t i = t.phase; i < n; i += kPhases) {
    const int64_t k = i * b + col;
    dz[k] = (float)((double)p[k] * ((double)dp[k] - g));
  }
}

__global__ __launch_bounds__(kThreads) void l1_normalize_kernel(int64_t n, int32_t b,
                                                                const float *__restrict__ u,
                                                                float *__restrict__ x,
                                                                double *__restrict__ sums) {
  __shared__ Lds lds;
  const Tile t = tile(b);
  const int col = t.col;
  double s = column_part<false>(n, t, [&](int64_t i) { return (double)u[i * b + col]; });
  s = combine<false>(s, lds);
  if (!t.valid) return;  // no barrier below
  if (t.phase == 0) sums[col] = s;
#pragma unroll 4
  for (int64_t i = t.phase; i < n; i += kPhases)
    x[i * b + col] = (float)((double)u[i * b + col] / s);
}

__global__ __launch_bounds__(kThreads) void l1_normalize_backward_kernel(
    int64_t n, int32_t b, const float *__restrict__ x, const double *__restrict__ sums,
    const float *__restrict__ dx, float *__restrict__ du) {
  __shared__ Lds lds;
  const Tile t = tile(b);
  const int col = t.col;
  double g = column_part<false>(
      n, t, [&](int64_t i) { return (double)dx[i * b + col] * (double)x[i * b + col]; });
  g = combine<false>(g, lds);
  if (!t.valid) return;  // no barrier below
  const double s = sums[col];
#pragma unroll 4
  for (int64_t i = t.phase; i < n; i += kPhases) {
    const int64_t k = i * b + col;
    du[k] = (float)(((double)dx[k] - g) / s);
  }
}

__global__ __launch_bounds__(kThreads) void softmax_xent_kernel(int64_t n, int32_t b,
                                                                const float *__restrict__ z,
                                                                const float *__restrict__ tg,
                                                                double *__restrict__ col_loss,
                                                                float *__restrict__ dz) {
  __shared__ Lds lds;
  const Tile t = tile(b);
  const int col = t.col;
  double m, s;
  softmax_stats(n, b, z, t, lds, &m, &s);
  const double log_z = m + log(s);
  // Sum of the targets and of t * log p, per column.
  double tsum = column_part<false>(n, t, [&](int64_t i) { return (double)tg[i * b + col]; });
  double tlogp = column_part<false>(n, t, [&](int64_t i) {
    return (double)tg[i * b + col] * ((double)z[i * b + col] - log_z);
  });
  tsum = combine<false>(tsum, lds);
  tlogp = combine<false>(tlogp, lds);
  if (!t.valid) return;  // no barrier below
  if (t.phase == 0) col_loss[col] = -tlogp;
  const double inv_b = 1.0 / (double)b;
#pragma unroll 4
  for (int64_t i = t.phase; i < n; i += kPhases) {
    const int64_t k = i * b + col;
    const double pk = exp((double)z[k] - m) / s;
    dz[k] = (float)((pk * tsum - (double)tg[k]) * inv_b);
  }
}

// loss[0] = (col_loss[0] + ... + col_loss[b-1]) / b, added in order.  The
// workgroup stages 1024 values at a time in LDS (one load per thread, all in
// flight together) and thread 0 adds them in index order.
constexpr int kMeanThreads = 1024;

__global__ __launch_bounds__(kMeanThreads) void mean_kernel(int32_t b,
                                                            const double *__restrict__ col_loss,
                                                            double *__restrict__ loss) {
  __shared__ double stage[kMeanThreads];
  double s = 0.0;
  for (int32_t c0 = 0; c0 < b; c0 += kMeanThreads) {
    const int32_t c = c0 + (int32_t)threadIdx.x;
    __syncthreads();  // thread 0 is done with the previous batch
    stage[threadIdx.x] = c < b ? col_loss[c] : 0.0;
    __syncthreads();
    if (threadIdx.x == 0) {
      const int32_t m = b - c0 < kMeanThreads ? b - c0 : kMeanThreads;
      for (int32_t k = 0; k < m; ++k) s += stage[k];
    }
  }
  if (threadIdx.x == 0) loss[0] = s / (double)b;
}

dim3 grid_for(int32_t b) { return dim3((unsigned)((b + kCols - 1) / kCols)); }

kbc_status launched() { return hipGetLastError() == hipSuccess ? KBC_OK : KBC_EHIP; }

}  // namespace

extern "C" {

kbc_status kbc_softmax(int64_t n, int32_t b, const float *z, float *p, void *stream) {
  if (n < 1 || b < 1 || !z || !p) return KBC_EINVAL;
  hipLaunchKernelGGL(softmax_kernel, grid_for(b), dim3(kThreads), 0,
                     static_cast<hipStream_t>(stream), n, b, z, p);
  return launched();
}

kbc_status kbc_softmax_backward(int64_t n, int32_t b, const float *p, const float *dp, float *dz,
                                void *stream) {
  if (n < 1 || b < 1 || !p || !dp || !dz) return KBC_EINVAL;
  hipLaunchKernelGGL(softmax_backward_kernel, grid_for(b), dim3(kThreads), 0,
                     static_cast<hipStream_t>(stream), n, b, p, dp, dz);
  return launched();
}

kbc_status kbc_l1_normalize(int64_t n, int32_t b, const float *u, float *x, double *sums,
                            void *stream) {
  if (n < 1 || b < 1 || !u || !x || !sums) return KBC_EINVAL;
  hipLaunchKernelGGL(l1_normalize_kernel, grid_for(b), dim3(kThreads), 0,
                     static_cast<hipStream_t>(stream), n, b, u, x, sums);
  return launched();
}

kbc_status kbc_l1_normalize_backward(int64_t n, int32_t b, const float *x, const double *sums,
                                     const float *dx, float *du, void *stream) {
  if (n < 1 || b < 1 || !x || !sums || !dx || !du) return KBC_EINVAL;
  hipLaunchKernelGGL(l1_normalize_backward_kernel, grid_for(b), dim3(kThreads), 0,
                     static_cast<hipStream_t>(stream), n, b, x, sums, dx, du);
  return launched();
}

kbc_status kbc_softmax_xent(int64_t n, int32_t b, const float *z, const float *t,
                            double *col_loss, double *loss, float *dz, void *stream) {
  if (n < 1 || b < 1 || !z || !t || !col_loss || !loss || !dz) return KBC_EINVAL;
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipLaunchKernelGGL(softmax_xent_kernel, grid_for(b), dim3(kThreads), 0, s, n, b, z, t, col_loss,
                     dz);
  if (hipGetLastError() != hipSuccess) return KBC_EHIP;
  hipLaunchKernelGGL(mean_kernel, dim3(1), dim3(kMeanThreads), 0, s, b, col_loss, loss);
  return launched();
}

}  // extern "C"
