// chain_glue.hip -- column-wise operations between the hops of a multi-hop
// chain (Sec. 3.2): softmax over relations, L1 normalisation of entity
// weights, softmax cross-entropy of the last hop, and their backwards.
//
// Every operation reduces over the n rows of each column of an [n][b]
// batch-contiguous array.  A workgroup owns 64 consecutive columns; its 256
// threads are 4 row phases of 64 lanes, lane c on column c of the tile, so
// each wavefront reads 64 consecutive floats of a row (coalesced).  Phase p
// visits rows p, p + 4, p + 8, ...; the four phase partials are combined
// through LDS in phase order.  Sums and maxima are taken in double, in that
// fixed order, so results are bitwise reproducible.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "kbchain.h"

namespace {

constexpr int kCols = 64;
constexpr int kPhases = 4;
constexpr int kThreads = kCols * kPhases;

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

// Combines the four phase values of each column: the sum (or maximum) over
// phases 0..3 in order, returned to every thread of the column.
template <bool MAX>
__device__ double combine(double v, double (&lds)[kPhases][kCols]) {
  const int c = threadIdx.x % kCols, p = threadIdx.x / kCols;
  __syncthreads();  // earlier readers of lds are done
  lds[p][c] = v;
  __syncthreads();
  double r = lds[0][c];
  for (int q = 1; q < kPhases; ++q) {
    const double w = lds[q][c];
    r = MAX ? (w > r ? w : r) : r + w;
  }
  return r;
}

// Maximum and sum of exp(z - max) of each column of z.
__device__ void softmax_stats(int64_t n, int32_t b, const float *z, const Tile &t,
                              double (&lds)[kPhases][kCols], double *m_out, double *s_out) {
  double m = -INFINITY;
  if (t.valid)
    for (int64_t i = t.phase; i < n; i += kPhases) {
      const double v = (double)z[i * b + t.col];
      m = (v > m || v != v) ? v : m;  // a NaN wins and propagates
    }
  m = combine<true>(m, lds);
  double s = 0.0;
  if (t.valid)
    for (int64_t i = t.phase; i < n; i += kPhases) s += exp((double)z[i * b + t.col] - m);
  s = combine<false>(s, lds);
  *m_out = m;
  *s_out = s;
}

__global__ __launch_bounds__(kThreads) void softmax_kernel(int64_t n, int32_t b,
                                                           const float *__restrict__ z,
                                                           float *__restrict__ p) {
  __shared__ double lds[kPhases][kCols];
  const Tile t = tile(b);
  double m, s;
  softmax_stats(n, b, z, t, lds, &m, &s);
  if (!t.valid) return;  // no barrier below
  for (int64_t i = t.phase; i < n; i += kPhases)
    p[i * b + t.col] = (float)(exp((double)z[i * b + t.col] - m) / s);
}

__global__ __launch_bounds__(kThreads) void softmax_backward_kernel(int64_t n, int32_t b,
                                                                    const float *__restrict__ p,
                                                                    const float *__restrict__ dp,
                                                                    float *__restrict__ dz) {
  __shared__ double lds[kPhases][kCols];
  const Tile t = tile(b);
  double g = 0.0;
  if (t.valid)
    for (int64_t i = t.phase; i < n; i += kPhases)
      g += (double)dp[i * b + t.col] * (double)p[i * b + t.col];
  g = combine<false>(g, lds);
  if (!t.valid) return;  // no barrier below
  for (int64_t i = t.phase; i < n; i += kPhases) {
    const int64_t k = i * b + t.col;
    dz[k] = (float)((double)p[k] * ((double)dp[k] - g));
  }
}

__global__ __launch_bounds__(kThreads) void l1_normalize_kernel(int64_t n, int32_t b,
                                                                const float *__restrict__ u,
                                                                float *__restrict__ x,
                                                                double *__restrict__ sums) {
  __shared__ double lds[kPhases][kCols];
  const Tile t = tile(b);
  double s = 0.0;
  if (t.valid)
    for (int64_t i = t.phase; i < n; i += kPhases) s += (double)u[i * b + t.col];
  s = combine<false>(s, lds);
  if (!t.valid) return;  // no barrier below
  if (t.phase == 0) sums[t.col] = s;
  for (int64_t i = t.phase; i < n; i += kPhases)
    x[i * b + t.col] = (float)((double)u[i * b + t.col] / s);
}

__global__ __launch_bounds__(kThreads) void l1_normalize_backward_kernel(
    int64_t n, int32_t b, const float *__restrict__ x, const double *__restrict__ sums,
    const float *__restrict__ dx, float *__restrict__ du) {
  __shared__ double lds[kPhases][kCols];
  const Tile t = tile(b);
  double g = 0.0;
  if (t.valid)
    for (int64_t i = t.phase; i < n; i += kPhases)
      g += (double)dx[i * b + t.col] * (double)x[i * b + t.col];
  g = combine<false>(g, lds);
  if (!t.valid) return;  // no barrier below
  const double s = sums[t.col];
  for (int64_t i = t.phase; i < n; i += kPhases) {
    const int64_t k = i * b + t.col;
    du[k] = (float)(((double)dx[k] - g) / s);
  }
}

__global__ __launch_bounds__(kThreads) void softmax_xent_kernel(int64_t n, int32_t b,
                                                                const float *__restrict__ z,
                                                                const float *__restrict__ tg,
                                                                double *__restrict__ col_loss,
                                                                float *__restrict__ dz) {
  __shared__ double lds[kPhases][kCols];
  const Tile t = tile(b);
  double m, s;
  softmax_stats(n, b, z, t, lds, &m, &s);
  const double log_z = m + log(s);
  // Sum of the targets and of t * log p, per column.
  double tsum = 0.0, tlogp = 0.0;
  if (t.valid)
    for (int64_t i = t.phase; i < n; i += kPhases) {
      const double tv = (double)tg[i * b + t.col];
      tsum += tv;
      tlogp += tv * ((double)z[i * b + t.col] - log_z);
    }
  tsum = combine<false>(tsum, lds);
  tlogp = combine<false>(tlogp, lds);
  if (!t.valid) return;  // no barrier below
  if (t.phase == 0) col_loss[t.col] = -tlogp;
  const double inv_b = 1.0 / (double)b;
  for (int64_t i = t.phase; i < n; i += kPhases) {
    const int64_t k = i * b + t.col;
    const double pk = exp((double)z[k] - m) / s;
    dz[k] = (float)((pk * tsum - (double)tg[k]) * inv_b);
  }
}

// loss[0] = (col_loss[0] + ... + col_loss[b-1]) / b, added in order by one thread.
__global__ void mean_kernel(int32_t b, const double *__restrict__ col_loss,
                            double *__restrict__ loss) {
  if (blockIdx.x != 0 || threadIdx.x != 0) return;
  double s = 0.0;
  for (int32_t c = 0; c < b; ++c) s += col_loss[c];
  loss[0] = s / (double)b;
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
  hipLaunchKernelGGL(mean_kernel, dim3(1), dim3(64), 0, s, b, col_loss, loss);
  return launched();
}

}  // extern "C"
