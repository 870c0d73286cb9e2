// kernels.hip -- gfx950 kernels for relation-set following on a reified KB.
//
// All three passes (forward Y, backward dX, backward dR; Eq. 4 and its
// gradients) are the same operation on a differently sorted triple list: a
// segmented sum, over the triples of a row, of the elementwise product of two
// gathered b-wide rows,
//
//     out[row] = sum over triples p of the row of  w[p] * A[a[p]] (.) B[b_id[p]]
//
//     forward : rows = objects,   A = X  (a = subject),  B = R  (b_id = relation)
//     dX      : rows = subjects,  A = dY (a = object),   B = R  (b_id = relation)
//     dR      : rows = relations, A = X  (a = subject),  B = dY (b_id = object)
//
// Activations are entity-major and batch-contiguous ([N][b] float32), so each
// gather is one contiguous b-wide row: a lane group of LPT lanes reads it with
// VEC-float (16-byte when VEC = 4) loads, lane l owning columns
// [col0 + l*VEC, col0 + l*VEC + VEC).  The sorted triple list is cut into
// equal chunks and a lane group walks one chunk sequentially, so a row sum
// needs no cross-lane reduction at all: every lane accumulates its own
// columns and writes them when the row ends.  A row that crosses a chunk
// boundary writes one double partial per chunk to a workspace slot and the
// combine kernel adds them up in chunk order.  No atomics anywhere: every
// output element is written by exactly one lane, with a fixed summation
// order, so results are bitwise reproducible.
//
// Arithmetic: each product w * a * b is formed in double (the product of two
// floats is exact in double) and accumulated in double; the float output is
// one rounding of that sum.  The work is bound by memory traffic (two gathered
// rows per triple against two flops per element), so the double arithmetic
// costs no time while it keeps long Zipf-hub rows accurate.
#include "kernels.h"

#include <climits>

namespace kbf {

namespace {

#ifndef KBF_UNROLL
#define KBF_UNROLL 8
#endif
#ifndef KBF_NT_ENTRIES
#define KBF_NT_ENTRIES 0
#endif
#ifndef KBF_NT_STORES
#define KBF_NT_STORES 0
#endif

constexpr int kBlock = 256;         // threads per workgroup (4 wavefronts of 64)
constexpr int kUnroll = KBF_UNROLL; // triples whose loads a lane group keeps in flight

// The triple stream is read once per pass: non-temporal loads keep it from
// evicting the gathered activation rows that Zipf-hot ids reuse from cache.
typedef int native_int4 __attribute__((ext_vector_type(4)));
typedef float native_float4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ int4 load_entry(const int4 *p) {
#if KBF_NT_ENTRIES
  const native_int4 v = __builtin_nontemporal_load(reinterpret_cast<const native_int4 *>(p));
  return make_int4(v.x, v.y, v.z, v.w);
#else
  return *p;
#endif
}

template <int VEC>
__device__ __forceinline__ void load_row(const float *__restrict__ p, float (&v)[VEC]) {
  if constexpr (VEC == 4) {
    const float4 t = *reinterpret_cast<const float4 *>(p);
    v[0] = t.x;
    v[1] = t.y;
    v[2] = t.z;
    v[3] = t.w;
  } else {
    v[0] = *p;
  }
}

template <int VEC>
__device__ __forceinline__ void store_row(float *__restrict__ p, const double (&acc)[VEC]) {
  if constexpr (VEC == 4) {
#if KBF_NT_STORES
    native_float4 v = {(float)acc[0], (float)acc[1], (float)acc[2], (float)acc[3]};
    __builtin_nontemporal_store(v, reinterpret_cast<native_float4 *>(p));
#else
    *reinterpret_cast<float4 *>(p) =
        make_float4((float)acc[0], (float)acc[1], (float)acc[2], (float)acc[3]);
#endif
  } else {
    *p = (float)acc[0];
  }
}

template <int VEC>
__device__ __forceinline__ void load_slot(const double *__restrict__ p, double (&v)[VEC]) {
  if constexpr (VEC == 4) {
    const double2 t0 = reinterpret_cast<const double2 *>(p)[0];
    const double2 t1 = reinterpret_cast<const double2 *>(p)[1];
    v[0] = t0.x;
    v[1] = t0.y;
    v[2] = t1.x;
    v[3] = t1.y;
  } else {
    v[0] = *p;
  }
}

template <int VEC>
__device__ __forceinline__ void store_slot(double *__restrict__ p, const double (&acc)[VEC]) {
  if constexpr (VEC == 4) {
    reinterpret_cast<double2 *>(p)[0] = make_double2(acc[0], acc[1]);
    reinterpret_cast<double2 *>(p)[1] = make_double2(acc[2], acc[3]);
  } else {
    *p = acc[0];
  }
}

// One lane group (LPT lanes) per chunk of the sorted triple stream; chunks
// are visited grid-stride so a capped (persistent) grid works too.  Every
// chunk holds the same number of positions, so the work is balanced whatever
// the row lengths.  With B_IN_LDS the workgroup first copies B's column slice
// [B_rows][W] into LDS (the relation table R is tiny: N_R x b floats).
template <int VEC, int LPT, bool B_IN_LDS, bool WEIGHTED>
__global__ __launch_bounds__(kBlock) void stream_kernel(StreamArgs a) {
  constexpr int W = LPT * VEC;
  constexpr int GPB = kBlock / LPT;
  extern __shared__ float lds_b[];
  const int lane = threadIdx.x % LPT;
  const int grp = threadIdx.x / LPT;
  const int col0 = blockIdx.y * W;
  const int c = col0 + lane * VEC;
  const bool active = c < a.b;
  const size_t bb = (size_t)a.b;

  if constexpr (B_IN_LDS) {
    const int64_t total = a.B_rows * W;
    for (int64_t e = threadIdx.x; e < total; e += kBlock) {
      const int64_t k = e / W;
      const int cc = col0 + (int)(e - k * W);
      lds_b[e] = cc < a.b ? a.B[k * bb + cc] : 0.0f;
    }
    __syncthreads();
  }

  // Loads never sit behind a branch, so all kUnroll gathers of a step are in
  // flight together: lanes past b read column 0 and store nothing, and the
  // step past the end of a chunk re-reads its last position and adds nothing.
  const int cl = active ? c : 0;
  const int64_t n_chunks = (a.n + a.chunk - 1) / a.chunk;
  const int64_t stride = (int64_t)gridDim.x * GPB;
  for (int64_t g = (int64_t)blockIdx.x * GPB + grp; g < n_chunks; g += stride) {
    const int64_t p0 = g * a.chunk;
    const int64_t p1 = min(p0 + (int64_t)a.chunk, a.n);
    double acc[VEC];
#pragma unroll
    for (int v = 0; v < VEC; ++v) acc[v] = 0.0;

    // Software pipeline: the entries of the next step are loaded while this
    // step's gathers are in flight.
    int4 e_next[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) e_next[u] = load_entry(a.entries + min(p0 + u, p1 - 1));
    for (int64_t p = p0; p < p1; p += kUnroll) {
      const int cnt = (int)min((int64_t)kUnroll, p1 - p);
      int4 e[kUnroll];
      float xa[kUnroll][VEC], xb[kUnroll][VEC];
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) e[u] = e_next[u];
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        load_row<VEC>(a.A + (size_t)e[u].x * bb + cl, xa[u]);
        if constexpr (B_IN_LDS)
          load_row<VEC>(lds_b + (size_t)e[u].y * W + lane * VEC, xb[u]);
        else
          load_row<VEC>(a.B + (size_t)e[u].y * bb + cl, xb[u]);
      }
#pragma unroll
      for (int u = 0; u < kUnroll; ++u)
        e_next[u] = load_entry(a.entries + min(p + kUnroll + u, p1 - 1));
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        if (u < cnt) {
          if constexpr (WEIGHTED) {
            const double w = (double)__int_as_float(e[u].w);
#pragma unroll
            for (int v = 0; v < VEC; ++v) acc[v] += w * (double)xa[u][v] * (double)xb[u][v];
          } else {
#pragma unroll
            for (int v = 0; v < VEC; ++v) acc[v] += (double)xa[u][v] * (double)xb[u][v];
          }
          const int f = e[u].z;
          if (f != INT_MIN) {
            if (active) {
              if (f >= 0)
                store_row<VEC>(a.out + (size_t)f * bb + c, acc);
              else
                store_slot<VEC>(a.slots + (size_t)(-(f + 1)) * bb + c, acc);
            }
#pragma unroll
            for (int v = 0; v < VEC; ++v) acc[v] = 0.0;
          }
        }
      }
    }
  }
}

// Adds slots [first, first + n) in increasing order; writes the float row or
// a next-level slot.
template <int VEC, int LPT>
__global__ __launch_bounds__(kBlock) void combine_kernel(const int4 *__restrict__ tasks,
                                                         int64_t n_tasks,
                                                         double *__restrict__ slots, int32_t b,
                                                         float *__restrict__ out) {
  constexpr int W = LPT * VEC;
  constexpr int GPB = kBlock / LPT;
  const int lane = threadIdx.x % LPT;
  const int grp = threadIdx.x / LPT;
  const int c = blockIdx.y * W + lane * VEC;
  if (c >= b) return;  // no barrier below
  const size_t bb = (size_t)b;
  const int64_t stride = (int64_t)gridDim.x * GPB;
  for (int64_t t = (int64_t)blockIdx.x * GPB + grp; t < n_tasks; t += stride) {
    const int4 tk = tasks[t];  // first, n, dst
    double acc[VEC];
#pragma unroll
    for (int v = 0; v < VEC; ++v) acc[v] = 0.0;
    for (int i = 0; i < tk.y; i += kUnroll) {
      const int n = min(kUnroll, tk.y - i);
      double part[kUnroll][VEC];
#pragma unroll
      for (int u = 0; u < kUnroll; ++u)
        load_slot<VEC>(slots + (size_t)(tk.x + i + min(u, n - 1)) * bb + c, part[u]);
#pragma unroll
      for (int u = 0; u < kUnroll; ++u)
        if (u < n) {
#pragma unroll
          for (int v = 0; v < VEC; ++v) acc[v] += part[u][v];
        }
    }
    if (tk.z >= 0)
      store_row<VEC>(out + (size_t)tk.z * bb + c, acc);
    else
      store_slot<VEC>(slots + (size_t)(-(tk.z + 1)) * bb + c, acc);
  }
}

template <int VEC>
__global__ __launch_bounds__(kBlock) void zero_rows_kernel(const int32_t *__restrict__ rows,
                                                           int64_t n_rows, int32_t b,
                                                           float *__restrict__ out) {
  const int per_row = b / VEC;
  const int64_t total = n_rows * per_row;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total; e += stride) {
    const int64_t q = e / per_row;
    const int j = (int)(e - q * per_row);
    float *p = out + (size_t)rows[q] * (size_t)b + (size_t)j * VEC;
    if constexpr (VEC == 4)
      *reinterpret_cast<float4 *>(p) = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    else
      *p = 0.0f;
  }
}

template <int VEC, bool LDS, bool WT>
const void *stream_fn(int lpt) {
  switch (lpt) {
    case 1: return reinterpret_cast<const void *>(&stream_kernel<VEC, 1, LDS, WT>);
    case 2: return reinterpret_cast<const void *>(&stream_kernel<VEC, 2, LDS, WT>);
    case 4: return reinterpret_cast<const void *>(&stream_kernel<VEC, 4, LDS, WT>);
    case 8: return reinterpret_cast<const void *>(&stream_kernel<VEC, 8, LDS, WT>);
    case 16: return reinterpret_cast<const void *>(&stream_kernel<VEC, 16, LDS, WT>);
    case 32: return reinterpret_cast<const void *>(&stream_kernel<VEC, 32, LDS, WT>);
    case 64: return reinterpret_cast<const void *>(&stream_kernel<VEC, 64, LDS, WT>);
  }
  return nullptr;
}

const void *stream_fn_for(const ColumnTiling &t, bool lds, bool wt) {
  if (t.vec == 4) {
    if (lds) return wt ? stream_fn<4, true, true>(t.lpt) : stream_fn<4, true, false>(t.lpt);
    return wt ? stream_fn<4, false, true>(t.lpt) : stream_fn<4, false, false>(t.lpt);
  }
  if (lds) return wt ? stream_fn<1, true, true>(t.lpt) : stream_fn<1, true, false>(t.lpt);
  return wt ? stream_fn<1, false, true>(t.lpt) : stream_fn<1, false, false>(t.lpt);
}

template <int VEC>
const void *combine_fn(int lpt) {
  switch (lpt) {
    case 1: return reinterpret_cast<const void *>(&combine_kernel<VEC, 1>);
    case 2: return reinterpret_cast<const void *>(&combine_kernel<VEC, 2>);
    case 4: return reinterpret_cast<const void *>(&combine_kernel<VEC, 4>);
    case 8: return reinterpret_cast<const void *>(&combine_kernel<VEC, 8>);
    case 16: return reinterpret_cast<const void *>(&combine_kernel<VEC, 16>);
    case 32: return reinterpret_cast<const void *>(&combine_kernel<VEC, 32>);
    case 64: return reinterpret_cast<const void *>(&combine_kernel<VEC, 64>);
  }
  return nullptr;
}

int64_t blocks_for(int64_t items, int per_block, int max_blocks) {
  int64_t g = (items + per_block - 1) / per_block;
  if (max_blocks > 0 && g > max_blocks) g = max_blocks;
  if (g > (int64_t)INT32_MAX) g = INT32_MAX;
  return g < 1 ? 1 : g;
}

}  // namespace

ColumnTiling column_tiling(int32_t b) {
  ColumnTiling t;
  t.vec = (b % 4 == 0) ? 4 : 1;
  const int lanes = (b + t.vec - 1) / t.vec;
  int lpt = 1;
  while (lpt < lanes && lpt < 64) lpt <<= 1;
  t.lpt = lpt;
  t.width = lpt * t.vec;
  t.n_slices = (b + t.width - 1) / t.width;
  return t;
}

size_t stream_lds_bytes(int32_t b, int64_t B_rows) {
  const ColumnTiling t = column_tiling(b);
  return (size_t)B_rows * (size_t)t.width * sizeof(float);
}

hipError_t prepare_stream_lds(int32_t b, size_t bytes) {
  const ColumnTiling t = column_tiling(b);
  for (bool wt : {false, true}) {
    const void *fn = stream_fn_for(t, true, wt);
    if (!fn) return hipErrorInvalidValue;
    hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_stream(const StreamArgs &a, bool weighted, bool b_in_lds, int max_blocks,
                         hipStream_t s) {
  if (a.n == 0) return hipSuccess;
  const ColumnTiling t = column_tiling(a.b);
  const void *fn = stream_fn_for(t, b_in_lds, weighted);
  if (!fn) return hipErrorInvalidValue;
  const int64_t n_chunks = (a.n + a.chunk - 1) / a.chunk;
  const dim3 grid((unsigned)blocks_for(n_chunks, kBlock / t.lpt, max_blocks),
                  (unsigned)t.n_slices);
  const size_t lds = b_in_lds ? stream_lds_bytes(a.b, a.B_rows) : 0;
  StreamArgs arg = a;
  void *params[] = {&arg};
  return hipLaunchKernel(fn, grid, dim3(kBlock), params, lds, s);
}

hipError_t launch_combine(const int4 *tasks, int64_t n_tasks, double *slots, int32_t b,
                          float *out, hipStream_t s) {
  if (n_tasks == 0) return hipSuccess;
  const ColumnTiling t = column_tiling(b);
  const void *fn = t.vec == 4 ? combine_fn<4>(t.lpt) : combine_fn<1>(t.lpt);
  if (!fn) return hipErrorInvalidValue;
  const dim3 grid((unsigned)blocks_for(n_tasks, kBlock / t.lpt, 0), (unsigned)t.n_slices);
  void *params[] = {&tasks, &n_tasks, &slots, &b, &out};
  return hipLaunchKernel(fn, grid, dim3(kBlock), params, 0, s);
}

hipError_t launch_zero_rows(const int32_t *rows, int64_t n_rows, int32_t b, float *out,
                            hipStream_t s) {
  if (n_rows == 0) return hipSuccess;
  const int vec = (b % 4 == 0) ? 4 : 1;
  const int64_t items = n_rows * (b / vec);
  const dim3 grid((unsigned)blocks_for(items, kBlock, 256 * 64));
  if (vec == 4)
    hipLaunchKernelGGL(zero_rows_kernel<4>, grid, dim3(kBlock), 0, s, rows, n_rows, b, out);
  else
    hipLaunchKernelGGL(zero_rows_kernel<1>, grid, dim3(kBlock), 0, s, rows, n_rows, b, out);
  return hipGetLastError();
}

}  // namespace kbf
