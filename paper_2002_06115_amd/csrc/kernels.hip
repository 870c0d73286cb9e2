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
// [col0 + l*VEC, col0 + l*VEC + VEC).  A lane group owns a whole piece (at
// most a few hundred triples of one row), so a row sum needs no cross-lane
// reduction at all: every lane accumulates its own columns.  Rows longer than
// a piece write double partials to workspace slots that the combine kernel
// adds up in piece order.  No atomics anywhere: every output element is
// written by exactly one lane, with a fixed summation order, so results are
// bitwise reproducible.
//
// Arithmetic: each product w * a * b is formed in double (the product of two
// floats is exact in double) and accumulated in double; the float output is
// one rounding of that sum.  The work is bound by memory traffic (two gathered
// rows per triple against two flops per element), so the double arithmetic
// costs no time while it keeps long Zipf-hub rows accurate.
#include "kernels.h"

namespace kbf {

namespace {

constexpr int kBlock = 256;   // threads per workgroup (4 wavefronts of 64)
constexpr int kUnroll = 8;    // triples whose loads a lane group keeps in flight

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
    *reinterpret_cast<float4 *>(p) =
        make_float4((float)acc[0], (float)acc[1], (float)acc[2], (float)acc[3]);
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

// One lane group (LPT lanes) per piece; pieces are visited grid-stride so a
// capped (persistent) grid works too.  With B_IN_LDS the workgroup first
// copies B's column slice [B_rows][W] into LDS (the relation table R is tiny:
// N_R x b floats) and every triple then reads its B row from LDS.
template <int VEC, int LPT, bool B_IN_LDS>
__global__ __launch_bounds__(kBlock) void pieces_kernel(PiecesArgs a) {
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

  const int64_t stride = (int64_t)gridDim.x * GPB;
  for (int64_t t = (int64_t)blockIdx.x * GPB + grp; t < a.n_pieces; t += stride) {
    const int4 pc = a.pieces[t];  // start, len, dst
    double acc[VEC];
#pragma unroll
    for (int v = 0; v < VEC; ++v) acc[v] = 0.0;

    for (int i = 0; i < pc.y; i += kUnroll) {
      const int n = min(kUnroll, pc.y - i);
      int2 id[kUnroll];
      float w[kUnroll];
      float xa[kUnroll][VEC], xb[kUnroll][VEC];
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        if (u < n) {
          id[u] = a.pairs[pc.x + i + u];
          w[u] = a.weight ? a.weight[pc.x + i + u] : 1.0f;
        }
      }
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        if (u < n && active) {
          load_row<VEC>(a.A + (size_t)id[u].x * bb + c, xa[u]);
          if constexpr (B_IN_LDS)
            load_row<VEC>(lds_b + (size_t)id[u].y * W + lane * VEC, xb[u]);
          else
            load_row<VEC>(a.B + (size_t)id[u].y * bb + c, xb[u]);
        } else {
#pragma unroll
          for (int v = 0; v < VEC; ++v) xa[u][v] = xb[u][v] = 0.0f;
        }
      }
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        if (u < n) {
#pragma unroll
          for (int v = 0; v < VEC; ++v)
            acc[v] += (double)w[u] * (double)xa[u][v] * (double)xb[u][v];
        }
      }
    }
    if (active) {
      if (pc.z >= 0)
        store_row<VEC>(a.out + (size_t)pc.z * bb + c, acc);
      else
        store_slot<VEC>(a.slots + (size_t)(-(pc.z + 1)) * bb + c, acc);
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
        if (u < n) load_slot<VEC>(slots + (size_t)(tk.x + i + u) * bb + c, part[u]);
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

template <int VEC, bool LDS>
const void *pieces_fn(int lpt) {
  switch (lpt) {
    case 1: return reinterpret_cast<const void *>(&pieces_kernel<VEC, 1, LDS>);
    case 2: return reinterpret_cast<const void *>(&pieces_kernel<VEC, 2, LDS>);
    case 4: return reinterpret_cast<const void *>(&pieces_kernel<VEC, 4, LDS>);
    case 8: return reinterpret_cast<const void *>(&pieces_kernel<VEC, 8, LDS>);
    case 16: return reinterpret_cast<const void *>(&pieces_kernel<VEC, 16, LDS>);
    case 32: return reinterpret_cast<const void *>(&pieces_kernel<VEC, 32, LDS>);
    case 64: return reinterpret_cast<const void *>(&pieces_kernel<VEC, 64, LDS>);
  }
  return nullptr;
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

size_t pieces_lds_bytes(int32_t b, int64_t B_rows) {
  const ColumnTiling t = column_tiling(b);
  return (size_t)B_rows * (size_t)t.width * sizeof(float);
}

hipError_t prepare_pieces_lds(int32_t b, size_t bytes) {
  const ColumnTiling t = column_tiling(b);
  const void *fn = t.vec == 4 ? pieces_fn<4, true>(t.lpt) : pieces_fn<1, true>(t.lpt);
  if (!fn) return hipErrorInvalidValue;
  return hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
}

hipError_t launch_pieces(const PiecesArgs &a, bool b_in_lds, int max_blocks, hipStream_t s) {
  if (a.n_pieces == 0) return hipSuccess;
  const ColumnTiling t = column_tiling(a.b);
  const void *fn = t.vec == 4 ? (b_in_lds ? pieces_fn<4, true>(t.lpt) : pieces_fn<4, false>(t.lpt))
                              : (b_in_lds ? pieces_fn<1, true>(t.lpt) : pieces_fn<1, false>(t.lpt));
  if (!fn) return hipErrorInvalidValue;
  const dim3 grid((unsigned)blocks_for(a.n_pieces, kBlock / t.lpt, max_blocks),
                  (unsigned)t.n_slices);
  const size_t lds = b_in_lds ? pieces_lds_bytes(a.b, a.B_rows) : 0;
  PiecesArgs arg = a;
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
