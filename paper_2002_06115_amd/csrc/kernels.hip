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
//     dR      : rows = relations, A = dY (a = object),   B = X  (b_id = subject)
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
#include "plan.h"

#include <hip/hip_ext.h>

#include <algorithm>
#include <climits>
#include <cstdio>
#include <map>
#include <string>
#include <tuple>
#include <mutex>
#include <utility>

// Structured-buffer loads (LLVM's amdgcn struct buffer load intrinsics): the
// bytes at `off` of record `idx` of a descriptor whose records are `stride`
// bytes apart.  A record index at or past the descriptor's record count
// returns zeros without a memory access, so a gathered row needs no multiply
// for its address and a marker's index (bit 31 set) needs no select.  (At
// file scope: an intrinsic declared by its assembler name needs external
// linkage.)
typedef float kbf_float4 __attribute__((ext_vector_type(4)));
__device__ kbf_float4 struct_buffer_load_f32x4(__amdgpu_buffer_rsrc_t rsrc, int idx, int off,
                                               int soff, int aux)
    __asm("llvm.amdgcn.struct.ptr.buffer.load.v4f32");
__device__ float struct_buffer_load_f32(__amdgpu_buffer_rsrc_t rsrc, int idx, int off, int soff,
                                        int aux) __asm("llvm.amdgcn.struct.ptr.buffer.load.f32");

namespace kbf {

namespace {

constexpr int kBlock = 256;   // threads per workgroup (4 wavefronts of 64)
constexpr int kMaxLpt = 32;   // widest lane group (column_tiling)
// Workgroups of the stream kernel when the B table sits in LDS: 12 waves,
// so that two workgroups (two copies of a table of up to kMaxLdsB bytes) fill
// a CU at the six waves per SIMD that the kernel's registers allow; 16 waves,
// one workgroup per CU, for a table of up to kMaxLdsBig bytes.  The LDS
// variants are compiled for the larger block and read blockDim at run time.
constexpr int kBlockLds = 768;
constexpr int kBlockLdsBig = 1024;
constexpr int kUnroll = 8;    // entries per step; a lane group keeps their loads in flight
// The residual hop's empty-row fill: pieces per lane group, rows per batch.
constexpr int kFillPieces = 4;
constexpr int kFillBatch = 4;
static_assert(kChunkQuantum % kUnroll == 0, "a chunk is a whole number of steps");
static_assert(kUnroll == kStepEntries, "the planner's kSameA flags assume this step length");

// Buffer-resource word 3 for gfx9-family buffers, and an offset past any raw
// buffer this library makes (such a load returns zeros without touching
// memory; tables are at most this many bytes).
constexpr int kRawBufferWord3 = 0x00020000;
constexpr uint32_t kOutOfRange = 0xFFFFFFF0u;
// Largest record stride of a buffer descriptor (a 14-bit field), in bytes.
constexpr uint64_t kMaxStride = 16383;

// Checked builds (KBFOLLOW_CHECKED) validate every row, slot and combine
// index before it is used: KBF_CHECKED(i, n) is i when 0 <= i < n, else 0 (a
// valid index) with one more count in a device-wide counter, so a planning
// bug shows up as a count instead of an out-of-bounds access.  In normal
// builds KBF_CHECKED(i, n) is just (i): the same code as without checks.
#ifdef KBFOLLOW_CHECKED
__device__ unsigned long long g_violations;
__device__ __forceinline__ int64_t checked(int64_t i, int64_t n) {
  if (i >= 0 && i < n) return i;
  atomicAdd(&g_violations, 1ull);
  return 0;
}
#define KBF_CHECKED(i, n) checked((i), (n))
#else
#define KBF_CHECKED(i, n) (i)
#endif

template <class F, int... I>
__device__ __forceinline__ void static_for_impl(F &f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
// f(std::integral_constant<int, i>) for i = 0 .. N-1, unrolled at compile time.
template <int N, class F>
__device__ __forceinline__ void static_for(F &&f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// Value of lane SRC of this lane's group of LPT lanes (LPT a power of two,
// at most 32): ds_swizzle's bitmask mode (no LDS memory is touched), source
// lane = (lane & and_mask) | SRC within each 32-lane half.
template <int LPT, int SRC>
__device__ __forceinline__ int group_bcast(int v) {
  static_assert(LPT >= 1 && LPT <= 32 && (LPT & (LPT - 1)) == 0, "lane groups of 1..32");
  if constexpr (LPT == 1) {
    return v;
  } else {
    constexpr int and_mask = 0x1f & ~(LPT - 1);
    return __builtin_amdgcn_ds_swizzle(v, and_mask | (SRC << 5));
  }
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

typedef float native_float4 __attribute__((ext_vector_type(4)));

// Record index that no table of this library reaches.
constexpr uint32_t kNoRecord = 0xFFFFFFFFu;

// VEC floats at byte `off` of record `idx` of a structured buffer (zeros when
// idx is past its last record).
template <int VEC>
__device__ __forceinline__ void gather_row(__amdgpu_buffer_rsrc_t rsrc, uint32_t idx,
                                           uint32_t off, float (&v)[VEC]) {
  if constexpr (VEC == 4) {
    const native_float4 t = struct_buffer_load_f32x4(rsrc, (int)idx, (int)off, 0, 0);
    v[0] = t[0];
    v[1] = t[1];
    v[2] = t[2];
    v[3] = t[3];
  } else {
    v[0] = struct_buffer_load_f32(rsrc, (int)idx, (int)off, 0, 0);
  }
}

// VEC floats at byte offset `off` of a raw buffer (zeros when off is past its end).
template <int VEC>
__device__ __forceinline__ void load_row_buffer(__amdgpu_buffer_rsrc_t rsrc, uint32_t off,
                                                float (&v)[VEC]) {
  if constexpr (VEC == 4) {
    const auto t = __builtin_amdgcn_raw_buffer_load_b128(rsrc, (int)off, 0, 0);
    v[0] = __int_as_float(t[0]);
    v[1] = __int_as_float(t[1]);
    v[2] = __int_as_float(t[2]);
    v[3] = __int_as_float(t[3]);
  } else {
    v[0] = __int_as_float(__builtin_amdgcn_raw_buffer_load_b32(rsrc, (int)off, 0, 0));
  }
}

// VEC floats of LDS at p (16-byte aligned when VEC = 4).
template <int VEC>
__device__ __forceinline__ void lds_row(const float *p, float (&v)[VEC]) {
  if constexpr (VEC == 4) {
    const native_float4 t = *reinterpret_cast<const native_float4 *>(p);
    v[0] = t[0];
    v[1] = t[1];
    v[2] = t[2];
    v[3] = t[3];
  } else {
    v[0] = *p;
  }
}
template <int VEC>
__device__ __forceinline__ void lds_store(float *p, const float (&v)[VEC]) {
  if constexpr (VEC == 4)
    *reinterpret_cast<native_float4 *>(p) = native_float4{v[0], v[1], v[2], v[3]};
  else
    *p = v[0];
}

// Output rows are written once and not read again by the pass: non-temporal
// stores keep them from displacing gathered rows in the caches.
template <int VEC>
__device__ __forceinline__ void store_row(float *__restrict__ p, const double (&acc)[VEC]) {
  if constexpr (VEC == 4) {
    const native_float4 v = {(float)acc[0], (float)acc[1], (float)acc[2], (float)acc[3]};
    __builtin_nontemporal_store(v, reinterpret_cast<native_float4 *>(p));
  } else {
    __builtin_nontemporal_store((float)acc[0], p);
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

template <int VEC>
__device__ __forceinline__ void store_slot_buffer(__amdgpu_buffer_rsrc_t rsrc, uint32_t off,
                                                  const double (&acc)[VEC]) {
  typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
  typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
  if constexpr (VEC == 4) {
    const double2 lo = make_double2(acc[0], acc[1]), hi = make_double2(acc[2], acc[3]);
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, lo), rsrc, (int)off, 0, 0);
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, hi), rsrc, (int)(off + 16), 0,
                                           0);
  } else {
    __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2, acc[0]), rsrc, (int)off, 0, 0);
  }
}

// Stores of VEC floats / doubles at byte offset `off` of a raw buffer; rows
// written once per pass use the non-temporal policy.
constexpr int kNonTemporal = 2;
template <int VEC>
__device__ __forceinline__ void store_row_buffer(__amdgpu_buffer_rsrc_t rsrc, uint32_t off,
                                                 const double (&y)[VEC]) {
  if constexpr (VEC == 4) {
    const native_float4 v = {(float)y[0], (float)y[1], (float)y[2], (float)y[3]};
    __builtin_amdgcn_raw_buffer_store_b128(
        __builtin_bit_cast(__attribute__((ext_vector_type(4))) unsigned int, v), rsrc, (int)off, 0,
        kNonTemporal);
  } else {
    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint((float)y[0]), rsrc, (int)off, 0,
                                          kNonTemporal);
  }
}

// One lane group (LPT lanes) per chunk of the entry stream; chunks are
// visited grid-stride so a capped (persistent) grid works too.  Every chunk
// holds the same number of entries, so the work is balanced whatever the row
// lengths.
//
// Inside a row the triples come in runs of equal B id.  The group reads the
// B row once, at the run's first triple, keeps it in registers for the run,
// and adds w * A[a] * B[b_id] for every triple with one double FMA per
// column (the product of two floats is exact in double).
//
// With BUF (A, B, the output and the workspace each under 4 GB, rows of at
// most kMaxStride bytes) all reads are buffer loads: A and B rows through
// structured buffers (record = row id), the residual variants' rows and the
// stores through raw 32-bit byte offsets.  Where no row is needed (A at
// markers and where the step's previous entry gathered the same row, B
// except at run starts) the record or offset is out of range, so the lane
// gets zeros and generates no memory traffic, and no load sits behind a
// branch.  A marker therefore finds A = 0 and a held B row of 0, so its FMA
// adds an exact zero; a repeated row takes the previous entry's values.
// Without BUF, plain loads read row 0 at markers and the values are masked
// instead.
//
// With LDSB (buffer loads only) the workgroup first copies its column
// slice of the whole B table into LDS, and a run start reads its B row from
// there when the FMAs need it.  No B row is then held in registers while a
// step's gathers are in flight, which leaves room for more waves per SIMD,
// and the B reads leave the L2 alone.  Used when the table fits (R for the
// forward and dX passes: at most kMaxLdsB bytes per slice with 768-thread
// workgroups, kMaxLdsBig with 1024; see launch_stream).
//
// The hard-KB variants with B in LDS (4 floats per lane; 8 lanes per group
// with the paired entry fetch, 8 or more for the residual hop) need 83 or 84
// VGPRs, more than six waves per SIMD allow; they are compiled for six waves
// (80 VGPRs, a few registers spilled around the chunk loop, outside the
// steps), which measured faster than losing the second workgroup per CU or
// keeping B in registers (residual forward on the large KB 0.89 -> 0.84 ms).
// The same cap on the soft-KB variants or on narrower lane groups spilled
// inside the loop and ran slower, so they keep the compiler's own
// allocation.
template <int VEC, int LPT, bool WEIGHTED, bool RES, bool LDSB>
constexpr int stream_min_waves() {
  return (LDSB && !WEIGHTED && VEC == 4 && (RES ? LPT >= 8 : LPT == 8)) ? 6 : 1;
}

template <int VEC, int LPT, bool BUF, bool WEIGHTED, bool RES, bool LDSB>
__global__ __launch_bounds__((LDSB ? kBlockLdsBig : kBlock),
                             (stream_min_waves<VEC, LPT, WEIGHTED, RES, LDSB>())) void
stream_kernel(StreamArgs a) {
  static_assert(BUF || !LDSB, "the LDS copy of B goes with raw buffer loads");
  const int BLK = LDSB ? (int)blockDim.x : kBlock;  // kBlockLds or kBlockLdsBig
  const int GPB = BLK / LPT;
  constexpr int W = LPT * VEC;  // columns of one slice
  extern __shared__ float b_lds[];  // [B_rows][W] with LDSB
  const int lane = threadIdx.x % LPT;
  const int grp = threadIdx.x / LPT;
  const int c = blockIdx.y * (LPT * VEC) + lane * VEC;
  const bool active = c < a.b;
  const size_t bb = (size_t)a.b;
  // Lanes past b read column 0 and store nothing.
  const int cl = active ? c : 0;
  const uint32_t row_bytes = (uint32_t)a.b * (uint32_t)sizeof(float);
  const uint32_t col_bytes = (uint32_t)cl * (uint32_t)sizeof(float);

  // (Only used with BUF, where every table is known to be under 4 GB.)
  auto rsrc = [](const void *p, uint64_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), 0, (int)(uint32_t)bytes,
                                             kRawBufferWord3);
  };
  // A and B are gathered by row: structured buffers of row_bytes records
  // (row_bytes is at most kMaxStride with BUF).  The residual variants keep
  // raw byte offsets, which measured faster there (their marker rows read
  // A too, so the record index needs a select either way, and the struct
  // addresses cost them registers).
  auto rows_rsrc = [&](const void *p, int64_t rows) {
    return RES ? rsrc(p, (uint64_t)rows * row_bytes)
               : __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), (short)row_bytes,
                                                   (int)rows, kRawBufferWord3);
  };
  const __amdgpu_buffer_rsrc_t arsrc = rows_rsrc(a.A, a.A_rows);
  const __amdgpu_buffer_rsrc_t brsrc = rows_rsrc(a.B, a.B_rows);
  const __amdgpu_buffer_rsrc_t orsrc = rsrc(a.out, (uint64_t)a.out_rows * row_bytes);
  const __amdgpu_buffer_rsrc_t srsrc =
      rsrc(a.slots, (uint64_t)a.n_slots * a.b * sizeof(double));

  // This workgroup's chunk list: the blocks with blockIdx.x % n_lists == x
  // (all on XCD x) share list x, grid-stride.
  const int nl = a.n_lists;
  const int xl = (int)(blockIdx.x % (unsigned)nl);
  int64_t c_begin = 0, c_end = 0;
#pragma unroll
  for (int i = 0; i < kMaxChunkLists; ++i)
    if (i == xl) {
      c_begin = a.list_chunk[i];
      c_end = a.list_chunk[i + 1];
    }
  const int64_t wg_in_list = blockIdx.x / nl;
  const int64_t wgs_in_list = ((int64_t)gridDim.x - xl + nl - 1) / nl;
  const int64_t stride = wgs_in_list * GPB;

  if constexpr (LDSB) {
    // Columns [col0, col0 + W) of every B row; columns past b read as zeros.
    const int col0 = blockIdx.y * W;
    const int64_t n_lds = a.B_rows * W;
    for (int64_t i = (int64_t)threadIdx.x * VEC; i < n_lds; i += (int64_t)BLK * VEC) {
      const int64_t r = i / W;
      const int j = (int)(i % W);
      float v[VEC];
      if (col0 + j < a.b) {
        load_row<VEC>(a.B + (size_t)KBF_CHECKED(r, a.B_rows) * bb + col0 + j, v);
      } else {
#pragma unroll
        for (int q = 0; q < VEC; ++q) v[q] = 0.0f;
      }
      lds_store<VEC>(b_lds + i, v);
    }
    __syncthreads();
  }

  // Each lane loads K of a step's kUnroll entries (lane + k * LPT) and the
  // group shares them by broadcast, so one load instruction fetches the
  // entries of every lane group in the wavefront.  (The prefetch after a
  // chunk's last step reads the next chunk's first entries, or the stream's
  // last entry at its end, and is not used.)
  constexpr int K = (kUnroll + LPT - 1) / LPT;
  auto fetch = [&](int64_t p, int2 (&mine)[K], float (&wmine)[K]) {
#pragma unroll
    for (int k = 0; k < K; ++k) {
      const int64_t q = min(p + min(lane + k * LPT, kUnroll - 1), a.n - 1);
      mine[k] = a.entries[q];
      if constexpr (WEIGHTED) wmine[k] = a.weights[q];
    }
  };
  // Two steps' entries, 2 per lane (entries p + 2l and p + 2l + 1 of lane
  // l < kUnroll; lanes past it repeat the last pair).  p and the stream
  // length are multiples of kUnroll, so every pair is 16-byte aligned and
  // the clamp keeps it inside the stream.
  // Only for groups of exactly eight lanes: not in the residual variants,
  // whose register-capped LDS form spilled more with it and ran 0.7 % slower,
  // nor with wider groups, whose LDS form would need the same cap and whose
  // short chunks (small KBs) would then spill every other step.
  constexpr bool kPairFetch = !WEIGHTED && !RES && K == 1 && LPT == kUnroll;
  auto fetch2 = [&](int64_t p, int4 &mine) {
    const int64_t q = min(p + 2 * min(lane, kUnroll - 1), a.n - 2);
    mine = reinterpret_cast<const int4 *>(a.entries)[q / 2];
  };

  for (int64_t g = c_begin + wg_in_list * GPB + grp; g < c_end; g += stride) {
    const int64_t p0 = KBF_CHECKED(g, a.n / a.chunk) * a.chunk;
    const int64_t p1 = p0 + a.chunk;
    double acc[VEC];
    float held_b[VEC];  // the current run's B row
#pragma unroll
    for (int v = 0; v < VEC; ++v) {
      acc[v] = 0.0;
      held_b[v] = 0.0f;
    }

    // Software pipeline: the entries of the next step are loaded while this
    // step's gathers are in flight.  With lane groups of eight lanes or more
    // (and no weights) one 16-byte load per lane fetches two steps' entries
    // (lane l entries 2l and 2l + 1 of the pair), so the steps run in pairs
    // and only the second of a pair issues a fetch: one entry load per two
    // steps in front of their sixteen row gathers.
    int2 mine_next[K];
    float wmine_next[K];
    int4 mine2 = make_int4(0, 0, 0, 0);
    if constexpr (kPairFetch)
      fetch2(p0, mine2);
    else
      fetch(p0, mine_next, wmine_next);
    // One step of kUnroll entries from p; H is its half of a pair (0 or 1)
    // or -1 for the one-step fetch.
    auto step = [&](const int64_t p, auto hc) {
      constexpr int H = decltype(hc)::value;
      int2 e[kUnroll];
      float w[kUnroll];
      float xa[kUnroll][VEC], xb[kUnroll][VEC];
      static_for<kUnroll>([&](auto uc) {
        constexpr int u = decltype(uc)::value;
        if constexpr (H >= 0) {
          constexpr int src = (kUnroll / 2) * H + u / 2;
          const int ex = (u % 2) ? mine2.z : mine2.x;
          const int ey = (u % 2) ? mine2.w : mine2.y;
          e[u] = make_int2(group_bcast<LPT, src>(ex), group_bcast<LPT, src>(ey));
        } else {
          const int2 m = mine_next[u / LPT];
          e[u] = make_int2(group_bcast<LPT, u % LPT>(m.x), group_bcast<LPT, u % LPT>(m.y));
          if constexpr (WEIGHTED)
            w[u] = __int_as_float(group_bcast<LPT, u % LPT>(__float_as_int(wmine_next[u / LPT])));
        }
      });
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const bool triple = e[u].x >= 0;
        const bool run_start = triple && (e[u].x & kRunStart);
        // The entry before it in this step gathered the same A row: no read
        // (the FMAs below take that row again).  Never at a step's first
        // entry; the residual variants read the row again (the reuse cost
        // their register-capped LDS form more spills than it saved).
        const bool same_a = !RES && u > 0 && triple && (e[u].y & kSameA);
        const int32_t bid = e[u].y & kIdMask;  // a triple's B row
        // A marker that writes row j of a residual pass reads A[j] for gamma * A[j].
        const bool res_row = RES && !triple && e[u].y >= 0;
        const uint32_t ia = triple ? (uint32_t)(e[u].x & kIdMask) : (uint32_t)e[u].y;
        if constexpr (BUF && !RES) {
          // A triple's record is its id; a marker's x (-1) with the run-start
          // bit cleared is past every table, so it reads zeros.
#if defined(KBFOLLOW_CHECKED)
          const uint32_t ra =
              (triple && !same_a) ? (uint32_t)KBF_CHECKED(ia, a.A_rows) : kNoRecord;
#else
          const uint32_t ra = same_a ? kNoRecord : ((uint32_t)e[u].x & ~(uint32_t)kRunStart);
#endif
          gather_row<VEC>(arsrc, ra, col_bytes, xa[u]);
          if constexpr (!LDSB)
            gather_row<VEC>(brsrc, run_start ? (uint32_t)KBF_CHECKED(bid, a.B_rows) : kNoRecord,
                            col_bytes, xb[u]);
        } else if constexpr (BUF) {
          load_row_buffer<VEC>(arsrc,
                               ((triple && !same_a) || res_row)
                                   ? (uint32_t)KBF_CHECKED(ia, a.A_rows) * row_bytes + col_bytes
                                   : kOutOfRange,
                               xa[u]);
          if constexpr (!LDSB)
            load_row_buffer<VEC>(brsrc,
                                 run_start ? (uint32_t)KBF_CHECKED(bid, a.B_rows) * row_bytes +
                                                 col_bytes
                                           : kOutOfRange,
                                 xb[u]);
        } else {
          // A residual row comes from Z (A itself for the residual hop).
          const float *src = res_row ? a.Z : a.A;
          load_row<VEC>(src + (size_t)(triple ? KBF_CHECKED(ia, a.A_rows)
                                              : res_row ? KBF_CHECKED(ia, a.out_rows) : 0) *
                                  bb +
                              cl,
                        xa[u]);
          load_row<VEC>(a.B + (size_t)(run_start ? KBF_CHECKED(bid, a.B_rows) : 0) * bb + cl,
                        xb[u]);
        }
      }
      if constexpr (H < 0)
        fetch(p + kUnroll, mine_next, wmine_next);
      else if constexpr (H == 1)
        fetch2(p + kUnroll, mine2);
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const bool triple = e[u].x >= 0;
        const bool run_start = triple && (e[u].x & kRunStart);
        // A repeated A row was not read again: take the previous entry's
        // (plain loads read it again, the same values).
        if constexpr (BUF && !RES) {
          if (u > 0) {
            const bool same_a = triple && (e[u].y & kSameA);
#pragma unroll
            for (int v = 0; v < VEC; ++v) xa[u][v] = same_a ? xa[u - 1][v] : xa[u][v];
          }
        }
        // Run starts take the new B row; markers take the zeros their
        // out-of-range B load returned (masked explicitly without BUF).
        if constexpr (LDSB) {
          if (run_start) {
            lds_row<VEC>(b_lds + (size_t)KBF_CHECKED(e[u].y & kIdMask, a.B_rows) * W + lane * VEC,
                         held_b);
          } else if (!triple) {
#pragma unroll
            for (int v = 0; v < VEC; ++v) held_b[v] = 0.0f;
          }
        }
#pragma unroll
        for (int v = 0; v < VEC; ++v) {
          if constexpr (!LDSB) {
            const float nb = (BUF || triple) ? xb[u][v] : 0.0f;
            held_b[v] = (run_start || !triple) ? nb : held_b[v];
          }
          double t = (double)xa[u][v];
          if constexpr (WEIGHTED) t *= (double)w[u];
          // Zero at markers (also the residual row's A and plain loads' row 0).
          if constexpr (RES || !BUF) t = triple ? t : 0.0;
          acc[v] = __builtin_fma(t, (double)held_b[v], acc[v]);
        }
        const int f = e[u].y;
        if (!triple) {
        if (active && f != INT_MIN) {
          double y[VEC];
#pragma unroll
          for (int v = 0; v < VEC; ++v)
            y[v] = (RES && f >= 0) ? acc[v] + (double)a.gamma * (double)xa[u][v] : acc[v];
          if (f >= 0) {
            if constexpr (BUF)
              store_row_buffer<VEC>(
                  orsrc, (uint32_t)KBF_CHECKED(f, a.out_rows) * row_bytes + col_bytes, y);
            else
              store_row<VEC>(a.out + (size_t)KBF_CHECKED(f, a.out_rows) * bb + c, y);
          } else {
            if constexpr (BUF)
              store_slot_buffer<VEC>(
                  srsrc,
                  ((uint32_t)KBF_CHECKED(-(f + 1), a.n_slots) * (uint32_t)a.b + (uint32_t)c) *
                      (uint32_t)sizeof(double),
                  y);
            else
              store_slot<VEC>(a.slots + (size_t)KBF_CHECKED(-(f + 1), a.n_slots) * bb + c, y);
          }
        }
        // The marker ends the row: restart the sum (only the lanes of
        // groups at a marker execute this).
#pragma unroll
        for (int v = 0; v < VEC; ++v) acc[v] = 0.0;
        }
      }
    };
    if constexpr (kPairFetch) {
      // Chunks are whole steps; an odd last step runs alone.
      for (int64_t p = p0; p < p1; p += 2 * kUnroll) {
        step(p, std::integral_constant<int, 0>{});
        if (p + kUnroll >= p1) break;
        step(p + kUnroll, std::integral_constant<int, 1>{});
      }
    } else {
      for (int64_t p = p0; p < p1; p += kUnroll) step(p, std::integral_constant<int, -1>{});
    }
  }
}

// Adds slots [first, first + n) in increasing order; writes the float row or
// a next-level slot.  `block` of `n_blocks` blocks share the tasks.
template <int VEC, int LPT>
__device__ __forceinline__ void combine_tasks(const int4 *__restrict__ tasks, int64_t n_tasks,
                                              double *__restrict__ slots, int64_t n_slots,
                                              int32_t b, float *out, int64_t out_rows,
                                              const float *res, float gamma, int64_t block,
                                              int64_t n_blocks) {
  constexpr int W = LPT * VEC;
  constexpr int GPB = kBlock / LPT;
  const int lane = threadIdx.x % LPT;
  const int grp = threadIdx.x / LPT;
  const int c = blockIdx.y * W + lane * VEC;
  if (c >= b) return;  // no barrier below
  const size_t bb = (size_t)b;
  const int64_t stride = n_blocks * GPB;
  for (int64_t t = block * GPB + grp; t < n_tasks; t += stride) {
    const int4 tk = tasks[t];  // first, n, dst
    double acc[VEC];
#pragma unroll
    for (int v = 0; v < VEC; ++v) acc[v] = 0.0;
    for (int i = 0; i < tk.y; i += kUnroll) {
      const int n = min(kUnroll, tk.y - i);
      double part[kUnroll][VEC];
#pragma unroll
      for (int u = 0; u < kUnroll; ++u)
        load_slot<VEC>(slots + (size_t)KBF_CHECKED(tk.x + i + min(u, n - 1), n_slots) * bb + c,
                       part[u]);
#pragma unroll
      for (int u = 0; u < kUnroll; ++u)
        if (u < n) {
#pragma unroll
          for (int v = 0; v < VEC; ++v) acc[v] += part[u][v];
        }
    }
    if (tk.z >= 0) {
      const size_t row = (size_t)KBF_CHECKED(tk.z, out_rows);
      if (res) {
        float r[VEC];
        load_row<VEC>(res + row * bb + c, r);
#pragma unroll
        for (int v = 0; v < VEC; ++v) acc[v] += (double)gamma * (double)r[v];
      }
      store_row<VEC>(out + row * bb + c, acc);
    } else {
      store_slot<VEC>(slots + (size_t)KBF_CHECKED(-(int64_t)tk.z - 1, n_slots) * bb + c, acc);
    }
  }
}

// Writes the rows no triple reaches, given as pieces of consecutive rows
// (first, count); lanes over the columns as in the stream kernel.  PACKED: a
// lane group writes LPT consecutive pieces, whose descriptors its lanes fetch
// with one load (lane j the j-th) and share by shuffles, so that one load
// stands in front of the stores of 64 pieces per wave.  Otherwise one piece
// per group: the residual hop's rows each need a load of X of their own.
// `block` of `n_blocks` blocks share the pieces.
template <int VEC, int LPT, bool PACKED>
__device__ __forceinline__ void zero_pieces(const int2 *__restrict__ pieces, int64_t n_pieces,
                                            int32_t b, float *out, int64_t out_rows,
                                            const float *res, float gamma, int64_t block,
                                            int64_t n_blocks) {
  constexpr int W = LPT * VEC;
  constexpr int GPB = kBlock / LPT;
  const int lane = threadIdx.x % LPT;
  const int grp = threadIdx.x / LPT;
  const int c = blockIdx.y * W + lane * VEC;
  const size_t bb = (size_t)b;
  if constexpr (PACKED) {
    const int64_t stride = n_blocks * kBlock;
    for (int64_t t0 = (block * GPB + grp) * LPT; t0 < n_pieces; t0 += stride) {
      const int64_t t = t0 + lane;
      int2 mine = make_int2(0, 0);  // past the end: a piece of no rows
      if (t < n_pieces) mine = pieces[t];
      const int base = (int)(threadIdx.x % 64) - lane;  // lane 0 of this group in the wave
      for (int j = 0; j < LPT; ++j) {
        const int first = __shfl(mine.x, base + j);
        const int count = __shfl(mine.y, base + j);
        if (c >= b) continue;  // after the shuffles, which every lane joins
        for (int i = 0; i < count; ++i) {
          const double z[VEC] = {};
          // Non-temporal, like every output row: plain stores would leave
          // the rows dirty in the caches, to be written back during the next
          // pass.
          store_row<VEC>(out + (size_t)KBF_CHECKED((int64_t)first + i, out_rows) * bb + c, z);
        }
      }
    }
  } else {
    // gamma * res[row] into out[row].  A lane group takes kFillPieces
    // consecutive pieces (every lane loads the same descriptors) and walks
    // their rows as one flat sequence, kFillBatch rows at a time: all of a
    // batch's row loads are issued before its stores, so the mostly one- or
    // two-row pieces of a Zipf KB still keep many loads in flight.  (res may
    // be out itself: each row is read and then written by the same lane.)
    if (c >= b) return;  // no barrier or shuffle below
    const int64_t stride = n_blocks * GPB * kFillPieces;
    for (int64_t t0 = (block * GPB + grp) * kFillPieces; t0 < n_pieces; t0 += stride) {
      int first[kFillPieces], start[kFillPieces], end[kFillPieces];
      int total = 0;
#pragma unroll
      for (int j = 0; j < kFillPieces; ++j) {
        const int2 pc = (t0 + j < n_pieces) ? pieces[t0 + j] : make_int2(0, 0);
        first[j] = pc.x;
        start[j] = total;
        total += pc.y;
        end[j] = total;
      }
      for (int k0 = 0; k0 < total; k0 += kFillBatch) {
        int row[kFillBatch];
        float r[kFillBatch][VEC];
#pragma unroll
        for (int u = 0; u < kFillBatch; ++u) {
          const int k = k0 + u;
          row[u] = -1;
#pragma unroll
          for (int j = 0; j < kFillPieces; ++j)
            row[u] = (k >= start[j] && k < end[j]) ? first[j] + (k - start[j]) : row[u];
#pragma unroll
          for (int v = 0; v < VEC; ++v) r[u][v] = 0.0f;
          if (row[u] >= 0)
            load_row<VEC>(res + (size_t)KBF_CHECKED((int64_t)row[u], out_rows) * bb + c, r[u]);
        }
#pragma unroll
        for (int u = 0; u < kFillBatch; ++u) {
          if (row[u] < 0) continue;
          double y[VEC];
#pragma unroll
          for (int v = 0; v < VEC; ++v) y[v] = 0.0 + (double)gamma * (double)r[u][v];
          store_row<VEC>(out + (size_t)KBF_CHECKED((int64_t)row[u], out_rows) * bb + c, y);
        }
      }
    }
  }
}

// A later combine level.
template <int VEC, int LPT>
__global__ __launch_bounds__(kBlock) void combine_kernel(const int4 *__restrict__ tasks,
                                                         int64_t n_tasks,
                                                         double *__restrict__ slots,
                                                         int64_t n_slots, int32_t b,
                                                         float *out, int64_t out_rows,
                                                         const float *res, float gamma) {
  combine_tasks<VEC, LPT>(tasks, n_tasks, slots, n_slots, b, out, out_rows, res, gamma,
                          blockIdx.x, gridDim.x);
}

// The first combine level and the empty rows in one launch: blocks
// [0, combine_blocks) take the combine tasks, the others the empty-row
// pieces.  The two write disjoint rows; the combine's dependent slot reads
// overlap with the fill's stores instead of forming a launch of their own.
template <int VEC, int LPT, bool PACKED>
__global__ __launch_bounds__(kBlock) void tail_kernel(TailArgs a) {
  if ((int64_t)blockIdx.x < a.combine_blocks)
    combine_tasks<VEC, LPT>(a.tasks, a.n_tasks, a.slots, a.n_slots, a.b, a.out, a.out_rows,
                            a.res, a.gamma, blockIdx.x, a.combine_blocks);
  else
    zero_pieces<VEC, LPT, PACKED>(a.pieces, a.n_pieces, a.b, a.out, a.out_rows, a.res, a.gamma,
                                  (int64_t)blockIdx.x - a.combine_blocks,
                                  (int64_t)gridDim.x - a.combine_blocks);
}

template <int VEC, bool BUF, bool WT, bool RES, bool LDSB>
const void *stream_fn(int lpt) {
  switch (lpt) {
    case 1: return reinterpret_cast<const void *>(&stream_kernel<VEC, 1, BUF, WT, RES, LDSB>);
    case 2: return reinterpret_cast<const void *>(&stream_kernel<VEC, 2, BUF, WT, RES, LDSB>);
    case 4: return reinterpret_cast<const void *>(&stream_kernel<VEC, 4, BUF, WT, RES, LDSB>);
    case 8: return reinterpret_cast<const void *>(&stream_kernel<VEC, 8, BUF, WT, RES, LDSB>);
    case 16: return reinterpret_cast<const void *>(&stream_kernel<VEC, 16, BUF, WT, RES, LDSB>);
    case 32: return reinterpret_cast<const void *>(&stream_kernel<VEC, 32, BUF, WT, RES, LDSB>);
  }
  return nullptr;
}

template <int VEC, bool BUF, bool LDSB>
const void *stream_fn_sel(int lpt, bool wt, bool res) {
  if (wt)
    return res ? stream_fn<VEC, BUF, true, true, LDSB>(lpt)
               : stream_fn<VEC, BUF, true, false, LDSB>(lpt);
  return res ? stream_fn<VEC, BUF, false, true, LDSB>(lpt)
             : stream_fn<VEC, BUF, false, false, LDSB>(lpt);
}

// Plain loads never take the LDS copy of B.
const void *stream_fn_for(const ColumnTiling &t, bool buf, bool lds, bool wt, bool res) {
  if (t.vec == 4) {
    if (!buf) return stream_fn_sel<4, false, false>(t.lpt, wt, res);
    return lds ? stream_fn_sel<4, true, true>(t.lpt, wt, res)
               : stream_fn_sel<4, true, false>(t.lpt, wt, res);
  }
  if (!buf) return stream_fn_sel<1, false, false>(t.lpt, wt, res);
  return lds ? stream_fn_sel<1, true, true>(t.lpt, wt, res)
             : stream_fn_sel<1, true, false>(t.lpt, wt, res);
}

// Workgroups of `fn` (`block` threads, lds_bytes of dynamic LDS) that fit
// one CU at once, from the runtime's occupancy calculator; cached per kernel,
// block and LDS size.  0 when the query fails.
int blocks_per_cu(const void *fn, int block, size_t lds_bytes) {
  static std::mutex mu;
  static std::map<std::tuple<const void *, int, size_t>, int> cache;
  std::lock_guard<std::mutex> lock(mu);
  const auto key = std::make_tuple(fn, block, lds_bytes);
  auto it = cache.find(key);
  if (it != cache.end()) return it->second;
  int n = 0;
  if ((lds_bytes > 0 && hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize,
                                            (int)kMaxLdsBig) != hipSuccess) ||
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, fn, block, lds_bytes) != hipSuccess) {
    (void)hipGetLastError();
    n = 0;
  }
  cache[key] = n;
  return n;
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
  }
  return nullptr;
}

template <int VEC, bool PACKED>
const void *tail_fn(int lpt) {
  switch (lpt) {
    case 1: return reinterpret_cast<const void *>(&tail_kernel<VEC, 1, PACKED>);
    case 2: return reinterpret_cast<const void *>(&tail_kernel<VEC, 2, PACKED>);
    case 4: return reinterpret_cast<const void *>(&tail_kernel<VEC, 4, PACKED>);
    case 8: return reinterpret_cast<const void *>(&tail_kernel<VEC, 8, PACKED>);
    case 16: return reinterpret_cast<const void *>(&tail_kernel<VEC, 16, PACKED>);
    case 32: return reinterpret_cast<const void *>(&tail_kernel<VEC, 32, PACKED>);
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

ColumnTiling column_tiling(int32_t b) { return column_tiling_max(b, kMaxLpt); }

ColumnTiling column_tiling_max(int32_t b, int max_lpt) {
  ColumnTiling t;
  t.vec = (b % 4 == 0) ? 4 : 1;
  const int lanes = (b + t.vec - 1) / t.vec;
  // Lane groups of at most kMaxLpt lanes: wider rows are cut into column
  // slices of 128 columns (4 floats per lane), each a pass of its own over the
  // entries.  A slice's rows are still whole cache lines, and the table a
  // slice gathers from is half the size, so more of it stays in the
  // Infinity Cache: at b = 256 on a 2 M-entity KB, 64-lane groups took
  // 4.02 / 4.03 ms for the dX / dR passes, two 32-lane slices 3.71 / 3.82.
  int lpt = 1;
  while (lpt < lanes && lpt < max_lpt) lpt <<= 1;
  t.lpt = lpt;
  t.width = lpt * t.vec;
  t.n_slices = (b + t.width - 1) / t.width;
  return t;
}

namespace {

// The stream-kernel instance, grid and LDS size launch_stream uses for `a`.
struct StreamChoice {
  const void *fn = nullptr;
  dim3 grid;
  int block = 0;
  size_t lds_bytes = 0;
  int vec = 0, lpt = 0;
  bool buf = false, wt = false, res = false, ldsb = false;
};

hipError_t choose_stream(const StreamArgs &a, const StreamOptions &o, StreamChoice *c) {
  const ColumnTiling t = column_tiling(a.b);
  if (a.chunk % kChunkQuantum != 0 || a.n % a.chunk != 0) return hipErrorInvalidValue;
  // Raw-buffer offsets are 32-bit and a structured buffer's record stride is
  // at most kMaxStride bytes: tables of 4 GB or more, or rows of more than
  // 4095 floats, take plain loads.
  const uint64_t row_bytes = (uint64_t)a.b * sizeof(float);
  const uint64_t lim = kOutOfRange;
  const bool buf = !o.plain_loads && (!a.residual || a.Z == a.A) && row_bytes <= kMaxStride &&
                   (uint64_t)a.A_rows * row_bytes <= lim &&
                   (uint64_t)a.B_rows * row_bytes <= lim && (uint64_t)a.out_rows * row_bytes <= lim &&
                   (uint64_t)a.n_slots * (uint64_t)a.b * sizeof(double) <= lim;
  const bool wt = a.weights != nullptr, res = a.residual != 0;
  if (a.n_lists < 1 || a.n_lists > kMaxChunkLists || a.list_chunk[0] != 0 ||
      a.list_chunk[a.n_lists] != a.n / a.chunk)
    return hipErrorInvalidValue;
  // Every list gets the same number of workgroups (blockIdx.x % n_lists
  // picks the list), enough for its longest list.
  int64_t longest = 0;
  for (int x = 0; x < a.n_lists; ++x) {
    if (a.list_chunk[x + 1] < a.list_chunk[x]) return hipErrorInvalidValue;
    longest = std::max<int64_t>(longest, a.list_chunk[x + 1] - a.list_chunk[x]);
  }
  const int nl = a.n_lists;
  // The register variant's lane groups: at most o.max_lpt lanes wide.
  const ColumnTiling tr = column_tiling_max(a.b, std::max(1, std::min(o.max_lpt, kMaxLpt)));
  const void *reg_fn = stream_fn_for(tr, buf, false, wt, res);
  if (!reg_fn) return hipErrorInvalidValue;
  c->buf = buf;
  c->wt = wt;
  c->res = res;
  c->vec = t.vec;
  // B's column slice in LDS when it fits and the LDS variant keeps at least
  // as many waves on a CU as the register variant: where it needs more
  // registers per lane than its workgroup can be given (b = 4 .. 16, the
  // soft KB), or where the register variant runs at eight waves per SIMD
  // already (b = 1), B stays in registers.  A slice of at most kMaxLdsB bytes
  // goes with two 768-thread workgroups per CU; for the hard KB a slice of up
  // to kMaxLdsBig bytes goes with one 1024-thread workgroup, and rows wider
  // than 32 columns whose slice is too large are cut into 32-column slices
  // (one 128-byte line of every row each) when that makes B fit.  The grid
  // is as many workgroups as the CUs hold at once, each copying its slice of
  // the table once and walking its chunks grid-stride.
  if (buf && o.b_in_lds) {
    const bool hard = !wt && !res;
    ColumnTiling tl = t;
    size_t lds_bytes = (size_t)a.B_rows * (size_t)tl.width * sizeof(float);
    if (hard && lds_bytes > kMaxLdsB && t.vec == 4 && t.width > 32) {
      tl = column_tiling_max(a.b, 8);
      lds_bytes = (size_t)a.B_rows * (size_t)tl.width * sizeof(float);
    }
    const int blk = lds_bytes <= kMaxLdsB ? kBlockLds : kBlockLdsBig;
    if (lds_bytes <= (hard ? kMaxLdsBig : kMaxLdsB)) {
      const void *fn = stream_fn_for(tl, true, true, wt, res);
      if (!fn) return hipErrorInvalidValue;
      const int per_cu = blocks_per_cu(fn, blk, lds_bytes);
      const int reg_per_cu = blocks_per_cu(reg_fn, kBlock, 0);
      if (per_cu > 0 && per_cu * blk >= reg_per_cu * kBlock) {
        const int64_t cap = (int64_t)per_cu * (o.n_cu > 0 ? o.n_cu : 1);
        const int64_t per_list = std::max<int64_t>(1, std::min<int64_t>(
            (longest + blk / tl.lpt - 1) / (blk / tl.lpt), cap / nl));
        if (per_list * nl > (int64_t)INT32_MAX) return hipErrorInvalidValue;
        c->fn = fn;
        c->grid = dim3((unsigned)(per_list * nl), (unsigned)tl.n_slices);
        c->block = blk;
        c->lds_bytes = lds_bytes;
        c->lpt = tl.lpt;
        c->ldsb = true;
        return hipSuccess;
      }
    }
  }
  const int64_t per_list = std::max<int64_t>(1, (longest + kBlock / tr.lpt - 1) / (kBlock / tr.lpt));
  if (per_list * nl > (int64_t)INT32_MAX) return hipErrorInvalidValue;
  c->fn = reg_fn;
  c->grid = dim3((unsigned)(per_list * nl), (unsigned)tr.n_slices);
  c->block = kBlock;
  c->lds_bytes = 0;
  c->lpt = tr.lpt;
  c->ldsb = false;
  return hipSuccess;
}

const char *tf(bool v) { return v ? "true" : "false"; }

}  // namespace

hipError_t launch_stream(const StreamArgs &a, const StreamOptions &o, hipStream_t s,
                         hipEvent_t start, hipEvent_t stop) {
  if (a.n == 0) return hipSuccess;
  StreamChoice c;
  hipError_t e = choose_stream(a, o, &c);
  if (e != hipSuccess) return e;
  StreamArgs arg = a;
  void *params[] = {&arg};
  if (start || stop)
    return hipExtLaunchKernel(c.fn, c.grid, dim3(c.block), params, c.lds_bytes, s, start, stop, 0);
  return hipLaunchKernel(c.fn, c.grid, dim3(c.block), params, c.lds_bytes, s);
}

std::string describe_stream(const StreamArgs &a, const StreamOptions &o) {
  if (a.n == 0) return "";
  StreamChoice c;
  if (choose_stream(a, o, &c) != hipSuccess) return "";
  char buf[160];
  std::snprintf(buf, sizeof buf, "stream_kernel<%d, %d, %s, %s, %s, %s>", c.vec, c.lpt,
                tf(c.buf), tf(c.wt), tf(c.res), tf(c.ldsb));
  return buf;
}

std::string describe_tail(const TailArgs &a) {
  if (a.n_tasks == 0 && a.n_pieces == 0) return "";
  const ColumnTiling t = column_tiling(a.b);
  char buf[96];
  std::snprintf(buf, sizeof buf, "tail_kernel<%d, %d, %s>", t.vec, t.lpt, tf(a.res == nullptr));
  return buf;
}

std::string describe_combine(int32_t b) {
  const ColumnTiling t = column_tiling(b);
  char buf[96];
  std::snprintf(buf, sizeof buf, "combine_kernel<%d, %d>", t.vec, t.lpt);
  return buf;
}

hipError_t launch_combine(const int4 *tasks, int64_t n_tasks, double *slots, int64_t n_slots,
                          int32_t b, float *out, int64_t out_rows, const float *res, float gamma,
                          hipStream_t s) {
  if (n_tasks == 0) return hipSuccess;
  const ColumnTiling t = column_tiling(b);
  const void *fn = t.vec == 4 ? combine_fn<4>(t.lpt) : combine_fn<1>(t.lpt);
  if (!fn) return hipErrorInvalidValue;
  const dim3 grid((unsigned)blocks_for(n_tasks, kBlock / t.lpt, 0), (unsigned)t.n_slices);
  void *params[] = {&tasks, &n_tasks, &slots, &n_slots, &b, &out, &out_rows, &res, &gamma};
  return hipLaunchKernel(fn, grid, dim3(kBlock), params, 0, s);
}

hipError_t launch_tail(const TailArgs &args, hipStream_t s) {
  if (args.n_tasks == 0 && args.n_pieces == 0) return hipSuccess;
  const ColumnTiling t = column_tiling(args.b);
  const bool packed = args.res == nullptr;
  const void *fn = t.vec == 4 ? (packed ? tail_fn<4, true>(t.lpt) : tail_fn<4, false>(t.lpt))
                              : (packed ? tail_fn<1, true>(t.lpt) : tail_fn<1, false>(t.lpt));
  if (!fn) return hipErrorInvalidValue;
  TailArgs a = args;
  // One combine task per lane group.  Empty rows, packed: LPT pieces per
  // lane group, 256 per block; residual: kFillPieces pieces per lane group.
  a.combine_blocks = a.n_tasks > 0 ? blocks_for(a.n_tasks, kBlock / t.lpt, 0) : 0;
  const int64_t zero_blocks =
      a.n_pieces > 0
          ? blocks_for(a.n_pieces, packed ? kBlock : (kBlock / t.lpt) * kFillPieces, 0)
          : 0;
  if (a.combine_blocks + zero_blocks > (int64_t)INT32_MAX) return hipErrorInvalidValue;
  const dim3 grid((unsigned)(a.combine_blocks + zero_blocks), (unsigned)t.n_slices);
  void *params[] = {&a};
  return hipLaunchKernel(fn, grid, dim3(kBlock), params, 0, s);
}

hipError_t checked_violations(unsigned long long *count, bool reset) {
#ifdef KBFOLLOW_CHECKED
  hipError_t e = hipMemcpyFromSymbol(count, HIP_SYMBOL(g_violations), sizeof *count);
  if (e != hipSuccess || !reset) return e;
  const unsigned long long zero = 0;
  return hipMemcpyToSymbol(HIP_SYMBOL(g_violations), &zero, sizeof zero);
#else
  (void)count;
  (void)reset;
  return hipErrorNotSupported;
#endif
}

}  // namespace kbf
