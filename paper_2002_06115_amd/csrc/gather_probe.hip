// gather_probe.hip -- measurement helper, not part of the follow operation.
//
// Times a pure gather of b-wide float rows in a given index order: the memory
// traffic of a follow pass's per-triple row reads with nothing else (no
// second operand, no products, no row boundaries, no output rows).  A pass's
// time against this probe's time on the same index stream tells how far the
// pass is from the memory system's own rate for that access pattern.
//
// A sequential read and a copy of a large buffer give the streaming rates
// beside it.
//
// Same lane layout as the follow kernels: a lane group of LPT lanes reads one
// row (lane l owns columns [4l, 4l + 4)) and walks one chunk of the index
// stream, U rows in flight per step; the group adds its rows in float and
// writes the sum once, so the loads cannot be dropped.
#include <hip/hip_runtime.h>

#include <cstdint>

namespace {

constexpr int kBlock = 256;
constexpr int kU = 16;

template <int LPT>
__global__ __launch_bounds__(kBlock) void gather_sum_kernel(const int32_t *__restrict__ idx,
                                                            int64_t n, int32_t chunk,
                                                            const float *__restrict__ X,
                                                            int32_t b, float *__restrict__ out) {
  constexpr int GPB = kBlock / LPT;
  const int lane = threadIdx.x % LPT;
  const int grp = threadIdx.x / LPT;
  const int64_t g = (int64_t)blockIdx.x * GPB + grp;
  const int64_t n_chunks = (n + chunk - 1) / chunk;
  const int c = lane * 4;
  if (g >= n_chunks || c >= b) return;  // no barrier below
  const int64_t p0 = g * chunk;
  const int64_t p1 = p0 + chunk < n ? p0 + chunk : n;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int64_t p = p0; p < p1; p += kU) {
    float4 v[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      // Past the chunk's end the last row is read again and not added.
      const int64_t q = p + u < p1 ? p + u : p1 - 1;
      v[u] = *reinterpret_cast<const float4 *>(X + (size_t)idx[q] * b + c);
    }
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      if (p + u < p1) {
        acc.x += v[u].x;
        acc.y += v[u].y;
        acc.z += v[u].z;
        acc.w += v[u].w;
      }
    }
  }
  *reinterpret_cast<float4 *>(out + g * b + c) = acc;
}

template <int LPT>
void launch(const int32_t *idx, int64_t n, int32_t chunk, const float *X, int32_t b, float *out,
            hipStream_t s) {
  const int64_t n_chunks = (n + chunk - 1) / chunk;
  const dim3 grid((unsigned)((n_chunks + kBlock / LPT - 1) / (kBlock / LPT)));
  hipLaunchKernelGGL(gather_sum_kernel<LPT>, grid, dim3(kBlock), 0, s, idx, n, chunk, X, b, out);
}

typedef float native_float4 __attribute__((ext_vector_type(4)));

// Sequential read of n float4s, grid-stride; one float per thread is written.
__global__ __launch_bounds__(kBlock) void stream_read_kernel(const native_float4 *__restrict__ X,
                                                             int64_t n, float *__restrict__ out) {
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  float acc = 0.f;
  for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < n; i += stride) {
    const native_float4 v = __builtin_nontemporal_load(X + i);
    acc += (v.x + v.y) + (v.z + v.w);
  }
  out[(int64_t)blockIdx.x * kBlock + threadIdx.x] = acc;
}

// Copy of n float4s, grid-stride, non-temporal stores.
__global__ __launch_bounds__(kBlock) void stream_copy_kernel(const native_float4 *__restrict__ X,
                                                             int64_t n,
                                                             native_float4 *__restrict__ Y) {
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < n; i += stride)
    __builtin_nontemporal_store(__builtin_nontemporal_load(X + i), Y + i);
}

// Fill of n float4s with zeros, grid-stride, non-temporal stores.
__global__ __launch_bounds__(kBlock) void stream_write_kernel(int64_t n,
                                                              native_float4 *__restrict__ Y) {
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  const native_float4 z = {0.f, 0.f, 0.f, 0.f};
  for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < n; i += stride)
    __builtin_nontemporal_store(z, Y + i);
}

// One untimed launch, then `reps` launches between two events on `s`;
// *ms = mean time of one.  0 on success, -2 on a HIP error.
template <class Run>
int time_launches(Run run, int reps, hipStream_t s, float *ms) {
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (hipEventCreate(&e0) != hipSuccess) return -2;
  if (hipEventCreate(&e1) != hipSuccess) {
    (void)hipEventDestroy(e0);
    return -2;
  }
  run();
  hipError_t err = hipEventRecord(e0, s);
  for (int r = 0; r < reps && err == hipSuccess; ++r) {
    run();
    err = hipGetLastError();
  }
  if (err == hipSuccess) err = hipEventRecord(e1, s);
  if (err == hipSuccess) err = hipEventSynchronize(e1);
  float t = 0.f;
  if (err == hipSuccess) err = hipEventElapsedTime(&t, e0, e1);
  (void)hipEventDestroy(e0);
  (void)hipEventDestroy(e1);
  if (err != hipSuccess) return -2;
  *ms = t / reps;
  return 0;
}

}  // namespace

extern "C" {

// Reads n_float4 float4s of DEVICE X once, front to back, `reps` timed
// launches after one untimed; *ms receives the mean time of one.  `out` is
// DEVICE float scratch of at least n_blocks * 256 floats; n_blocks >= 1.
// Returns 0, -1 for bad arguments, -2 for a HIP error.
int kbp_stream_read_time(const void *X, int64_t n_float4, int32_t n_blocks, float *out,
                         int32_t reps, void *stream, float *ms) {
  if (!X || !out || !ms || n_float4 < 1 || n_blocks < 1 || reps < 1) return -1;
  hipStream_t s = static_cast<hipStream_t>(stream);
  auto run = [&]() {
    hipLaunchKernelGGL(stream_read_kernel, dim3((unsigned)n_blocks), dim3(kBlock), 0, s,
                       static_cast<const native_float4 *>(X), n_float4, out);
  };
  return time_launches(run, reps, s, ms);
}

// Copies n_float4 float4s from DEVICE X to DEVICE Y (not overlapping), front
// to back, `reps` timed launches after one untimed; *ms receives the mean
// time of one.  n_blocks >= 1 workgroups of 256.  Returns 0, -1 for bad
// arguments, -2 for a HIP error.
int kbp_stream_copy_time(const void *X, void *Y, int64_t n_float4, int32_t n_blocks, int32_t reps,
                         void *stream, float *ms) {
  if (!X || !Y || !ms || n_float4 < 1 || n_blocks < 1 || reps < 1) return -1;
  hipStream_t s = static_cast<hipStream_t>(stream);
  auto run = [&]() {
    hipLaunchKernelGGL(stream_copy_kernel, dim3((unsigned)n_blocks), dim3(kBlock), 0, s,
                       static_cast<const native_float4 *>(X), n_float4,
                       static_cast<native_float4 *>(Y));
  };
  return time_launches(run, reps, s, ms);
}

// Writes zeros over n_float4 float4s of DEVICE Y, front to back, `reps`
// timed launches after one untimed; *ms receives the mean time of one.
// n_blocks >= 1 workgroups of 256.  Returns 0, -1 for bad arguments, -2 for
// a HIP error.
int kbp_stream_write_time(void *Y, int64_t n_float4, int32_t n_blocks, int32_t reps, void *stream,
                          float *ms) {
  if (!Y || !ms || n_float4 < 1 || n_blocks < 1 || reps < 1) return -1;
  hipStream_t s = static_cast<hipStream_t>(stream);
  auto run = [&]() {
    hipLaunchKernelGGL(stream_write_kernel, dim3((unsigned)n_blocks), dim3(kBlock), 0, s,
                       n_float4, static_cast<native_float4 *>(Y));
  };
  return time_launches(run, reps, s, ms);
}

// Gathers rows X[idx[p]] for p in [0, n) (DEVICE int32 idx, DEVICE float X
// [rows][b], b % 4 == 0, 4 <= b <= 256, every idx[p] a valid row) in chunks of
// `chunk` indices per lane group, and writes one b-wide float sum per chunk to
// DEVICE out [ceil(n / chunk)][b].  `reps` launches are timed with HIP events
// on `stream` after one untimed launch; *ms receives the mean time of one.
// Returns 0, or -1 for bad arguments, -2 for a HIP error.
int kbp_gather_time(const int32_t *idx, int64_t n, int32_t chunk, const float *X, int32_t b,
                    float *out, int32_t reps, void *stream, float *ms) {
  if (!idx || !X || !out || !ms || n < 1 || chunk < 1 || reps < 1 || b % 4 != 0 || b < 4 ||
      b > 256)
    return -1;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int lanes = b / 4;
  int lpt = 1;
  while (lpt < lanes) lpt <<= 1;
  auto run = [&]() {
    switch (lpt) {
      case 1: launch<1>(idx, n, chunk, X, b, out, s); break;
      case 2: launch<2>(idx, n, chunk, X, b, out, s); break;
      case 4: launch<4>(idx, n, chunk, X, b, out, s); break;
      case 8: launch<8>(idx, n, chunk, X, b, out, s); break;
      case 16: launch<16>(idx, n, chunk, X, b, out, s); break;
      case 32: launch<32>(idx, n, chunk, X, b, out, s); break;
      default: launch<64>(idx, n, chunk, X, b, out, s); break;
    }
  };
  return time_launches(run, reps, s, ms);
}

}  // extern "C"
