// Streaming-read reference: reads a buffer once with 16-byte nontemporal
// loads, four in flight per thread, and keeps nothing.  bench.py times it over
// buffers the size of each HBM-bound decode launch (rotating through more
// memory than the last-level cache holds) for the rate a plain stream of that
// size reaches on this GPU, the ceiling its kernels are compared against.
#include "ks_internal.h"

#include <algorithm>

namespace ks {

typedef uint32_t u32x4c __attribute__((ext_vector_type(4)));

// Workgroup b reads the contiguous range [b per, (b + 1) per) of 16-byte
// chunks, its threads four chunks apart in flight, the last workgroup also the
// remainder.
template <int NT>
__global__ __launch_bounds__(NT) void k_stream_read(const u32x4c* __restrict__ src, size_t n16,
                                                    size_t per, float* sink) {
  constexpr int D = 4;
  const size_t b0 = (size_t)blockIdx.x * per;
  const size_t b1 = blockIdx.x + 1 == gridDim.x ? n16 : b0 + per;
  uint32_t acc = 0;
  size_t i = b0 + threadIdx.x;
  for (; i + (D - 1) * NT < b1; i += D * NT) {
    u32x4c v[D];
#pragma unroll
    for (int u = 0; u < D; ++u) v[u] = __builtin_nontemporal_load(src + i + u * NT);
#pragma unroll
    for (int u = 0; u < D; ++u) acc ^= v[u].x;
  }
  for (; i < b1; i += NT) acc ^= __builtin_nontemporal_load(src + i).x;
  // keeps the loads: the sink is written only for one value of the running xor,
  // and never read for results
  if (acc == 0x9e3779b9u) sink[0] = 1.0f;
}

}  // namespace ks

using namespace ks;

extern "C" ks_status ks_stream_read(const void* src, size_t bytes, float* sink, void* stream) {
  if (!src || !sink || bytes < 16 || bytes % 16 != 0 || ((uintptr_t)src & 15) != 0) {
    set_error("ks_stream_read: null pointer, or bytes / src not a multiple of 16");
    return KS_EINVAL;
  }
  const size_t n16 = bytes / 16;
  // the shapes that streamed best in a sweep of workgroup counts and sizes:
  // 2048 workgroups of 256 threads up to 128 MiB, 256 of 1024 above
  hipStream_t st = (hipStream_t)stream;
  if (bytes <= ((size_t)128 << 20)) {
    const size_t nwg = std::max<size_t>(1, std::min<size_t>(2048, n16 / 256));
    KS_LAUNCH(k_stream_read<256>, dim3((unsigned)nwg), dim3(256), 0, st,
              (const u32x4c*)src, n16, n16 / nwg, sink);
  } else {
    KS_LAUNCH(k_stream_read<1024>, dim3(256), dim3(1024), 0, st, (const u32x4c*)src,
              n16, n16 / 256, sink);
  }
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) {
    set_error(std::string("ks_stream_read: ") + hipGetErrorString(e));
    return KS_EHIP;
  }
  return KS_OK;
}
