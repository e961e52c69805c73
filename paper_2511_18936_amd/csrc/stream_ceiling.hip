// Streaming-read ceiling: a kernel that does nothing but read a byte range
// with the loads the decode attention kernels use for their pages (16-byte
// nontemporal loads, 1 KiB contiguous per wave instruction, several in flight
// per wave, each wave a contiguous slice).  The time it takes for the same
// bytes is the bandwidth an HBM-streaming kernel can reach on this GPU, the
// reference beside the nominal 8 TB/s.  Measurement support only: not on the
// decode path.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "swan_bench.h"

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <int U>
__global__ __launch_bounds__(64) void stream_read_kernel(const char* __restrict__ src,
                                                         int64_t chunks, uint32_t* sink) {
  const int lane = threadIdx.x;
  const int64_t nw = gridDim.x, w = blockIdx.x;
  const int64_t c0 = chunks * w / nw, c1 = chunks * (w + 1) / nw;
  u32x4 acc = {0u, 0u, 0u, 0u};
  int64_t c = c0;
  for (; c + U <= c1; c += U) {
    u32x4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u)
      v[u] = __builtin_nontemporal_load((const u32x4*)(src + (c + u) * 1024 + lane * 16));
#pragma unroll
    for (int u = 0; u < U; ++u) acc ^= v[u];
  }
  for (; c < c1; ++c) acc ^= __builtin_nontemporal_load((const u32x4*)(src + c * 1024 + lane * 16));
  // one word per wave, so that the loads are kept
  uint32_t x = acc.x ^ acc.y ^ acc.z ^ acc.w;
  for (int o = 32; o > 0; o >>= 1) x ^= __shfl_xor(x, o);
  if (lane == 0) sink[w] = x;
}

}  // namespace

extern "C" int32_t swan_stream_read(const void* buf, size_t bytes, int32_t waves,
                                    int32_t loads_in_flight, uint32_t* sink, void* stream) {
  if (!buf || !sink || waves < 1 || waves > (1 << 20)) return 1;
  if (((uintptr_t)buf & 15) != 0) return 1;
  const int64_t chunks = (int64_t)(bytes / 1024);
  if (chunks == 0) return 0;
  const hipStream_t s = (hipStream_t)stream;
  const char* src = (const char*)buf;
  switch (loads_in_flight) {
    case 4:
      hipLaunchKernelGGL(stream_read_kernel<4>, dim3(waves), dim3(64), 0, s, src, chunks, sink);
      break;
    case 8:
      hipLaunchKernelGGL(stream_read_kernel<8>, dim3(waves), dim3(64), 0, s, src, chunks, sink);
      break;
    case 16:
      hipLaunchKernelGGL(stream_read_kernel<16>, dim3(waves), dim3(64), 0, s, src, chunks, sink);
      break;
    default:
      return 1;
  }
  return hipGetLastError() == hipSuccess ? 0 : 5;
}
