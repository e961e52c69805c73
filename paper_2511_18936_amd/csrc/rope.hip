// Rotary position embedding (RoPE) of the Llama models the paper evaluates,
// for the query and key rows of a layer before the SWAN rotation: the paper
// rotates post-RoPE queries and keys, which is why P_QK cannot be folded into
// W_Q / W_K (Sec. 4.2).  Dims j and j + 64 of a row at position pos rotate by
// the angle pos * base^(-2j/128) ("rotate half" pairing), computed in float64
// and rounded once to the storage type, so the rows are what the cache's exact
// rotation then sees.
#include "swan_device.h"
#include "swan_internal.h"

namespace swan {

// one workgroup per row (b, h, i), lane j handles the pair (j, j + 64)
template <typename T>
__global__ __launch_bounds__(64) void rope_kernel(RopeLaunch a) {
  const int row = blockIdx.x;
  const int i = row % a.n;
  const int b = row / a.n / a.H;
  const int j = threadIdx.x;
  const T* x = (const T*)a.x + (int64_t)row * kD;
  T* y = (T*)a.y + (int64_t)row * kD;
  const double pos = (double)a.pos0[b] + (double)i;
  const double ang = pos * pow(a.base, -(2.0 * j) / kD);
  double s, c;
  sincos(ang, &s, &c);
  const double x0 = (double)(float)x[j], x1 = (double)(float)x[j + kD / 2];
  const double y0 = x0 * c - x1 * s;
  const double y1 = x1 * c + x0 * s;
  if constexpr (sizeof(T) == 2) {
    ((uint16_t*)y)[j] = (uint16_t)f64_to_f16_bits(y0);
    ((uint16_t*)y)[j + kD / 2] = (uint16_t)f64_to_f16_bits(y1);
  } else {
    y[j] = (float)y0;
    y[j + kD / 2] = (float)y1;
  }
}

hipError_t launch_rope(const RopeLaunch& a) {
  const dim3 grid(a.B * a.H * a.n);
  if (a.dtype == SWAN_F32)
    hipLaunchKernelGGL(rope_kernel<float>, grid, dim3(64), 0, a.stream, a);
  else
    hipLaunchKernelGGL(rope_kernel<_Float16>, grid, dim3(64), 0, a.stream, a);
  return hipGetLastError();
}

}  // namespace swan
