// One MHA attention launch for a batch whose sequences have several k_pad
// (Algorithm 1, attention part, with a per-sequence k): each sparse wave runs
// the body specialised on its own sequence's k_pad tier (the larger of its
// keys' and values' k_pad, rounded up to 16, 32, 48, 64, 80, 96 or 128; the
// smaller pages take spare groups), so a page pays for at most its tier, and
// one grid orders every sequence's splits longest first instead of several
// launches sharing the GPU side by side.  The tiers keep the kernel within
// registers: with every k_pad as a case (the one-page-at-a-time bodies of
// k_pad 104-120 among them) the compiler spills to scratch memory.  The fp16
// and E4M3 storage formats only; the body is in decode_mha.h.
#include "decode_mha.h"

namespace swan {

// Grid: n * Hq dense-buffer waves, then n * Hq * f.n_splits sparse waves,
// split-major (waves past a sequence's split count return at once).
template <typename T>
__global__ __launch_bounds__(64) void attn_fused_kernel(DecodeLaunch a, FusedSeqs f) {
  __shared__ __attribute__((aligned(16))) float qrep[(kD + 1) * kQRep];
  __shared__ __attribute__((aligned(16))) float acc[(kD + 1) * kAccCols];
  const int lane = threadIdx.x;
  const int U = f.n * a.Hq;
  int w = blockIdx.x;
  if (w < U) {
    buffer_wave<T>(a, f.seq[w / a.Hq], w % a.Hq, qrep, acc, lane);
    return;
  }
  w -= U;
  const int ui = w % U, split = w / U;
  const int i = ui / a.Hq, hq = ui % a.Hq;
  const int b = f.seq[i];
  switch (f.kp8[i]) {  // uniform over the wave
#define SWAN_KP8_CASE(n)                                                \
  case n:                                                               \
    sparse_wave<T, n, true>(a, b, hq, split, qrep, acc, lane);          \
    break;
    SWAN_KP8_CASE(2) SWAN_KP8_CASE(4) SWAN_KP8_CASE(6) SWAN_KP8_CASE(8)
    SWAN_KP8_CASE(10) SWAN_KP8_CASE(12) SWAN_KP8_CASE(16)
#undef SWAN_KP8_CASE
    default:
      break;
  }
}

int fused_tier(int kp8) { return kp8 <= 12 ? (kp8 + 1) & ~1 : 16; }

hipError_t launch_attn_fused(const DecodeLaunch& a, const FusedSeqs& f) {
  const dim3 grid(f.n * a.Hq * (f.n_splits + 1));
  if (a.dtype == SWAN_F16)
    hipLaunchKernelGGL(attn_fused_kernel<_Float16>, grid, dim3(64), 0, a.stream, a, f);
  else if (a.dtype == SWAN_F16_E4M3)
    hipLaunchKernelGGL(attn_fused_kernel<E4M3V>, grid, dim3(64), 0, a.stream, a, f);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace swan
