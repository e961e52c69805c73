// Launches of the MHA decode kernel (decode_mha.h) for sequences whose keys and
// values have different k_pad, as in the key/value retention ablation of
// Appendix A.5 (Table 2).  The kernel is specialised on the larger k_pad and
// takes each role's own page size and active groups at run time, so each
// role's pages are still read once, at their own size.  These instances live
// in their own translation unit so that they compile in parallel with the
// equal-k_pad ones.
#include "decode_mha.h"

namespace swan {

template <typename T, int KP8>
static hipError_t launch_attn_asym_k(const DecodeLaunch& a, const SeqGroup& g) {
  const dim3 grid(g.n * a.Hq * (g.n_splits + 1));
  hipLaunchKernelGGL((attn_kernel<T, KP8, true>), grid, dim3(64), 0, a.stream, a, g);
  return hipGetLastError();
}

template <typename T>
static hipError_t launch_attn_asym_t(const DecodeLaunch& a, const SeqGroup& g, int kp8) {
  switch (kp8) {
#define SWAN_KP8_CASE(n) \
  case n:                \
    return launch_attn_asym_k<T, n>(a, g);
    SWAN_KP8_CASE(1) SWAN_KP8_CASE(2) SWAN_KP8_CASE(3) SWAN_KP8_CASE(4)
    SWAN_KP8_CASE(5) SWAN_KP8_CASE(6) SWAN_KP8_CASE(7) SWAN_KP8_CASE(8)
    SWAN_KP8_CASE(9) SWAN_KP8_CASE(10) SWAN_KP8_CASE(11) SWAN_KP8_CASE(12)
    SWAN_KP8_CASE(13) SWAN_KP8_CASE(14) SWAN_KP8_CASE(15) SWAN_KP8_CASE(16)
#undef SWAN_KP8_CASE
    default:
      return hipErrorInvalidValue;
  }
}

hipError_t launch_attn_asym(const DecodeLaunch& a, const SeqGroup& g, int kp8) {
  if (a.dtype == SWAN_F16) return launch_attn_asym_t<_Float16>(a, g, kp8);
  if (a.dtype == SWAN_F16_E4M3) return launch_attn_asym_t<E4M3V>(a, g, kp8);
  return launch_attn_asym_t<float>(a, g, kp8);
}

}  // namespace swan
