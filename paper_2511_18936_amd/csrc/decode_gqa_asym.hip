// Launches of the GQA decode kernel (decode_gqa.h) for sequences whose keys and
// values have different k_pad (Appendix A.5, Table 2).  The kernel is
// specialised on the larger k_pad; its score wave takes the keys' page size
// and active groups at run time and its value wave the values'.  Kept in a
// translation unit of its own so that it compiles in parallel with the
// equal-k_pad launches.
#include "decode_gqa.h"

namespace swan {

template <typename T, int KP8, int GH>
static hipError_t launch_gqa_asym_k(const DecodeLaunch& a, const SeqGroup& g) {
  const int G = a.Hq / a.Hkv;
  const dim3 grid(g.n * a.Hq + g.n * a.Hkv * (G / GH) * g.n_splits);
  hipLaunchKernelGGL((attn_gqa_kernel<T, KP8, GH, true>), grid, dim3(128), 0, a.stream, a, g);
  return hipGetLastError();
}

template <typename T, int GH>
static hipError_t launch_gqa_asym_g(const DecodeLaunch& a, const SeqGroup& g, int kp8) {
  switch (kp8) {
#define SWAN_KP8_CASE(n) \
  case n:                \
    return launch_gqa_asym_k<T, n, GH>(a, g);
    SWAN_KP8_CASE(1) SWAN_KP8_CASE(2) SWAN_KP8_CASE(3) SWAN_KP8_CASE(4)
    SWAN_KP8_CASE(5) SWAN_KP8_CASE(6) SWAN_KP8_CASE(7) SWAN_KP8_CASE(8)
    SWAN_KP8_CASE(9) SWAN_KP8_CASE(10) SWAN_KP8_CASE(11) SWAN_KP8_CASE(12)
    SWAN_KP8_CASE(13) SWAN_KP8_CASE(14) SWAN_KP8_CASE(15) SWAN_KP8_CASE(16)
#undef SWAN_KP8_CASE
    default:
      return hipErrorInvalidValue;
  }
}

template <typename T>
static hipError_t launch_gqa_asym_t(const DecodeLaunch& a, const SeqGroup& g, int kp8) {
  switch (gqa_heads_per_wave(a.Hq / a.Hkv)) {
    case 8:
      return launch_gqa_asym_g<T, 8>(a, g, kp8);
    case 4:
      return launch_gqa_asym_g<T, 4>(a, g, kp8);
    case 2:
      return launch_gqa_asym_g<T, 2>(a, g, kp8);
    default:
      return hipErrorInvalidValue;
  }
}

hipError_t launch_attn_gqa_asym(const DecodeLaunch& a, const SeqGroup& g, int kp8) {
  if (a.dtype == SWAN_F16_E4M3) return launch_gqa_asym_t<E4M3V>(a, g, kp8);
  return launch_gqa_asym_t<_Float16>(a, g, kp8);
}

}  // namespace swan
