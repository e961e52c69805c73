// Two-pass decode, pass 1 of 2: the scores.  Used for sequences whose keys and
// values keep different numbers of components (their k_pad differ), as in the
// key/value retention ablation of Appendix A.5 (Table 2).  The one-pass kernels
// are specialised on a single k_pad for both roles; splitting the pass lets
// each kernel be specialised on its own role's k_pad.
//
// score_kernel: one wave per (sequence, GH query heads of one KV head, token
// split), one token per lane, streaming the key pages once for the GH heads:
//   s_h = q_hat_h . k  (log2 units: q_hat carries scale * log2(e)), gathered
//   from the rotated queries replicated in LDS as in the one-pass kernels;
//   every lane writes its token's score to the head's row of the workspace
//   (tokens past the end get -inf), and the split's exact maximum m_h goes to
//   word 0 of the head's partial for that split.
// The value pass (decode_value_pass.hip) then needs no running rescale.
#include "decode_gqa_common.h"

namespace swan {

// per-lane scores of one key page for GH heads
template <typename T, int KP8, int GH>
__device__ __forceinline__ void page_scores(const PageRegs<T, KP8>& kr, bool valid,
                                            const float* ql, float* s) {
  if (!valid) {
#pragma unroll
    for (int h = 0; h < GH; ++h) s[h] = -INFINITY;
    return;
  }
  if constexpr (GH == 1)
    s[0] = page_score<T, KP8>(kr, ql);
  else
    gather_scores<T, KP8, GH>(kr, ql, s);
}

// q_rep layout [dim][R][GH]; GH = 1 is the one-pass MHA layout [dim][kQRep]
template <int GH>
constexpr int score_replicas() {
  return GH == 1 ? kQRep : qrep_replicas<GH>();
}

// Grid: g.n * Hkv * (G / GH) * g.n_splits waves, split-major.
template <typename T, int KP8, int GH>
__global__ __launch_bounds__(64) void score_kernel(DecodeLaunch a, SeqGroup g) {
  constexpr int R = score_replicas<GH>();
  __shared__ __attribute__((aligned(16))) float qrep[kD * R * GH];
  const int lane = threadIdx.x;
  const int G = a.Hq / a.Hkv;
  const int HC = G / GH;  // head chunks per KV head
  const int units = g.n * a.Hkv * HC;
  const int split = blockIdx.x / units;
  const int ui = blockIdx.x % units;
  const int b = g.seq[ui / (a.Hkv * HC)];
  const int h = (ui / HC) % a.Hkv;
  const int hq0 = h * G + (ui % HC) * GH;
  const int L = a.tab.len[b];
  const int S = L > a.bb ? L - a.bb : 0;
  const int np = pages_for(S);
  const int nsb = a.tab.nsplit[b];
  const int ns = np < nsb ? np : nsb;
  if (split >= ns) return;
  const int pbeg = split_begin(split, ns, np);
  const int pend = split_begin(split + 1, ns, np);
  const int64_t pbytes = page_bytes_of(Fmt<T>::kValBytes, a.tab.kact[0][b]);
  const char* kbase =
      (const char*)a.k_pages + a.tab.page_off[0][b] + (int64_t)h * a.n_pages_cap * pbytes;

  // q_rep[dim][r][head]: lane writes dims lane and lane + 64
  const float* qh = a.qhat + ((int64_t)b * a.Hq + hq0) * kD;
#pragma unroll
  for (int hh = 0; hh < 2; ++hh) {
    const int d = lane + 64 * hh;
#pragma unroll
    for (int j = 0; j < GH; ++j) {
      const float v = qh[j * kD + d];
#pragma unroll
      for (int r = 0; r < R; ++r) qrep[(d * R + r) * GH + j] = v;
    }
  }
  wave_lds_fence();
  const float* ql = qrep + (lane & (R - 1)) * GH;
  float* srow = a.scores + ((int64_t)b * a.Hq + hq0) * a.score_stride + lane;
  float mx[GH], s[GH];
#pragma unroll
  for (int j = 0; j < GH; ++j) mx[j] = -INFINITY;
  auto consume = [&](const PageRegs<T, KP8>& kr, int p) {
    page_scores<T, KP8, GH>(kr, p * kPage + lane < S, ql, s);
#pragma unroll
    for (int j = 0; j < GH; ++j) {
      srow[j * a.score_stride + (int64_t)p * kPage] = s[j];
      mx[j] = fmaxf(mx[j], s[j]);
    }
  };
  constexpr int kChunks = KP8 * PageRegs<T, KP8>::VCH;
  if constexpr (kChunks <= 12) {  // two register sets: one page in flight
    PageRegs<T, KP8> ka, kb;
    const int plast = pend - 1;
    load_page<T, KP8>(ka, kbase + pbeg * pbytes, lane);
    for (int p = pbeg; p < pend; p += 2) {
      const int p1 = p + 1 < plast ? p + 1 : plast;
      load_page<T, KP8>(kb, kbase + p1 * pbytes, lane);
      consume(ka, p);
      const int p2 = p + 2 < plast ? p + 2 : plast;
      load_page<T, KP8>(ka, kbase + p2 * pbytes, lane);
      if (p + 1 < pend) consume(kb, p + 1);
    }
  } else {  // large pages: one page at a time
    PageRegs<T, KP8> ka;
    for (int p = pbeg; p < pend; ++p) {
      load_page<T, KP8>(ka, kbase + p * pbytes, lane);
      consume(ka, p);
    }
  }
  const int pstride = a.n_splits + 1;
#pragma unroll
  for (int j = 0; j < GH; ++j) {
    const float m = wave_max(mx[j]);
    if (lane == 0) a.part[(((int64_t)b * a.Hq + hq0 + j) * pstride + split) * kPartFloats] = m;
  }
}

template <typename T, int KP8, int GH>
static hipError_t launch_score_k(const DecodeLaunch& a, const SeqGroup& g) {
  const dim3 grid(g.n * a.Hkv * (a.Hq / a.Hkv / GH) * g.n_splits);
  hipLaunchKernelGGL((score_kernel<T, KP8, GH>), grid, dim3(64), 0, a.stream, a, g);
  return hipGetLastError();
}

template <typename T, int GH>
static hipError_t launch_score_g(const DecodeLaunch& a, const SeqGroup& g, int kp8) {
  switch (kp8) {
#define SWAN_KP8_CASE(n) \
  case n:                \
    return launch_score_k<T, n, GH>(a, g);
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
static hipError_t launch_score_t(const DecodeLaunch& a, const SeqGroup& g, int kp8, int gh) {
  switch (gh) {
    case 1:
      return launch_score_g<T, 1>(a, g, kp8);
    case 2:
      return launch_score_g<T, 2>(a, g, kp8);
    case 4:
      return launch_score_g<T, 4>(a, g, kp8);
    case 8:
      return launch_score_g<T, 8>(a, g, kp8);
    default:
      return hipErrorInvalidValue;
  }
}

hipError_t launch_score_pass(const DecodeLaunch& a, const SeqGroup& g, int kp8_key) {
  const int gh = decode_heads_per_wave(a.dtype, a.Hq, a.Hkv);
  if (a.dtype == SWAN_F16) return launch_score_t<_Float16>(a, g, kp8_key, gh);
  if (a.dtype == SWAN_F16_E4M3) return launch_score_t<E4M3V>(a, g, kp8_key, gh);
  if (gh != 1) return hipErrorInvalidValue;
  return launch_score_g<float, 1>(a, g, kp8_key);
}

}  // namespace swan
