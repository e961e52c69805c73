// Two-pass decode, pass 2 of 2: the values (pass 1 is decode_score_pass.hip).
// For sequences whose keys and values have different k_pad (the key/value
// retention ablation of Appendix A.5); each launch is specialised on the
// values' k_pad.
//
// With the split's exact maximum m from pass 1, p = exp2(s - m) needs no
// running rescale.  Per (sequence, query head, split) the pass completes the
// partial (m, l = sum p, acc = sum p v) that the merge kernel reads.
//   value_kernel      (one query head per wave) one token per lane: reads the
//                     token's score and its value page entries and updates the
//                     lane-private accumulator acc[dim][lane] in LDS, as the
//                     one-pass kernel does
//   gqa_value_kernel  (GQA, fp16 storage: GH query heads per wave) the wave
//                     writes the page's probabilities for its GH heads to a
//                     P tile (fp16 hi + lo), scatters the value page into a
//                     dense V tile, and runs O += P . V on MFMA, as the value
//                     wave of the one-pass GQA kernel does
// Both launches also carry one dense-buffer wave per (sequence, query head),
// which writes the buffer's complete partial (slot n_splits).
#include "decode_gqa_common.h"

namespace swan {

hipError_t launch_score_pass(const DecodeLaunch& a, const SeqGroup& g, int kp8_key);

// dense-buffer wave w (< g.n * Hq) of a value launch
template <typename E>
__device__ __forceinline__ void ring_wave(const DecodeLaunch& a, const SeqGroup& g, int w,
                                          float* qs, float* pb, int lane) {
  const int G = a.Hq / a.Hkv;
  const int b = g.seq[w / a.Hq], hq = w % a.Hq, h = hq / G;
  const int bhq = b * a.Hq + hq;
  const int L = a.tab.len[b];
  const int nb = L < a.bb ? L : a.bb;
  if (nb == 0) return;
  const int64_t ring_off = ((int64_t)b * a.Hkv + h) * a.bb * kD;
  float* part = a.part + ((int64_t)bhq * (a.n_splits + 1) + a.n_splits) * kPartFloats;
  buffer_part<E>((const E*)a.k_ring + ring_off, (const E*)a.v_ring + ring_off, nb,
                 a.qhat + (int64_t)bhq * kD, qs, pb, lane, part);
}

// Grid: g.n * Hq dense-buffer waves, then g.n * Hq * g.n_splits sparse waves.
template <typename T, int KP8>
__global__ __launch_bounds__(64) void value_kernel(DecodeLaunch a, SeqGroup g) {
  __shared__ __attribute__((aligned(16))) float acc[kD * kAccCols];
  __shared__ __attribute__((aligned(16))) float qs[kD];
  const int lane = threadIdx.x;
  const int NB = g.n * a.Hq;
  int w = blockIdx.x;
  if (w < NB) {
    ring_wave<typename Fmt<T>::Elem>(a, g, w, qs, acc, lane);
    return;
  }
  w -= NB;
  const int split = w / NB;
  const int gi = w % NB;
  const int b = g.seq[gi / a.Hq], hq = gi % a.Hq, h = hq / (a.Hq / a.Hkv);
  const int bhq = b * a.Hq + hq;
  const int L = a.tab.len[b];
  const int S = L > a.bb ? L - a.bb : 0;
  const int np = pages_for(S);
  const int nsb = a.tab.nsplit[b];
  const int ns = np < nsb ? np : nsb;
  if (split >= ns) return;
  const int pbeg = split_begin(split, ns, np);
  const int pend = split_begin(split + 1, ns, np);
  const int64_t pbytes = page_bytes_of(Fmt<T>::kValBytes, a.tab.kact[1][b]);
  const char* vbase =
      (const char*)a.v_pages + a.tab.page_off[1][b] + (int64_t)h * a.n_pages_cap * pbytes;
  const float* srow = a.scores + (int64_t)bhq * a.score_stride + lane;
  float* part = a.part + ((int64_t)bhq * (a.n_splits + 1) + split) * kPartFloats;
  const float m = part[0];  // the split's maximum, written by the score pass

#pragma unroll 8
  for (int c = 0; c < kAccCols / 2; ++c)
    ((float4*)acc)[c * 64 + lane] = make_float4(0.f, 0.f, 0.f, 0.f);
  wave_lds_fence();
  float* acc_l = acc + lane;
  float l = 0.f;
  auto consume = [&](const PageRegs<T, KP8>& vr, float s, int p) {
    const bool valid = p * kPage + lane < S;
    const float pr = valid ? exp2f(s - m) : 0.f;
    l += pr;
    page_accumulate<T, KP8>(vr, acc_l, pr, valid);
  };
  constexpr int kChunks = KP8 * PageRegs<T, KP8>::VCH;
  if constexpr (kChunks <= 12) {  // two register sets: one page in flight
    PageRegs<T, KP8> va, vb;
    float sa, sb;
    const int plast = pend - 1;
    load_page<T, KP8>(va, vbase + pbeg * pbytes, lane);
    sa = srow[(int64_t)pbeg * kPage];
    for (int p = pbeg; p < pend; p += 2) {
      const int p1 = p + 1 < plast ? p + 1 : plast;
      load_page<T, KP8>(vb, vbase + p1 * pbytes, lane);
      sb = srow[(int64_t)p1 * kPage];
      consume(va, sa, p);
      const int p2 = p + 2 < plast ? p + 2 : plast;
      load_page<T, KP8>(va, vbase + p2 * pbytes, lane);
      sa = srow[(int64_t)p2 * kPage];
      if (p + 1 < pend) consume(vb, sb, p + 1);
    }
  } else {  // large pages: one page at a time
    PageRegs<T, KP8> va;
    for (int p = pbeg; p < pend; ++p) {
      load_page<T, KP8>(va, vbase + p * pbytes, lane);
      consume(va, srow[(int64_t)p * kPage], p);
    }
  }
  const float ltot = wave_sum(l);
  wave_lds_fence();
  reduce_acc(acc, lane, part);
  if (lane == 0) part[1] = ltot;
}

// LDS of the GQA value wave: the tiles of gqa_scatter / gqa_mfma (one parity
// in use: a single wave orders its own LDS accesses)
template <int GH>
struct GqaValueLds {
  _Float16 vt[kD * kVtStride];
  _Float16 pt[2][2][GH][kPtStride];
  float fr[2][GH];
};

// Grid: g.n * Hq dense-buffer waves, then g.n * Hkv * (G / GH) * g.n_splits
// sparse waves, each for GH query heads of one KV head.
template <typename T, int KP8, int GH>
__global__ __launch_bounds__(64) void gqa_value_kernel(DecodeLaunch a, SeqGroup g) {
  __shared__ __attribute__((aligned(16))) GqaValueLds<GH> sh;
  const int lane = threadIdx.x;
  const int NB = g.n * a.Hq;
  int w = blockIdx.x;
  if (w < NB) {  // scratch: the value tile (128 + up to 4096 floats fit in its 4352)
    float* scratch = (float*)sh.vt;
    ring_wave<typename Fmt<T>::Elem>(a, g, w, scratch, scratch + kD, lane);
    return;
  }
  w -= NB;
  const int G = a.Hq / a.Hkv;
  const int HC = G / GH;
  const int units = g.n * a.Hkv * HC;
  const int split = w / units;
  const int ui = w % units;
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
  const int64_t pbytes = page_bytes_of(Fmt<T>::kValBytes, a.tab.kact[1][b]);
  const char* vbase =
      (const char*)a.v_pages + a.tab.page_off[1][b] + (int64_t)h * a.n_pages_cap * pbytes;
  const int pstride = a.n_splits + 1;
  const float* srow = a.scores + ((int64_t)b * a.Hq + hq0) * a.score_stride + lane;
  float m[GH], l[GH];
#pragma unroll
  for (int j = 0; j < GH; ++j) {
    m[j] = a.part[(((int64_t)b * a.Hq + hq0 + j) * pstride + split) * kPartFloats];
    l[j] = 0.f;
  }
  if (lane < GH) {  // exact maxima: the accumulator rows are never rescaled
    sh.fr[0][lane] = 1.f;
    sh.fr[1][lane] = 1.f;
  }
  f4 acc[8];
#pragma unroll
  for (int nt = 0; nt < 8; ++nt) acc[nt] = f4{0.f, 0.f, 0.f, 0.f};
  auto consume = [&](const PageRegs<T, KP8>& vr, const float* s, int p) {
    const bool valid = p * kPage + lane < S;
    wave_lds_fence();  // the previous page's tile reads come first
#pragma unroll
    for (int j = 0; j < GH; ++j) {
      const float pr = valid ? exp2f(s[j] - m[j]) : 0.f;
      l[j] += pr;
      const _Float16 hi = (_Float16)pr;
      sh.pt[0][0][j][lane] = hi;
      sh.pt[0][1][j][lane] = (_Float16)(pr - (float)hi);
    }
    gqa_scatter<T, KP8>(vr, valid, sh, lane);
    wave_lds_fence();
    gqa_mfma<GH>(sh, 0, lane, acc);
  };
  auto load_scores = [&](float* s, int p) {
#pragma unroll
    for (int j = 0; j < GH; ++j) s[j] = srow[j * a.score_stride + (int64_t)p * kPage];
  };
  PageRegs<T, KP8> va, vb;
  float sa[GH], sb[GH];
  const int plast = pend - 1;
  load_page<T, KP8>(va, vbase + pbeg * pbytes, lane);
  load_scores(sa, pbeg);
  for (int p = pbeg; p < pend; p += 2) {
    const int p1 = p + 1 < plast ? p + 1 : plast;
    load_page<T, KP8>(vb, vbase + p1 * pbytes, lane);
    load_scores(sb, p1);
    consume(va, sa, p);
    const int p2 = p + 2 < plast ? p + 2 : plast;
    load_page<T, KP8>(va, vbase + p2 * pbytes, lane);
    load_scores(sa, p2);
    if (p + 1 < pend) consume(vb, sb, p + 1);
  }
#pragma unroll
  for (int j = 0; j < GH; ++j) {
    const float lt = wave_sum(l[j]);
    if (lane == 0) a.part[(((int64_t)b * a.Hq + hq0 + j) * pstride + split) * kPartFloats + 1] = lt;
  }
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int hrow = 4 * (lane >> 4) + r;
    if (hrow < GH) {
      float* part = a.part + (((int64_t)b * a.Hq + hq0 + hrow) * pstride + split) * kPartFloats;
#pragma unroll
      for (int nt = 0; nt < 8; ++nt) part[4 + 16 * nt + (lane & 15)] = acc[nt][r];
    }
  }
}

template <typename T, int KP8, int GH>
static hipError_t launch_value_k(const DecodeLaunch& a, const SeqGroup& g) {
  if constexpr (GH == 1) {
    const dim3 grid(g.n * a.Hq * (g.n_splits + 1));
    hipLaunchKernelGGL((value_kernel<T, KP8>), grid, dim3(64), 0, a.stream, a, g);
  } else {
    const dim3 grid(g.n * a.Hq + g.n * a.Hkv * (a.Hq / a.Hkv / GH) * g.n_splits);
    hipLaunchKernelGGL((gqa_value_kernel<T, KP8, GH>), grid, dim3(64), 0, a.stream, a, g);
  }
  return hipGetLastError();
}

template <typename T, int GH>
static hipError_t launch_value_g(const DecodeLaunch& a, const SeqGroup& g, int kp8) {
  switch (kp8) {
#define SWAN_KP8_CASE(n) \
  case n:                \
    return launch_value_k<T, n, GH>(a, g);
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
static hipError_t launch_value_t(const DecodeLaunch& a, const SeqGroup& g, int kp8, int gh) {
  switch (gh) {
    case 1:
      return launch_value_g<T, 1>(a, g, kp8);
    case 2:
      return launch_value_g<T, 2>(a, g, kp8);
    case 4:
      return launch_value_g<T, 4>(a, g, kp8);
    case 8:
      return launch_value_g<T, 8>(a, g, kp8);
    default:
      return hipErrorInvalidValue;
  }
}

hipError_t launch_two_pass(const DecodeLaunch& a, const SeqGroup& g, int kp8_key, int kp8_val) {
  // score_stride is 0 when no two-pass sequence has a sparse token: then the
  // score pass has nothing to do, and only the value pass's dense-buffer waves
  // do work (its sparse waves return before touching the scores)
  if (a.score_stride > 0) {
    if (!a.scores) return hipErrorInvalidValue;
    const hipError_t e = launch_score_pass(a, g, kp8_key);
    if (e != hipSuccess) return e;
  }
  const int gh = decode_heads_per_wave(a.dtype, a.Hq, a.Hkv);
  if (a.dtype == SWAN_F16) return launch_value_t<_Float16>(a, g, kp8_val, gh);
  if (a.dtype == SWAN_F16_E4M3) return launch_value_t<E4M3V>(a, g, kp8_val, gh);
  if (gh != 1) return hipErrorInvalidValue;
  return launch_value_g<float, 1>(a, g, kp8_val);
}

}  // namespace swan
