// Decode attention for grouped-query attention (GQA, G query heads per KV
// head), fp16 storage: one wave streams a KV head's pages once for GH of its
// query heads.
//
// Per 64-token page (one token per lane):
//   scores      s_h = q_hat_h . k for the GH heads: one vector gather of the
//               GH rotated queries per kept component (q_rep[dim][8][GH])
//   softmax     lazy reference per head (as in the MHA kernel), p_h written
//               to an LDS tile P[16][64] in fp16 as hi + lo parts
//   values      the page's kept value components are scattered into a zeroed
//               dense tile V[128 dims][64 tokens] (fp16, exact), and
//               O[16][128] += P[16][64] . V[64][128] runs on MFMA
//               (v_mfma_f32_16x16x16f16, fp32 accumulation, once for the hi
//               and once for the lo part of P, so p keeps ~22 bits)
// The accumulators stay in registers; rows >= GH of P are zero.  This is
// the dense contraction of the value update, done once for all heads of the
// group, instead of GH scatters into LDS accumulators.
#include "decode_common.h"

namespace swan {

typedef _Float16 h4 __attribute__((ext_vector_type(4)));
typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int kGRep = 8;         // replicas of the GH-head query rows (lane % 8)
constexpr int kVtStride = 68;    // halves per row of the value tile (64 + pad)
constexpr int kPtStride = 68;    // halves per row of the probability tile (64 + pad)

template <int GH>
struct QVec;
template <>
struct QVec<2> {
  typedef float type __attribute__((ext_vector_type(2)));
};
template <>
struct QVec<4> {
  typedef float type __attribute__((ext_vector_type(4)));
};
template <>
struct QVec<8> {
  typedef float type __attribute__((ext_vector_type(8)));
};

template <int KP8, int GH>
struct GqaState {
  float m[GH];   // reference maxima (log2 units), wave-uniform
  float l[GH];   // per-lane sums of exp2(s - m)
  f4 acc[8];     // O tile: n-tile nt, rows 4 * (lane / 16) + r, column 16 nt + lane % 16
  bool first;
};

template <int KP8, int GH>
__device__ __forceinline__ void gqa_page(const PageRegs<_Float16, KP8>& kr,
                                         const PageRegs<_Float16, KP8>& vr, bool valid,
                                         const float* qrep, _Float16* vt, _Float16* pt, int lane,
                                         GqaState<KP8, GH>& st) {
  using QV = typename QVec<GH>::type;
  // ---- scores for the GH heads ----
  float s[GH];
#pragma unroll
  for (int h = 0; h < GH; ++h) s[h] = 0.f;
  if (valid) {
    const float* ql = qrep + (lane & (kGRep - 1)) * GH;  // replica lane % 8
#pragma unroll
    for (int g = 0; g < KP8; ++g) {
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const float v = EntryVal<_Float16, KP8>::get(kr, g, u);
        const QV q = *(const QV*)(ql + entry_idx(kr, g, u) * (kGRep * GH));
#pragma unroll
        for (int h = 0; h < GH; ++h) s[h] = fmaf(q[h], v, s[h]);
      }
    }
  } else {
#pragma unroll
    for (int h = 0; h < GH; ++h) s[h] = -INFINITY;
  }
  // ---- lazy softmax reference per head ----
  float fr[4] = {1.f, 1.f, 1.f, 1.f};  // rescale of this lane's accumulator rows
  bool raised = false;
#pragma unroll
  for (int h = 0; h < GH; ++h) {
    if (st.first) {
      st.m[h] = wave_max(s[h]);
    } else if (__ballot(s[h] > st.m[h] + kTau) != 0) {
      const float pm = wave_max(s[h]);
      const float f = exp2f(st.m[h] - pm);
      st.l[h] *= f;
      st.m[h] = pm;
#pragma unroll
      for (int r = 0; r < 4; ++r)
        if (4 * (lane >> 4) + r == h) fr[r] = f;
      raised = true;
    }
  }
  st.first = false;
  if (raised) {
#pragma unroll
    for (int nt = 0; nt < 8; ++nt)
#pragma unroll
      for (int r = 0; r < 4; ++r) st.acc[nt][r] *= fr[r];
  }
  // ---- probability tile P[h][token] = hi + lo ----
  wave_lds_fence();  // the previous page's tile reads come first
#pragma unroll
  for (int h = 0; h < GH; ++h) {
    const float p = valid ? exp2f(s[h] - st.m[h]) : 0.f;
    st.l[h] += p;
    const _Float16 hi = (_Float16)p;
    pt[h * kPtStride + lane] = hi;
    pt[16 * kPtStride + h * kPtStride + lane] = (_Float16)(p - (float)hi);
  }
  // ---- dense value tile: zero, then scatter this page's kept components ----
  {
    u32x4* z = (u32x4*)vt;
    constexpr int kChunks = kD * kVtStride * 2 / 16;
#pragma unroll
    for (int c = lane; c < kChunks; c += 64) z[c] = u32x4{0u, 0u, 0u, 0u};
  }
  wave_lds_fence();
  if (valid) {
    uint16_t* vt16 = (uint16_t*)vt + lane;
#pragma unroll
    for (int g = 0; g < KP8; ++g) {
      const u32x4 c = vr.val[g];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const uint32_t w = c[u >> 1];
        vt16[entry_idx(vr, g, u) * kVtStride] = (uint16_t)((u & 1) ? (w >> 16) : (w & 0xFFFFu));
      }
    }
  }
  wave_lds_fence();
  // ---- O += P . V on MFMA (k-steps of 16 tokens, n-tiles of 16 dims) ----
  const int row = lane & 15;
  const int kq = 4 * (lane >> 4);
#pragma unroll
  for (int ks = 0; ks < 4; ++ks) {
    const h4 ahi = *(const h4*)(pt + row * kPtStride + 16 * ks + kq);
    const h4 alo = *(const h4*)(pt + 16 * kPtStride + row * kPtStride + 16 * ks + kq);
#pragma unroll
    for (int nt = 0; nt < 8; ++nt) {
      const h4 b = *(const h4*)(vt + (16 * nt + row) * kVtStride + 16 * ks + kq);
      st.acc[nt] = __builtin_amdgcn_mfma_f32_16x16x16f16(ahi, b, st.acc[nt], 0, 0, 0);
      st.acc[nt] = __builtin_amdgcn_mfma_f32_16x16x16f16(alo, b, st.acc[nt], 0, 0, 0);
    }
  }
}

// Grid: n * Hq dense-buffer waves (one per query head), then n * Hkv * (G /
// GH) * g.n_splits sparse waves, each for GH query heads of one KV head.
template <int KP8, int GH>
__global__ __launch_bounds__(64) void attn_gqa_kernel(DecodeLaunch a, SeqGroup g) {
  __shared__ __attribute__((aligned(16))) float qrep[kD * kGRep * GH];
  __shared__ __attribute__((aligned(16))) _Float16 vt[kD * kVtStride];
  __shared__ __attribute__((aligned(16))) _Float16 pt[2 * 16 * kPtStride];
  const int lane = threadIdx.x;
  const int G = a.Hq / a.Hkv;
  const int pstride = a.n_splits + 1;
  int w = blockIdx.x;
  const int NB = g.n * a.Hq;
  if (w < NB) {  // dense-buffer wave, one query head (scratch: the value tile)
    const int b = g.seq[w / a.Hq], hq = w % a.Hq, h = hq / G;
    const int bhq = b * a.Hq + hq;
    const int L = a.tab.len[b];
    const int nb = L < a.bb ? L : a.bb;
    if (nb == 0) return;
    const int64_t ring_off = ((int64_t)b * a.Hkv + h) * a.bb * kD;
    float* part = a.part + ((int64_t)bhq * pstride + a.n_splits) * kPartFloats;
    float* scratch = (float*)vt;  // 128 + up to 4096 floats (the tile holds 4352)
    buffer_part<_Float16>((const _Float16*)a.k_ring + ring_off,
                          (const _Float16*)a.v_ring + ring_off, nb, a.qhat + (int64_t)bhq * kD,
                          scratch, scratch + kD, lane, part);
    return;
  }
  w -= NB;
  const int HC = G / GH;               // head chunks per KV head
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
  const int pbeg = (int)((int64_t)split * np / ns);
  const int pend = (int)((int64_t)(split + 1) * np / ns);
  const int k = a.tab.kact[b];
  const int64_t pbytes = page_bytes_of(2, k);
  const int64_t unit_off = a.tab.page_off[b] + (int64_t)h * a.n_pages_cap * pbytes;
  const char* kbase = (const char*)a.k_pages + unit_off;
  const char* vbase = (const char*)a.v_pages + unit_off;

  // q_rep[dim][r][head]: lane writes dims lane and lane + 64, all replicas
  const float* qh = a.qhat + ((int64_t)b * a.Hq + hq0) * kD;
#pragma unroll
  for (int hh = 0; hh < 2; ++hh) {
    const int d = lane + 64 * hh;
    float q[GH];
#pragma unroll
    for (int j = 0; j < GH; ++j) q[j] = qh[j * kD + d];
#pragma unroll
    for (int r = 0; r < kGRep; ++r)
#pragma unroll
      for (int j = 0; j < GH; ++j) qrep[(d * kGRep + r) * GH + j] = q[j];
  }
  // P tile rows >= GH stay zero
  {
    u32x4* z = (u32x4*)pt;
#pragma unroll
    for (int c = lane; c < 2 * 16 * kPtStride * 2 / 16; c += 64) z[c] = u32x4{0u, 0u, 0u, 0u};
  }
  wave_lds_fence();

  GqaState<KP8, GH> st;
  st.first = true;
#pragma unroll
  for (int j = 0; j < GH; ++j) {
    st.m[j] = 0.f;
    st.l[j] = 0.f;
  }
#pragma unroll
  for (int nt = 0; nt < 8; ++nt) st.acc[nt] = f4{0.f, 0.f, 0.f, 0.f};

  PageRegs<_Float16, KP8> ka, va, kb, vb;
  const int plast = pend - 1;
  load_page<_Float16, KP8>(ka, kbase + pbeg * pbytes, lane);
  load_page<_Float16, KP8>(va, vbase + pbeg * pbytes, lane);
  for (int p = pbeg; p < pend; p += 2) {
    const int p1 = p + 1 < plast ? p + 1 : plast;
    load_page<_Float16, KP8>(kb, kbase + p1 * pbytes, lane);
    load_page<_Float16, KP8>(vb, vbase + p1 * pbytes, lane);
    gqa_page<KP8, GH>(ka, va, p * kPage + lane < S, qrep, vt, pt, lane, st);
    const int p2 = p + 2 < plast ? p + 2 : plast;
    load_page<_Float16, KP8>(ka, kbase + p2 * pbytes, lane);
    load_page<_Float16, KP8>(va, vbase + p2 * pbytes, lane);
    if (p + 1 < pend) gqa_page<KP8, GH>(kb, vb, (p + 1) * kPage + lane < S, qrep, vt, pt, lane, st);
  }

  // partials: rows h < GH of the O tile, with each head's m and l
#pragma unroll
  for (int j = 0; j < GH; ++j) {
    const float lt = wave_sum(st.l[j]);
    if (lane == 0) {
      float* part = a.part + (((int64_t)b * a.Hq + hq0 + j) * pstride + split) * kPartFloats;
      part[0] = st.m[j];
      part[1] = lt;
    }
  }
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int hrow = 4 * (lane >> 4) + r;
    if (hrow < GH) {
      float* part = a.part + (((int64_t)b * a.Hq + hq0 + hrow) * pstride + split) * kPartFloats;
#pragma unroll
      for (int nt = 0; nt < 8; ++nt) part[4 + 16 * nt + (lane & 15)] = st.acc[nt][r];
    }
  }
}

template <int KP8, int GH>
static hipError_t launch_gqa_k(const DecodeLaunch& a, const SeqGroup& g) {
  const int G = a.Hq / a.Hkv;
  const dim3 grid(g.n * a.Hq + g.n * a.Hkv * (G / GH) * g.n_splits);
  hipLaunchKernelGGL((attn_gqa_kernel<KP8, GH>), grid, dim3(64), 0, a.stream, a, g);
  return hipGetLastError();
}

template <int GH>
static hipError_t launch_gqa_g(const DecodeLaunch& a, const SeqGroup& g, int kp8) {
  switch (kp8) {
#define SWAN_KP8_CASE(n) \
  case n:                \
    return launch_gqa_k<n, GH>(a, g);
    SWAN_KP8_CASE(1) SWAN_KP8_CASE(2) SWAN_KP8_CASE(3) SWAN_KP8_CASE(4)
    SWAN_KP8_CASE(5) SWAN_KP8_CASE(6) SWAN_KP8_CASE(7) SWAN_KP8_CASE(8)
    SWAN_KP8_CASE(9) SWAN_KP8_CASE(10) SWAN_KP8_CASE(11) SWAN_KP8_CASE(12)
    SWAN_KP8_CASE(13) SWAN_KP8_CASE(14) SWAN_KP8_CASE(15) SWAN_KP8_CASE(16)
#undef SWAN_KP8_CASE
    default:
      return hipErrorInvalidValue;
  }
}

int gqa_heads_per_wave(int G) {
  if (G % 8 == 0) return 8;
  if (G % 4 == 0) return 4;
  if (G % 2 == 0) return 2;
  return 1;
}

hipError_t launch_attn_gqa(const DecodeLaunch& a, const SeqGroup& g, int kp8) {
  switch (gqa_heads_per_wave(a.Hq / a.Hkv)) {
    case 8:
      return launch_gqa_g<8>(a, g, kp8);
    case 4:
      return launch_gqa_g<4>(a, g, kp8);
    case 2:
      return launch_gqa_g<2>(a, g, kp8);
    default:
      return hipErrorInvalidValue;
  }
}

}  // namespace swan
