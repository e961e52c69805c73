// Decode attention for grouped-query attention (GQA, G query heads per KV
// head), fp16 storage with fp16 or E4M3 sparse values: one workgroup of two
// waves streams a KV head's pages once for GH of its query heads.
//
// Per 64-token page (one token per lane in each wave):
//   score wave  holds the key pages: s_h = q_hat_h . k for the GH heads, one
//               vector gather of the GH rotated queries per kept component
//               (q_rep[dim][replica][GH]); lazy softmax reference per head (as
//               in the MHA kernel); p_h goes to a double-buffered LDS tile
//               P[GH][64] in fp16 as hi + lo parts, with the rescale factor of
//               each head's accumulator row
//   value wave  holds the value pages: scatters the page's kept components
//               into a zeroed dense tile V[128 dims][64 tokens] (fp16, exact),
//               then O[16][128] += P[16][64] . V[64][128] on MFMA
//               (v_mfma_f32_16x16x16f16, fp32 accumulation, once for the hi
//               and once for the lo part of P, so p keeps ~22 bits)
// The waves meet at one workgroup barrier per page: the value wave's MFMA of
// page p overlaps the score wave's work on page p + 1.  The accumulators stay
// in the value wave's registers; rows >= GH of the MFMA's A operand are zero.
// This is the dense contraction of the value update, done once for all heads
// of the group, instead of GH scatters into LDS accumulators.
//
// This header holds the kernel, shared by the launches for equal and for
// different key / value k_pad.
#pragma once

#include "decode_gqa_common.h"

namespace swan {

// kRows: kD, plus the spare row kSpareRow when the kernel loads spare groups
template <int GH, int kRows>
struct GqaLds {
  float qrep[kRows * qrep_replicas<GH>() * GH];
  _Float16 vt[kRows * kVtStride];
  _Float16 pt[2][2][GH][kPtStride];  // [page parity][hi, lo][head][token]
  float fr[2][GH];                   // [page parity][head]: accumulator rescale
};

// score wave, one page: scores, softmax reference, P tile and rescale factors
template <typename T, int KP8, int GH, typename Lds>
__device__ __forceinline__ void gqa_scores(const PageRegs<T, KP8>& kr, bool valid, Lds& sh,
                                           int par, int lane, float* m, float* l, bool& first) {
  constexpr int R = qrep_replicas<GH>();
  float s[GH];
  if (valid) {
    gather_scores<T, KP8, GH>(kr, sh.qrep + (lane & (R - 1)) * GH, s);
  } else {
#pragma unroll
    for (int h = 0; h < GH; ++h) s[h] = -INFINITY;
  }
  float frl = 1.f;  // lane h < GH: rescale factor of head h
#pragma unroll
  for (int h = 0; h < GH; ++h) {
    if (first) {
      m[h] = wave_max(s[h]);
    } else if (__ballot(s[h] > m[h] + kTau) != 0) {
      const float pm = wave_max(s[h]);
      const float f = exp2f(m[h] - pm);
      l[h] *= f;
      m[h] = pm;
      if (lane == h) frl = f;
    }
  }
  first = false;
#pragma unroll
  for (int h = 0; h < GH; ++h) {
    const float p = valid ? exp2f(s[h] - m[h]) : 0.f;
    l[h] += p;
    const _Float16 hi = (_Float16)p;
    sh.pt[par][0][h][lane] = hi;
    sh.pt[par][1][h][lane] = (_Float16)(p - (float)hi);
  }
  if (lane < GH) sh.fr[par][lane] = frl;
}

// Grid: n * Hkv * (G / GH) * g.n_splits sparse blocks, each for GH query heads
// of one KV head, then n * Hq dense-buffer blocks (wave 0 serves one query head).  kAsym: keys and values have different k_pad, the larger being
// 8 KP8; each wave then takes its role's page size and loaded groups at run
// time, the rest being spare groups (load_page), for which q_rep and the value
// tile get a spare row kSpareRow.
template <typename T, int KP8, int GH, bool kAsym>
__global__ __launch_bounds__(128) void attn_gqa_kernel(DecodeLaunch a, SeqGroup g) {
  constexpr int R = qrep_replicas<GH>();
  __shared__ __attribute__((aligned(16))) GqaLds<GH, kAsym ? kD + 1 : kD> sh;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // 0: scores, 1: values
  const int lane = threadIdx.x & 63;
  const int G = a.Hq / a.Hkv;
  const int pstride = a.n_splits + 1;
  int w = blockIdx.x;
  const int HC = G / GH;               // head chunks per KV head
  const int units = g.n * a.Hkv * HC;
  const int nsparse = units * g.n_splits;
  if (w >= nsparse) {  // dense-buffer block, after the sparse ones: one wave (scratch: the value tile)
    if (wave != 0) return;
    const int wr = w - nsparse;
    const int b = g.seq[wr / a.Hq], hq = wr % a.Hq, h = hq / G;
    const int bhq = b * a.Hq + hq;
    const int L = a.tab.len[b];
    const int nb = L < a.bb ? L : a.bb;
    if (nb == 0) return;
    const int64_t ring_off = ((int64_t)b * a.Hkv + h) * a.bb * kD;
    float* part = a.part + ((int64_t)bhq * pstride + a.n_splits) * kPartFloats;
    float* scratch = (float*)sh.vt;  // 128 + up to 4096 floats (the tile holds 4352)
    buffer_part<_Float16>((const _Float16*)a.k_ring + ring_off,
                          (const _Float16*)a.v_ring + ring_off, nb, a.qhat + (int64_t)bhq * kD,
                          scratch, scratch + kD, lane, part);
    return;
  }
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
  if (split >= ns) return;  // uniform over the block
  const int pbeg = split_begin(split, ns, np, a.tab.flat[b] != 0);
  const int pend = split_begin(split + 1, ns, np, a.tab.flat[b] != 0);
  // the page size and loaded groups of this wave's role
  const int role = kAsym ? wave : 0;
  const int64_t pbytes = page_bytes_of(Fmt<T>::kValBytes, a.tab.kact[role][b]);
  const int n8 = kAsym ? kpad_of(a.tab.kact[role][b]) / 8 : KP8;
  const int64_t head_off = (int64_t)h * a.n_pages_cap * pbytes;
  // this wave's role pages.  Pages up to 192 bytes per lane (fp16 up to k_pad
  // 64) load the first page before the query replicas are filled, so that its
  // latency overlaps the fill and the barrier; larger pages keep their
  // registers free of it there (two waves per SIMD need the kernel within 256
  // registers).
  constexpr bool kEarly = sizeof(PageRegs<T, KP8>) <= 192;
  const char* rbase = wave == 0 ? (const char*)a.k_pages + a.tab.page_off[0][b] + head_off
                                : (const char*)a.v_pages + a.tab.page_off[1][b] + head_off;
  PageRegs<T, KP8> ra, rb;  // the wave's two page register sets
  if constexpr (kEarly) load_page<T, KP8>(ra, rbase + pbeg * pbytes, lane, n8);

  // q_rep[dim][r][head]: thread t writes dim t, all replicas
  {
    const int d = threadIdx.x;
    const float* qh = a.qhat + ((int64_t)b * a.Hq + hq0) * kD;
    float q[GH];
#pragma unroll
    for (int j = 0; j < GH; ++j) q[j] = qh[j * kD + d];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int j = 0; j < GH; ++j) sh.qrep[(d * R + r) * GH + j] = q[j];
    if (kAsym && d < R * GH) sh.qrep[kSpareRow * R * GH + d] = 0.f;  // the spare row's q is 0
  }
  __syncthreads();

  const int plast = pend - 1;
  if (wave == 0) {
    // ---- score wave ----
    const char* kbase = rbase;
    float m[GH], l[GH];
    bool first = true;
#pragma unroll
    for (int j = 0; j < GH; ++j) {
      m[j] = 0.f;
      l[j] = 0.f;
    }
    PageRegs<T, KP8>& ka = ra;
    PageRegs<T, KP8>& kb = rb;
    if constexpr (!kEarly) load_page<T, KP8>(ka, kbase + pbeg * pbytes, lane, n8);
    for (int p = pbeg; p < pend; p += 2) {
      const bool in1 = p + 1 <= plast;  // past the split: the resident spare arrays
      load_page<T, KP8>(kb, kbase + (in1 ? p + 1 : plast) * pbytes, lane, in1 ? n8 : 0);
      gqa_scores<T, KP8, GH>(ka, p * kPage + lane < S, sh, (p - pbeg) & 1, lane, m, l, first);
      __syncthreads();
      const bool in2 = p + 2 <= plast;
      load_page<T, KP8>(ka, kbase + (in2 ? p + 2 : plast) * pbytes, lane, in2 ? n8 : 0);
      if (p + 1 < pend) {
        gqa_scores<T, KP8, GH>(kb, (p + 1) * kPage + lane < S, sh, (p + 1 - pbeg) & 1, lane, m, l,
                               first);
        __syncthreads();
      }
    }
#pragma unroll
    for (int j = 0; j < GH; ++j) {
      const float lt = wave_sum(l[j]);
      if (lane == 0) {
        float* part = a.part + (((int64_t)b * a.Hq + hq0 + j) * pstride + split) * kPartFloats;
        part[0] = m[j];
        part[1] = lt;
      }
    }
  } else {
    // ---- value wave ----
    const char* vbase = rbase;
    f4 acc[8];
#pragma unroll
    for (int nt = 0; nt < 8; ++nt) acc[nt] = f4{0.f, 0.f, 0.f, 0.f};
    PageRegs<T, KP8>& va = ra;
    PageRegs<T, KP8>& vb = rb;
    if constexpr (!kEarly) load_page<T, KP8>(va, vbase + pbeg * pbytes, lane, n8);
    for (int p = pbeg; p < pend; p += 2) {
      const bool in1 = p + 1 <= plast;  // past the split: the resident spare arrays
      load_page<T, KP8>(vb, vbase + (in1 ? p + 1 : plast) * pbytes, lane, in1 ? n8 : 0);
      gqa_scatter<T, KP8>(va, p * kPage + lane < S, sh, lane);
      __syncthreads();
      gqa_mfma<GH, T>(sh, (p - pbeg) & 1, lane, acc);
      const bool in2 = p + 2 <= plast;
      load_page<T, KP8>(va, vbase + (in2 ? p + 2 : plast) * pbytes, lane, in2 ? n8 : 0);
      if (p + 1 < pend) {
        gqa_scatter<T, KP8>(vb, (p + 1) * kPage + lane < S, sh, lane);
        __syncthreads();
        gqa_mfma<GH, T>(sh, (p + 1 - pbeg) & 1, lane, acc);
      }
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
}

}  // namespace swan
