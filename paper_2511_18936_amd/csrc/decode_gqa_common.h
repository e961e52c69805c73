// Device pieces of the GQA value update shared by the one-pass GQA kernel
// and the two-pass value kernel: the dense value tile V[128 dims][64 tokens]
// filled by a scatter of one page's kept components, and O += P . V on MFMA.
// `Lds` is any struct with members vt[kD * kVtStride] (fp16),
// pt[2][2][GH][kPtStride] (fp16 probabilities: [page parity][hi, lo][head][token])
// and fr[2][GH] (rescale factors of the accumulator rows).
#pragma once

#include "decode_common.h"

namespace swan {

typedef _Float16 h4 __attribute__((ext_vector_type(4)));
typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int kVtStride = 68;    // halves per row of the value tile (64 + pad)
constexpr int kVt8Stride = 68;   // bytes per row of the E4M3 value tile (64 + pad)
constexpr int kPtStride = 68;    // halves per row of the probability tile (64 + pad)

// replicas of the GH-head query rows (lane % R): 8 keep the gathers of 8
// consecutive lanes on distinct banks; 4 for GH = 8 to bound the LDS
template <int GH>
constexpr int qrep_replicas() {
  return GH >= 8 ? 4 : 8;
}

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

// s[h] = q_hat_h . k for this lane's token and GH heads, from q_rep[dim][R][GH]
// (ql: this lane's replica) and the key page's kept components
template <typename T, int KP8, int GH>
__device__ __forceinline__ void gather_scores(const PageRegs<T, KP8>& kr, const float* ql,
                                              float* s) {
  using QV = typename QVec<GH>::type;
  constexpr int R = qrep_replicas<GH>();
#pragma unroll
  for (int h = 0; h < GH; ++h) s[h] = 0.f;
#pragma unroll
  for (int g = 0; g < KP8; ++g) {
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const float v = EntryVal<T, KP8>::get(kr, g, u);
      const QV q = *(const QV*)(ql + entry_idx(kr, g, u) * (R * GH));
#pragma unroll
      for (int h = 0; h < GH; ++h) s[h] = fmaf(q[h], v, s[h]);
    }
  }
}

// zero N 16-byte chunks, 64 per wave store (the last one partial)
template <int N>
__device__ __forceinline__ void zero_chunks(u32x4* z, int lane) {
#pragma unroll
  for (int i = 0; i < N / 64; ++i) z[64 * i + lane] = u32x4{0u, 0u, 0u, 0u};
  if (N % 64 != 0 && lane < N % 64) z[64 * (N / 64) + lane] = u32x4{0u, 0u, 0u, 0u};
}

// value wave, one page: zero the value tile, scatter the kept components.
// E4M3 values go into a byte tile V8[dims][tokens] of their codes (code 0 is +0),
// half the bytes to zero and to read back; the MFMA operand read decodes them.
template <typename T, int KP8, typename Lds>
__device__ __forceinline__ void gqa_scatter(const PageRegs<T, KP8>& vr, bool valid, Lds& sh,
                                            int lane) {
  wave_lds_fence();  // the previous page's tile reads come first
  if constexpr (std::is_same<T, E4M3V>::value) {
    constexpr int kRows = sizeof(sh.vt) / (kVtStride * 2);  // 128, or 129 with the spare row
    constexpr int kChunks = (kRows * kVt8Stride + 15) / 16;
    zero_chunks<kChunks>((u32x4*)sh.vt, lane);
    wave_lds_fence();
    if (valid) {
      uint8_t* vt8 = (uint8_t*)sh.vt + lane;
#pragma unroll
      for (int g = 0; g < KP8; ++g) {
        const u32x2 c = vr.val[g];
#pragma unroll
        for (int u = 0; u < 8; ++u)
          vt8[entry_idx(vr, g, u) * kVt8Stride] = (uint8_t)(((u < 4 ? c.x : c.y) >> (8 * (u & 3))) & 0xFFu);
      }
    }
    return;
  }
  zero_chunks<kD * kVtStride * 2 / 16>((u32x4*)sh.vt, lane);
  wave_lds_fence();
  if (valid) {
    uint16_t* vt16 = (uint16_t*)sh.vt + lane;
#pragma unroll
    for (int g = 0; g < KP8; ++g) {
#pragma unroll
      for (int u = 0; u < 8; ++u)
        vt16[entry_idx(vr, g, u) * kVtStride] = (uint16_t)entry_f16_bits<T, KP8>(vr, g, u);
    }
  }
}

// value wave, after the page barrier: rescale, then O += P . V on MFMA
// (k-steps of 16 tokens, n-tiles of 16 dims)
template <int GH, typename T, typename Lds>
__device__ __forceinline__ void gqa_mfma(const Lds& sh, int par, int lane, f4* acc) {
  const int row = lane & 15;
  const int kq = 4 * (lane >> 4);
  // accumulator rows 4 (lane / 16) + r hold head 4 (lane / 16) + r
  float fr[4];
  bool any = false;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int h = 4 * (lane >> 4) + r;
    fr[r] = h < GH ? sh.fr[par][h < GH ? h : 0] : 1.f;
  }
#pragma unroll
  for (int h = 0; h < GH; ++h) any |= sh.fr[par][h] != 1.f;
  if (any) {
#pragma unroll
    for (int nt = 0; nt < 8; ++nt)
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[nt][r] *= fr[r];
  }
  const bool arow = row < GH;
  const int rr = arow ? row : 0;
  const h4 zero = {(_Float16)0.f, (_Float16)0.f, (_Float16)0.f, (_Float16)0.f};
#pragma unroll
  for (int ks = 0; ks < 4; ++ks) {
    const h4 ahi = arow ? *(const h4*)&sh.pt[par][0][rr][16 * ks + kq] : zero;
    const h4 alo = arow ? *(const h4*)&sh.pt[par][1][rr][16 * ks + kq] : zero;
#pragma unroll
    for (int nt = 0; nt < 8; ++nt) {
      h4 b;
      if constexpr (std::is_same<T, E4M3V>::value) {
        typedef _Float16 h2 __attribute__((ext_vector_type(2)));
        const uint32_t w = *(const uint32_t*)((const uint8_t*)sh.vt +
                                              (16 * nt + row) * kVt8Stride + 16 * ks + kq);
        const h2 lo = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(w, 1.0f, false);
        const h2 hi = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(w, 1.0f, true);
        b = h4{lo.x, lo.y, hi.x, hi.y};
      } else {
        b = *(const h4*)(sh.vt + (16 * nt + row) * kVtStride + 16 * ks + kq);
      }
      acc[nt] = __builtin_amdgcn_mfma_f32_16x16x16f16(ahi, b, acc[nt], 0, 0, 0);
      acc[nt] = __builtin_amdgcn_mfma_f32_16x16x16f16(alo, b, acc[nt], 0, 0, 0);
    }
  }
}

}  // namespace swan
