// Device pieces shared by the decode attention kernels (MHA and GQA): page
// registers and loads, the lazy-softmax state, and the dense-buffer partial.
#pragma once

#include <type_traits>

#include "swan_device.h"
#include "swan_internal.h"

namespace swan {

constexpr float kTau = 8.0f;

// ---------------------------------------------------------------------------
// page registers: KP8 groups of 8 entries; VCH value chunks per group
// ---------------------------------------------------------------------------
template <typename T, int KP8>
struct PageRegs {
  static constexpr int CB = Fmt<T>::kChunkBytes;
  static constexpr int VCH = 8 * Fmt<T>::kValBytes / CB;
  using VChunk = typename std::conditional<CB == 16, u32x4, u32x2>::type;
  VChunk val[KP8 * VCH];
  u32x2 idx[KP8];
};

// Spare groups.  The registers hold KP8 groups of 8 entries; a page of a
// smaller k_pad = 8 n8 (n8 < KP8, wave-uniform) fills the first n8 of them.
// Groups n8..KP8-1 are loaded from the two read-only arrays below instead:
// value 0 and index kSpareRow, a row past the head dimension that the
// kernels using spare groups add to their LDS query replicas (zeroed), their
// accumulators and their value tiles.  So the compute runs over all KP8
// groups with no branch (a branch per group keeps the compiler from batching
// a page's LDS accesses), and the spare entries change nothing: 0 * q = 0 in
// the score, and the accumulator updates land in the spare row.  With
// n8 = KP8 (a compile-time constant) the selection folds away.
constexpr int kSpareRow = kD;
#define SWAN_X8(v) v, v, v, v, v, v, v, v
#define SWAN_X64(v) SWAN_X8(v), SWAN_X8(v), SWAN_X8(v), SWAN_X8(v), \
                    SWAN_X8(v), SWAN_X8(v), SWAN_X8(v), SWAN_X8(v)
static __device__ const u32x4 kZeroChunks[64] = {};  // a value chunk of 64 lanes
static __device__ const uint32_t kSpareIdx[128] = {SWAN_X64(0x80808080u),
                                                   SWAN_X64(0x80808080u)};  // kSpareRow bytes
#undef SWAN_X64
#undef SWAN_X8
static_assert(kSpareRow == 0x80, "the spare index bytes are 0x80");

// Loads one page into registers (nontemporal: the pages are streamed once).
// The addresses are global-memory pointers so that the choice between page
// and spare arrays stays a global load (a generic pointer would make it a
// flat load, which also holds up the waits for LDS accesses).
#define SWAN_GLOBAL __attribute__((address_space(1)))
template <typename T, int KP8>
__device__ __forceinline__ void load_page(PageRegs<T, KP8>& r, const char* page, int lane,
                                          int n8 = KP8) {
  using PR = PageRegs<T, KP8>;
  using Chunk = typename PR::VChunk;
  const SWAN_GLOBAL char* pg = (const SWAN_GLOBAL char*)page;
  const SWAN_GLOBAL char* vp = pg + lane * PR::CB;
  const SWAN_GLOBAL char* zp = (const SWAN_GLOBAL char*)kZeroChunks + lane * PR::CB;
#pragma unroll
  for (int c = 0; c < KP8 * PR::VCH; ++c) {
    const SWAN_GLOBAL char* src = c < n8 * PR::VCH ? vp + c * 64 * PR::CB : zp;
    r.val[c] = __builtin_nontemporal_load((const SWAN_GLOBAL Chunk*)src);
  }
  const SWAN_GLOBAL char* ip = pg + n8 * PR::VCH * 64 * PR::CB + lane * 8;  // past the values
  const SWAN_GLOBAL char* sp = (const SWAN_GLOBAL char*)kSpareIdx + lane * 8;
#pragma unroll
  for (int g = 0; g < KP8; ++g)
    r.idx[g] = __builtin_nontemporal_load((const SWAN_GLOBAL u32x2*)(g < n8 ? ip + g * 512 : sp));
}
#undef SWAN_GLOBAL

// E4M3 byte `sel` (compile-time after unrolling) of w, as float (exact).  The
// packed conversion decodes bytes 0-1 or 2-3 at once; the two entries of a
// pair call it with the same operands, so it is computed once for both.
__device__ __forceinline__ float e4m3_byte_to_f32(uint32_t w, int sel) {
  typedef float f2 __attribute__((ext_vector_type(2)));
  const f2 v = (sel & 2) ? __builtin_amdgcn_cvt_pk_f32_fp8((int)w, true)
                         : __builtin_amdgcn_cvt_pk_f32_fp8((int)w, false);
  return (sel & 1) ? v.y : v.x;
}

// E4M3 byte `sel` of w as binary16 bits (exact: binary16 holds every E4M3
// value), two bytes per conversion (scale 1)
__device__ __forceinline__ uint32_t e4m3_byte_to_f16_bits(uint32_t w, int sel) {
  typedef _Float16 h2 __attribute__((ext_vector_type(2)));
  const h2 v = (sel & 2) ? __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(w, 1.0f, true)
                         : __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(w, 1.0f, false);
  return (uint32_t)__builtin_bit_cast(uint16_t, (sel & 1) ? v.y : v.x);
}

// value of entry u (0..7) of group g, as float
template <typename T, int KP8>
struct EntryVal {
  __device__ static __forceinline__ float get(const PageRegs<T, KP8>& r, int g, int u) {
    if constexpr (std::is_same<T, E4M3V>::value) {
      const u32x2 c = r.val[g];
      return e4m3_byte_to_f32(u < 4 ? c.x : c.y, u);
    } else if constexpr (sizeof(T) == 2) {
      const u32x4 c = r.val[g];
      const uint32_t w = (u < 2) ? c.x : (u < 4) ? c.y : (u < 6) ? c.z : c.w;
      return f16_bits_to_f32((u & 1) ? (w >> 16) : (w & 0xFFFFu));
    } else {
      const u32x4 c = r.val[g * 2 + (u >> 2)];
      const int v = u & 3;
      const uint32_t w = (v == 0) ? c.x : (v == 1) ? c.y : (v == 2) ? c.z : c.w;
      return __uint_as_float(w);
    }
  }
};

// fp16 bits of entry u of group g (fp16 and E4M3 pages; exact either way)
template <typename T, int KP8>
__device__ __forceinline__ uint32_t entry_f16_bits(const PageRegs<T, KP8>& r, int g, int u) {
  if constexpr (std::is_same<T, E4M3V>::value) {
    const u32x2 c = r.val[g];
    return e4m3_byte_to_f16_bits(u < 4 ? c.x : c.y, u);
  } else {
    const uint32_t w = r.val[g][u >> 1];
    return (u & 1) ? (w >> 16) : (w & 0xFFFFu);
  }
}

template <typename T, int KP8>
__device__ __forceinline__ int entry_idx(const PageRegs<T, KP8>& r, int g, int u) {
  const uint32_t w = (u < 4) ? r.idx[g].x : r.idx[g].y;
  return (int)((w >> (8 * (u & 3))) & 0xFFu);
}

// LDS accesses of one wave execute in program order; this keeps the compiler
// from moving them across the point (no workgroup barrier: waves of one
// workgroup may take different branches).
__device__ __forceinline__ void wave_lds_fence() {
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
}

// ---------------------------------------------------------------------------
// lane-per-token sparse wave: q replicas, scores and the LDS accumulator
// ---------------------------------------------------------------------------
// LDS layouts of one wave (a workgroup is one wave):
//   qrep[dim][8]   the rotated query, 8 copies so that lanes l, l+8, ... of a
//                  half wave spread over the banks
//   acc[dim][64]   accumulators: lane t owns column t, so no two lanes ever
//                  update the same word
constexpr int kQRep = 8;
constexpr int kAccCols = 64;

template <typename T, int KP8>
__device__ __forceinline__ float page_score(const PageRegs<T, KP8>& r, const float* qrep_l) {
  float s0 = 0.f, s1 = 0.f;
#pragma unroll
  for (int g = 0; g < KP8; ++g) {
#pragma unroll
    for (int u = 0; u < 8; u += 2) {
      s0 = fmaf(qrep_l[entry_idx(r, g, u) * kQRep], EntryVal<T, KP8>::get(r, g, u), s0);
      s1 = fmaf(qrep_l[entry_idx(r, g, u + 1) * kQRep], EntryVal<T, KP8>::get(r, g, u + 1), s1);
    }
  }
  return s0 + s1;
}

// acc[idx][lane] += p * v for entries of groups G0 .. G0 + NG - 1 of this
// lane's token.  A token's indices are distinct, so all reads of the chunk can
// be issued before its writes.
template <typename T, int KP8, int G0, int NG>
__device__ __forceinline__ void accumulate_groups(const PageRegs<T, KP8>& r, float* acc_l,
                                                  float p) {
  float a[NG * 8];
#pragma unroll
  for (int g = 0; g < NG; ++g)
#pragma unroll
    for (int u = 0; u < 8; ++u) a[g * 8 + u] = acc_l[entry_idx(r, G0 + g, u) * kAccCols];
#pragma unroll
  for (int g = 0; g < NG; ++g)
#pragma unroll
    for (int u = 0; u < 8; ++u)
      a[g * 8 + u] = fmaf(p, EntryVal<T, KP8>::get(r, G0 + g, u), a[g * 8 + u]);
#pragma unroll
  for (int g = 0; g < NG; ++g)
#pragma unroll
    for (int u = 0; u < 8; ++u) acc_l[entry_idx(r, G0 + g, u) * kAccCols] = a[g * 8 + u];
}

// acc[idx][lane] += p * v for the k entries of this lane's token, in chunks
// of up to 64 entries (one LDS round trip per chunk).
template <typename T, int KP8>
__device__ __forceinline__ void page_accumulate(const PageRegs<T, KP8>& r, float* acc_l, float p,
                                                bool valid) {
  if (!valid) return;
  if constexpr (KP8 <= 8) {
    accumulate_groups<T, KP8, 0, KP8>(r, acc_l, p);
  } else {
    accumulate_groups<T, KP8, 0, 8>(r, acc_l, p);
    accumulate_groups<T, KP8, 8, KP8 - 8>(r, acc_l, p);
  }
}

// acc *= f (the whole accumulator of this wave)
__device__ __forceinline__ void rescale_acc(float* acc, int lane, float f) {
  wave_lds_fence();
#pragma unroll 8
  for (int c = 0; c < kAccCols / 2; ++c) {
    float4* p = (float4*)acc + c * 64 + lane;
    float4 v = *p;
    v.x *= f; v.y *= f; v.z *= f; v.w *= f;
    *p = v;
  }
  wave_lds_fence();
}

// part[4 + r] = the sum over the columns of acc row r; lane owns rows lane and
// lane + 64, its starting chunk staggered per lane to spread the banks
__device__ __forceinline__ void reduce_acc(const float* acc, int lane, float* __restrict__ part) {
  constexpr int kRowChunks = kAccCols / 4;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int r = lane + 64 * h;
    const float4* row = (const float4*)(acc + r * kAccCols);
    float sum = 0.f;
#pragma unroll
    for (int c = 0; c < kRowChunks; ++c) {
      const float4 v = row[(c + lane) & (kRowChunks - 1)];
      sum += (v.x + v.y) + (v.z + v.w);
    }
    part[4 + r] = sum;
  }
}

struct SoftmaxState {
  float m;     // reference maximum (log2 units), wave-uniform
  float l;     // per-lane sum of exp2(s - m)
  bool first;
};

// One wave: the dense buffer of one (sequence, kv head), for one query head.
// Lane t scores buffer token t (a dense 128-dim dot product), then lane l
// accumulates output dims 2l and 2l+1 over all buffer tokens.
template <typename T>
__device__ void buffer_part(const T* kring, const T* vring, int nb, const float* qh, float* qs,
                            float* pb, int lane, float* __restrict__ part) {
  constexpr int E = 16 / (int)sizeof(T);  // elements per 16-byte load
  qs[lane] = qh[lane];
  qs[lane + 64] = qh[lane + 64];
  wave_lds_fence();
  float mloc = -INFINITY;
  for (int t0 = 0; t0 < nb; t0 += 64) {
    const int t = t0 + lane;
    if (t < nb) {
      const u32x4* kr = (const u32x4*)(kring + (int64_t)t * kD);
      float s0 = 0.f, s1 = 0.f;
#pragma unroll 4
      for (int c = 0; c < kD / E; ++c) {
        const u32x4 w = kr[c];
#pragma unroll
        for (int e = 0; e < E; e += 2) {
          const int j = c * E + e;
          if constexpr (sizeof(T) == 2) {
            const uint32_t x = w[e / 2];
            s0 = fmaf(qs[j], f16_bits_to_f32(x & 0xFFFFu), s0);
            s1 = fmaf(qs[j + 1], f16_bits_to_f32(x >> 16), s1);
          } else {
            s0 = fmaf(qs[j], __uint_as_float(w[e]), s0);
            s1 = fmaf(qs[j + 1], __uint_as_float(w[e + 1]), s1);
          }
        }
      }
      const float s = s0 + s1;
      pb[t] = s;
      mloc = fmaxf(mloc, s);
    }
  }
  const float m = wave_max(mloc);
  float lloc = 0.f;
  for (int t0 = 0; t0 < nb; t0 += 64) {
    const int t = t0 + lane;
    if (t < nb) {
      const float p = exp2f(pb[t] - m);
      pb[t] = p;
      lloc += p;
    }
  }
  const float l = wave_sum(lloc);
  wave_lds_fence();
  float a0 = 0.f, a1 = 0.f;
  for (int t = 0; t < nb; ++t) {
    const float p = pb[t];
    const T* vr = vring + (int64_t)t * kD + 2 * lane;
    a0 = fmaf(p, (float)vr[0], a0);
    a1 = fmaf(p, (float)vr[1], a1);
  }
  part[4 + 2 * lane] = a0;
  part[4 + 2 * lane + 1] = a1;
  if (lane == 0) {
    part[0] = m;
    part[1] = l;
  }
}

}  // namespace swan
