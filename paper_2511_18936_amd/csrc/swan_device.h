// Device helpers for the gfx950 kernels: storage-type traits, correctly
// rounded float64 -> storage conversion, wave64 reductions.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace swan {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// ---------------------------------------------------------------------------
// float64 -> IEEE binary16, round to nearest, ties to even, from the bit
// pattern (one rounding step; converting through float32 would round twice).
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint16_t f64_to_f16_bits(double x) {
  const uint64_t bits = (uint64_t)__double_as_longlong(x);
  const uint32_t sign = (uint32_t)(bits >> 48) & 0x8000u;
  const uint64_t a = bits & 0x7FFFFFFFFFFFFFFFull;
  if (a >= 0x7FF0000000000000ull) {  // inf or NaN
    return (uint16_t)(sign | 0x7C00u | (a > 0x7FF0000000000000ull ? 0x0200u : 0u));
  }
  const int e = (int)(a >> 52) - 1023;            // unbiased exponent
  if (e > 15) return (uint16_t)(sign | 0x7C00u);  // >= 65536: overflow to inf
  if (a == 0) return (uint16_t)sign;
  uint64_t m = (a & 0x000FFFFFFFFFFFFFull);
  int shift;
  if ((a >> 52) == 0) {  // float64 subnormal: far below the binary16 range
    return (uint16_t)sign;
  }
  m |= 0x0010000000000000ull;                 // 53-bit significand
  shift = 42 + (e < -14 ? (-14 - e) : 0);     // 52 - 10, plus denormalisation
  if (shift > 63) return (uint16_t)sign;
  const uint64_t q = m >> shift;
  const uint64_t rem = m & ((1ull << shift) - 1);
  const uint64_t half = 1ull << (shift - 1);
  uint64_t r = q + ((rem > half || (rem == half && (q & 1))) ? 1 : 0);
  // normal: exponent field (e + 15) with the implicit bit folded into q
  uint32_t h = (e >= -14) ? (uint32_t)(((e + 14) << 10) + r) : (uint32_t)r;
  if (h >= 0x7C00u) h = 0x7C00u;
  return (uint16_t)(sign | h);
}

// float64 -> binary16 with one correct rounding, through float32: the value
// is first rounded to float32 with round-to-odd (truncate, then set the last
// bit if anything was cut off), which keeps enough information that the final
// hardware float32 -> binary16 round-to-nearest-even equals rounding the
// float64 value directly (float32 has 24 >= 11 + 2 significand bits).
__device__ __forceinline__ uint16_t f64_to_f16_bits_fast(double x) {
  // far below half the smallest binary16 subnormal: signed zero (also keeps
  // float32 denormals, which the hardware may flush, out of the path)
  if (fabs(x) < 0x1p-30) return (uint16_t)((__double_as_longlong(x) >> 48) & 0x8000);
  float y = (float)x;  // round to nearest even
  const double yd = (double)y;
  if (yd != x && !(x != x)) {
    uint32_t yb = __float_as_uint(y);
    // rounded away from zero: step back toward zero (same sign) to truncate
    if (fabs(yd) > fabs(x)) yb -= 1u;
    yb |= 1u;  // sticky bit: inexact
    y = __uint_as_float(yb);
  }
  const _Float16 hv = (_Float16)y;
  return __builtin_bit_cast(uint16_t, hv);
}

__device__ __forceinline__ float f16_bits_to_f32(uint32_t h) {
  _Float16 v = __builtin_bit_cast(_Float16, (uint16_t)h);
  return (float)v;
}

// Storage traits.  `Bits` is the raw integer of one stored element.
template <typename T>
struct Store;

template <>
struct Store<_Float16> {
  using Bits = uint16_t;
  static constexpr int kBytes = 2;
  static constexpr int kMagBits = 15;  // |x| as the low 15 bits, order-preserving
  __device__ static Bits from_f64(double x) { return f64_to_f16_bits(x); }
  __device__ static float to_f32(Bits b) { return f16_bits_to_f32(b); }
  __device__ static uint32_t mag(Bits b) { return (uint32_t)b & 0x7FFFu; }
};

template <>
struct Store<float> {
  using Bits = uint32_t;
  static constexpr int kBytes = 4;
  static constexpr int kMagBits = 31;
  __device__ static Bits from_f64(double x) { return __float_as_uint(__double2float_rn(x)); }
  __device__ static float to_f32(Bits b) { return __uint_as_float(b); }
  __device__ static uint32_t mag(Bits b) { return b & 0x7FFFFFFFu; }
};

// fp16 bits -> OCP FP8 E4M3 (bias 7, no infinities, 0x7f = NaN): nearest
// value, ties to the even code, magnitudes above 448 (and infinities) to 448,
// NaN to NaN, sign kept.  Integer arithmetic only: the fp16 value is
// sig * 2^e2 with an 11-bit significand; the E4M3 quantum at its magnitude is
// 2^eq with eq = max(E, -6) - 3 (E = its binary exponent), so the code is
// (eq + 9) * 8 + round(sig / 2^(eq - e2)) for subnormal and normal results
// alike (a rounding carry moves into the exponent field by itself).
__device__ __forceinline__ uint32_t f16_bits_to_e4m3(uint32_t h) {
  const uint32_t sign = (h >> 8) & 0x80u;
  const uint32_t a = h & 0x7FFFu;
  if (a >= 0x7C00u) return sign | (a > 0x7C00u ? 0x7Fu : 0x7Eu);
  if (a == 0u) return sign;
  const int e16 = (int)(a >> 10);
  const uint32_t sig = e16 ? (a & 0x3FFu) | 0x400u : a;
  const int e2 = (e16 ? e16 : 1) - 25;                  // value = sig * 2^e2
  const int E = (31 - __builtin_clz(sig)) + e2;         // binary exponent
  const int eq = (E > -6 ? E : -6) - 3;                 // log2 of the E4M3 quantum
  const int sh = eq - e2;                               // >= 1 for every fp16 input
  const uint32_t half = 1u << (sh - 1);
  const uint32_t r = (sig + half - 1u + ((sig >> sh) & 1u)) >> sh;  // round half to even
  uint32_t code = (uint32_t)((eq + 9) * 8) + r;
  if (code > 0x7Eu) code = 0x7Eu;                       // saturate at 448
  return sign | code;
}

// Storage formats.  The template argument of the decode and compress kernels
// names the element type of queries, outputs, new keys / values and the dense
// buffer (Elem) and the layout of sparse values: T values in 16-byte chunks of
// 16 / sizeof(T) entries, or, for E4M3V, one-byte E4M3 values in 8-byte chunks
// of 8 entries (with fp16 everywhere else).
struct E4M3V {};

template <typename T>
struct Fmt {
  using Elem = T;
  static constexpr int kValBytes = (int)sizeof(T);
  static constexpr int kChunkBytes = 16;
};
template <>
struct Fmt<E4M3V> {
  using Elem = _Float16;
  static constexpr int kValBytes = 1;
  static constexpr int kChunkBytes = 8;
};

// ---------------------------------------------------------------------------
// wave64 helpers
// ---------------------------------------------------------------------------
// wave64 reductions with DPP row shifts and row broadcasts (no LDS traffic);
// the result is read from lane 63 and returned to every lane
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}

__device__ __forceinline__ float wave_max(float v) {
  // identity -inf for lanes whose DPP source is out of the row
  auto mx = [](float x, float y) { return fmaxf(x, y); };
  v = mx(v, __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(-INFINITY),
                                                       __float_as_int(v), 0x111, 0xF, 0xF, false)));
  v = mx(v, __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(-INFINITY),
                                                       __float_as_int(v), 0x112, 0xF, 0xF, false)));
  v = mx(v, __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(-INFINITY),
                                                       __float_as_int(v), 0x114, 0xF, 0xF, false)));
  v = mx(v, __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(-INFINITY),
                                                       __float_as_int(v), 0x118, 0xF, 0xF, false)));
  v = mx(v, __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(-INFINITY),
                                                       __float_as_int(v), 0x142, 0xA, 0xF, false)));
  v = mx(v, __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(-INFINITY),
                                                       __float_as_int(v), 0x143, 0xC, 0xF, false)));
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
}

__device__ __forceinline__ float wave_sum(float v) {
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x111, 0xF, 0xF, false));
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x112, 0xF, 0xF, false));
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x114, 0xF, 0xF, false));
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x118, 0xF, 0xF, false));
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x142, 0xA, 0xF, false));
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x143, 0xC, 0xF, false));
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
}

__device__ __forceinline__ int lane_id() { return (int)__lane_id(); }

// number of set bits of `mask` in lanes strictly below this one
__device__ __forceinline__ int popc_below(uint64_t mask) {
  return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                        __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

}  // namespace swan
