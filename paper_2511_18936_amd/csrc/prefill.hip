// Compress-append of many tokens at once (prefill), fp16 storage (sparse
// values fp16 or E4M3).
//
// Same result as token-by-token Algorithm 1 (and as insert_kernel): each new
// key/value x is rotated, x_hat = x . P, and the exact x_hat is rounded once to
// fp16; tokens that stay in the buffer go to their ring slot, the others are
// pruned to their top-k magnitudes (ties: lower index) and packed.
//
// The rotation runs on int8 MFMA (v_mfma_i32_16x16x64_i8) with exact integer
// arithmetic.  Each token row is a fixed-point integer X (30 bits below a
// power of two above the row's largest magnitude) and P a fixed-point integer
// Y (38 bits below a power of two above its largest entry), each split into
// balanced base-256 digits (4 for X, 5 for Y, every digit in [-128, 127]).
// The digit products are accumulated exactly in int32, one accumulator per
// digit weight; the 17 digit pairs whose weight is within 5 digits of the top
// give x_hat up to a bounded remainder: the 3 dropped pairs (below 2^-38 of
// the two powers of two's product), plus the truncation of tiny entries of x
// (counted per row) or of P (bounded per column).  Each
// element is rounded to fp16 in two ways that must agree: both ends of its
// error interval (widened by the float64 and float32 roundings) are rounded
// through float32; about 7 elements in 10^4 disagree and get an exact
// certification in float64 (no fp16 rounding boundary within the bound of the
// computed value), and the few that fail that are recomputed in float64 from
// x and P.  Either way the stored value is the exact x_hat rounded once to
// fp16.
//
// A workgroup of 4 waves serves one (sequence, kv head, role): it first
// writes P's digits, in the MFMA operand layout, to LDS (80 KiB), then each
// wave handles its own 64-position blocks, one wave per SIMD:
//   rotation   per pair of 16-token tiles (their x rows loaded one pair
//              ahead): x digits in registers (A operands); 16 steps (16
//              output dims x 64 input dims) of 34 MFMAs on P digits read
//              from LDS one step ahead (B operands), issued in four parts,
//              each interleaved with the VALU work of one element of the
//              previous tile's conversion into the LDS row of its token
//   selection  one token per lane on its 128 stored values: a radix select
//              on bit planes of the magnitudes finds the kept dims (a 128-bit
//              mask; ties at the k-th largest to the lower dim)
//   output     each lane walks its kept dims in ascending order, 8 per page
//              chunk, reads their values from its LDS row and stores its page
//              slot chunk by chunk (a wave store is 1 KiB contiguous), or its
//              dense row to the ring
#include <type_traits>

#include "swan_device.h"
#include "swan_internal.h"

namespace swan {

typedef int32_t i32x4 __attribute__((ext_vector_type(4)));
typedef uint16_t u16x2 __attribute__((ext_vector_type(2)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));

constexpr int kRowHalves = 136;                // LDS row of one token's 128 fp16 values (+ pad)
constexpr int kPrefillBlocksPerWave = 8;       // 64-position blocks per wave
constexpr int kPrefillWaves = 4;               // waves per workgroup, sharing P's digits
constexpr int kXcds = 8;                       // MI355X: 8 XCDs, each with its own L2
constexpr int kStageBytes = 64 * kRowHalves * 2;  // the rows of one wave
// digit arithmetic of the rotation
constexpr int kXDigits = 4;                    // x: balanced base-256 digits
constexpr int kPDigits = 5;                    // P: balanced base-256 digits
constexpr int kXFix = 8 * kXDigits - 2;        // |X| < 2^30
constexpr int kPFix = 8 * kPDigits - 2;        // |Y| < 2^38
constexpr int kTopLevel = 5;                   // digit pairs (s, t) with s + t <= 5 ...
constexpr int kLevels = kTopLevel + 1;         // ... accumulated per weight s + t
// The 3 dropped pairs, (2,4) and (3,3) of weight 2^8 and (3,4) of weight 1 in
// units of the lowest digit product: each sums 128 products of at most 2^14.
constexpr double kDroppedUnits = (2.0 * 256.0 + 1.0) * 128.0 * 16384.0;
constexpr int kBDigBytes = 8 * 2 * kPDigits * 1024;   // [out tile][k step][digit][lane][16 B]
constexpr int kPrefillLds = kBDigBytes + kPrefillWaves * kStageBytes + 128 * 4 + 64;
constexpr uint16_t kUncertain = 0xFFFFu;       // a NaN pattern: never a rounded x_hat

// One step of a 16x16 bit-matrix transpose applied to both 16-bit halves of
// 16 words at once (row i of each matrix = half of w[i], column b = bit b):
// the k x k off-diagonal blocks of every 2k x 2k block trade places.
template <int K>
__device__ __forceinline__ void transpose_step(uint32_t* w, uint32_t mask) {
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    if (i & K) continue;
    const uint32_t t = ((w[i] >> K) ^ w[i + K]) & mask;
    w[i + K] ^= t;
    w[i] ^= t << K;
  }
}

// Bits 0-15 of a bit-plane word stand for a chunk's even dims, bits 16-31 for
// its odd ones; this puts them in dim order (bit i = dim 32 c + i).
__device__ __forceinline__ uint32_t spread16(uint32_t x) {
  x = (x | (x << 8)) & 0x00FF00FFu;
  x = (x | (x << 4)) & 0x0F0F0F0Fu;
  x = (x | (x << 2)) & 0x33333333u;
  return (x | (x << 1)) & 0x55555555u;
}
__device__ __forceinline__ uint32_t dim_order(uint32_t w) {
  return spread16(w & 0xFFFFu) | (spread16(w >> 16) << 1);
}

// The k dims kept from the 128 fp16 magnitudes in v (two per dword): the k
// largest, ties at the k-th largest to the lower dim, as a 128-bit mask in dim
// order.  Radix select on bit planes: the magnitudes of each 32-element chunk
// c are transposed so that pl[b][c] holds bit b of each element (bits 0-15:
// the chunk's even elements, 16-31: its odd ones); from the top bit down, the
// candidates still equal to the threshold prefix are split by the next bit,
// and those above it are collected.
__device__ __forceinline__ void kept_dims(const uint32_t* v, int k, uint32_t* kept) {
  uint32_t pl[15][4];
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    uint32_t w[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) w[i] = v[16 * c + i] & 0x7FFF7FFFu;
    transpose_step<8>(w, 0x00FF00FFu);
    transpose_step<4>(w, 0x0F0F0F0Fu);
    transpose_step<2>(w, 0x33333333u);
    transpose_step<1>(w, 0x55555555u);
#pragma unroll
    for (int b = 0; b < 15; ++b) pl[b][c] = w[b];  // plane 15 (the sign) is zero
  }
  uint32_t eq[4] = {~0u, ~0u, ~0u, ~0u}, gt[4] = {0u, 0u, 0u, 0u};
  int ngt = 0;
#pragma unroll
  for (int b = 14; b >= 0; --b) {
    uint32_t hi[4];
    int cnt = 0;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      hi[c] = eq[c] & pl[b][c];
      cnt += __popc(hi[c]);
    }
    const bool one = ngt + cnt >= k;  // the k-th largest has this bit set
    ngt += one ? 0 : cnt;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      gt[c] |= one ? 0u : hi[c];
      eq[c] = one ? hi[c] : (eq[c] & ~pl[b][c]);
    }
  }
  // eq: the elements equal to the k-th largest; k - ngt of them are kept,
  // lowest dims first
  int need = k - ngt;
  int neq = 0;
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    eq[c] = dim_order(eq[c]);
    neq += __popc(eq[c]);
  }
  if (neq > need) {  // ties: keep the lowest need of them
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      uint32_t keep = 0u, rest = eq[c];
      while (need > 0 && rest != 0u) {
        keep |= rest & (0u - rest);
        rest &= rest - 1u;
        --need;
      }
      eq[c] = keep;
    }
  }
#pragma unroll
  for (int c = 0; c < 4; ++c) kept[c] = dim_order(gt[c]) | eq[c];
}

// The lowest set dim of the 128-bit mask (lo: dims 0-63, hi: 64-127), cleared;
// branch-free.
__device__ __forceinline__ uint32_t pop_lowest(uint64_t& lo, uint64_t& hi) {
  const bool in_lo = lo != 0ull;
  const uint64_t m = in_lo ? lo : hi;
  const uint32_t d = (uint32_t)__builtin_ctzll(m) + (in_lo ? 0u : 64u);
  const uint64_t rest = m & (m - 1ull);
  lo = in_lo ? rest : lo;
  hi = in_lo ? hi : rest;
  return d;
}

// One token per lane: its page slot, written to global memory chunk by chunk
// (a wave's chunk store is 1 KiB, or 512 B, contiguous).  Entries 0..k-1 are
// the kept dims in ascending order with their values, read from the lane's
// LDS row; entries k..kp-1 the padding, value +0 at the lowest dims not kept.
// Per chunk the 8 dims are found first, then their 8 values read together;
// the padding lies in the last chunk (kp - k < 8).
template <typename F>
__device__ __forceinline__ void store_slot(const uint16_t* row, const uint32_t* kept, int k,
                                           int kp, char* page, int lane) {
  constexpr int VB = Fmt<F>::kValBytes;
  constexpr bool kE4M3 = std::is_same<F, E4M3V>::value;
  uint64_t klo = kept[0] | ((uint64_t)kept[1] << 32), khi = kept[2] | ((uint64_t)kept[3] << 32);
  uint64_t flo = ~klo, fhi = ~khi;
  char* ipage = page + 64 * kp * VB;
  for (int c = 0; c < kp / 8; ++c) {
    // kept entries in this chunk (uniform): 8 but in the last chunk, which
    // also holds the padding when k is not a multiple of 8
    const int nk = min(k - 8 * c, 8);
    uint32_t d[8], hb[8];
    if (nk == 8) {
#pragma unroll
      for (int q = 0; q < 8; ++q) d[q] = pop_lowest(klo, khi);
    } else {
#pragma unroll
      for (int q = 0; q < 8; ++q) d[q] = q < nk ? pop_lowest(klo, khi) : pop_lowest(flo, fhi);
    }
#pragma unroll
    for (int q = 0; q < 8; ++q) hb[q] = row[d[q] & 127u];
    uint32_t val[4] = {0u, 0u, 0u, 0u}, idx[2] = {0u, 0u};
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const uint32_t h = q < nk ? hb[q] : 0u;
      idx[q >> 2] |= d[q] << (8 * (q & 3));
      if constexpr (kE4M3)
        val[q >> 2] |= f16_bits_to_e4m3(h) << (8 * (q & 3));
      else
        val[q >> 1] |= h << (16 * (q & 1));
    }
    if constexpr (kE4M3)
      *(u32x2*)(page + c * 512 + lane * 8) = u32x2{val[0], val[1]};
    else
      *(u32x4*)(page + c * 1024 + lane * 16) = u32x4{val[0], val[1], val[2], val[3]};
    *(u32x2*)(ipage + c * 512 + lane * 8) = u32x2{idx[0], idx[1]};
  }
}

// v_perm_b32: byte i of the result is byte sel_i of the 8 bytes {hi : lo}
__device__ __forceinline__ uint32_t perm(uint32_t hi, uint32_t lo, uint32_t sel) {
  return __builtin_amdgcn_perm(hi, lo, sel);
}

// The balanced base-256 digits of four fixed-point values, as four int8 words
// (digit 0 = the top one).  yb = X + 0x808080: its low three bytes are the low
// digits plus 128, its top byte the top digit (two's complement).
__device__ __forceinline__ void digit_words(uint32_t a, uint32_t b, uint32_t c, uint32_t d,
                                            uint32_t* w) {
  const uint32_t ab_lo = perm(b, a, 0x05010400u), ab_hi = perm(b, a, 0x07030602u);
  const uint32_t cd_lo = perm(d, c, 0x05010400u), cd_hi = perm(d, c, 0x07030602u);
  w[3] = perm(cd_lo, ab_lo, 0x05040100u) ^ 0x80808080u;
  w[2] = perm(cd_lo, ab_lo, 0x07060302u) ^ 0x80808080u;
  w[1] = perm(cd_hi, ab_hi, 0x05040100u) ^ 0x80808080u;
  w[0] = perm(cd_hi, ab_hi, 0x07060302u);
}

// fixed-point value of one fp16 element: trunc(x * 2^shift) + 0x808080
__device__ __forceinline__ uint32_t fixed_biased(uint32_t hbits, int shift) {
  const float f = f16_bits_to_f32(hbits);
  return (uint32_t)(int32_t)__builtin_ldexpf(f, shift) + 0x00808080u;
}

// The fp16 rounding of a value y known to within E: y's own rounding when no
// fp16 rounding boundary lies within E of it, else kUncertain.  Branch-free:
// y is rounded to float32 with round-to-odd (round to nearest, then back
// toward zero and the last bit set when that was inexact), which keeps the
// information that the hardware float32 -> fp16 rounding needs to round y
// itself correctly; the distance to the boundary is measured in float64.
__device__ __forceinline__ uint32_t certified_f16(double y, double E) {
  const float yn = (float)y;
  const double back = (double)yn;
  const bool inexact = back != y;
  const bool away = fabs(back) > fabs(y);
  float y32 = __uint_as_float((__float_as_uint(yn) - (inexact && away ? 1u : 0u)) |
                              (inexact ? 1u : 0u));
  asm("" : "+v"(y32));  // two hardware conversions, not one software f64 -> f16
  const uint32_t hb = (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)y32);
  const uint32_t ex = (hb >> 10) & 31u;
  const double hd = (double)f16_bits_to_f32(hb);
  const double dist = fabs(y - hd);  // exact
  // half the spacing of fp16 values at hb on y's side: below a power of two the
  // spacing halves.  (E < half / 2 keeps the other side's boundary out of reach
  // too.)
  const double half = ex ? __builtin_ldexp(1.0, (int)ex - 26) : 0x1p-25;
  const bool below_pow2 = (hb & 0x3FFu) == 0u && ex > 1u && fabs(y) < fabs(hd);
  const double side = below_pow2 ? 0.5 * half : half;
  const bool ok = (ex != 31u) & (dist + E + fabs(y) * 0x1p-50 < side) & (E < 0.25 * half);
  return ok ? hb : kUncertain;
}

// x rounded to float32 and that rounded to fp16, both by the hardware (the
// empty asm keeps the compiler from fusing them into one software f64 -> f16
// conversion)
__device__ __forceinline__ uint32_t f16_via_f32(double x) {
  float f = (float)x;
  asm("" : "+v"(f));
  return (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)f);
}

__device__ __forceinline__ double wave_sum_f64(double v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

template <typename F>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1)))
void prefill_kernel(CompressLaunch a) {
  constexpr int VB = Fmt<F>::kValBytes, CB = Fmt<F>::kChunkBytes;
  extern __shared__ __attribute__((aligned(16))) char lds_all[];
  char* bdig = lds_all;
  float* colDY = (float*)(lds_all + kBDigBytes + kPrefillWaves * kStageBytes);  // [128]
  float* wgred = colDY + 128;                                                  // [4]
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  char* lds = lds_all + kBDigBytes + wave * kStageBytes;  // this wave's rows / page copy
  _Float16* rows = (_Float16*)lds;  // [64 tokens][kRowHalves]
  const int m16 = lane & 15, g4 = lane >> 4;
  // grid: (b, h, role, block group)
  // Workgroups go to the 8 XCDs round-robin by id, so XCD id % 8 gets the
  // (head, role) pairs u = xcd, xcd + 8, ...: its L2 then holds 1/8 of the P
  // matrices instead of all of them.  Pairs are padded to a multiple of 8.
  const int xcd = blockIdx.x % kXcds;
  int w = blockIdx.x / kXcds;
  const int ngrp = a.prefill_groups;
  const int grp = w % ngrp;
  w /= ngrp;
  const int b = w % a.B;
  const int u = xcd + kXcds * (w / a.B);  // (head, role) pair
  if (u >= 2 * a.Hkv) return;
  const int h = u >> 1;
  const int role = u & 1;
  const int len_old = a.tab.len[b];
  const int nnew = a.tab.nnew[b];
  if (nnew <= 0) return;
  const int len_new = len_old + nnew;
  const int blk0 = len_old / kPage;
  const int blk1 = (len_new - 1) / kPage;  // inclusive
  if (blk0 + grp * kPrefillWaves * kPrefillBlocksPerWave > blk1) return;  // uniform

  const _Float16* x = (const _Float16*)(role ? a.v_new : a.k_new) +
                      ((int64_t)b * a.Hkv + h) * a.n_new * kD;
  // NULL P_vo: values already in the rotated basis, stored as given
  const float* Prole = role ? a.P_vo : a.P_qk;
  const float* P = Prole ? Prole + (int64_t)h * kD * kD : nullptr;

  // ---- P's digits (once per workgroup) ----
  int G = 0;         // Y = trunc(P * 2^G), |Y| < 2^38
  float pmax = 0.f;  // largest |P|
  if (P) {
    float pm = 0.f;
    for (int r = 0; r < kD * kD / 256; ++r) pm = fmaxf(pm, fabsf(P[tid + 256 * r]));
    pm = wave_max(pm);
    if (lane == 0) wgred[wave] = pm;
    if (tid < kD) colDY[tid] = 0.f;
    __syncthreads();
    pmax = fmaxf(fmaxf(wgred[0], wgred[1]), fmaxf(wgred[2], wgred[3]));
    int pe = 0;
    if (pmax > 0.f) (void)__builtin_frexpf(pmax, &pe);  // pmax < 2^pe
    G = kPFix - pe;
    // vector v: 16 entries P[k][col], k = 64 ks + 16 g + j, as the 16 bytes of
    // lane (col % 16) + 16 g of the B operand of output tile col / 16, step ks
    for (int r = 0; r < 4; ++r) {
      const int v = tid + 256 * r;
      const int n = v & 15, g = (v >> 4) & 3, ks = (v >> 6) & 1, o = v >> 7;
      const int col = 16 * o + n;
      uint32_t dw[kPDigits][4] = {};
      double dy = 0.0;
      for (int j = 0; j < 16; ++j) {
        const double p = (double)P[(64 * ks + 16 * g + j) * kD + col];
        double yv = trunc(__builtin_ldexp(p, G));
        dy = fmax(dy, fabs(p - __builtin_ldexp(yv, -G)));  // exact
        for (int t = kPDigits - 1; t >= 1; --t) {
          const double q = floor((yv + 128.0) * (1.0 / 256.0));
          const int dgt = (int)(yv - 256.0 * q);  // in [-128, 127]
          dw[t][j >> 2] |= ((uint32_t)dgt & 0xFFu) << (8 * (j & 3));
          yv = q;
        }
        dw[0][j >> 2] |= ((uint32_t)(int)yv & 0xFFu) << (8 * (j & 3));  // |top| <= 64
      }
      for (int t = 0; t < kPDigits; ++t)
        *(u32x4*)(bdig + ((o * 2 + ks) * kPDigits + t) * 1024 + (n + 16 * g) * 16) =
            u32x4{dw[t][0], dw[t][1], dw[t][2], dw[t][3]};
      uint32_t dyb = __float_as_uint((float)dy);  // rounded up: a bound
      if ((double)__uint_as_float(dyb) < dy) dyb += 1u;
      atomicMax((unsigned int*)&colDY[col], dyb);
    }
    __syncthreads();
  }

  const int k = a.tab.kact[role][b];
  const int kp = kpad_of(k);
  const int64_t pbytes = page_bytes_of(VB, k);
  char* pages = (char*)(role ? a.v_pages : a.k_pages) + a.tab.page_off[role][b] +
                (int64_t)h * a.n_pages_cap * pbytes;
  uint16_t* ring = (uint16_t*)(role ? a.v_ring : a.k_ring) + ((int64_t)b * a.Hkv + h) * a.bb * kD;
  const int bbeg = blk0 + (grp * kPrefillWaves + wave) * kPrefillBlocksPerWave;
  const int bend = min(bbeg + kPrefillBlocksPerWave, blk1 + 1);

  // The x rows of a pair of 16-token tiles (lane (m16, g4): token 16 (2 tp +
  // T) + m16, dims 64 ks + 16 g4 + j), zero past the wave's blocks and the new
  // tokens.  They are loaded one tile pair ahead of their use.
  auto load_x = [&](int blk_, int tp_, u32x4 (&xv)[2][2][2]) {
#pragma unroll
    for (int T = 0; T < 2; ++T) {
      const int t = blk_ * kPage + 16 * (2 * tp_ + T) + m16 - len_old;
      if (blk_ < bend && t >= 0 && t < nnew) {
        const u32x4* src = (const u32x4*)(x + (int64_t)t * kD + 16 * g4);
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
          xv[T][ks][0] = src[8 * ks];
          xv[T][ks][1] = src[8 * ks + 1];
        }
      } else {
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) xv[T][ks][0] = xv[T][ks][1] = u32x4{0u, 0u, 0u, 0u};
      }
    }
  };
  u32x4 xnext[2][2][2];
  if (P) load_x(bbeg, 0, xnext);

  for (int blk = bbeg; blk < bend; ++blk) {
    const int pos0 = blk * kPage;
    bool uncertain = false;  // some element of the block needs the float64 path
    if (P) {
      // ---- rotation: two 16-token tiles at a time ----
#pragma unroll 1
      for (int tp = 0; tp < 2; ++tp) {
        i32x4 A[2][2][kXDigits];  // [tile][k step][digit]
        float Eb[2][4];           // per token of the result rows: bound without the P term
        float Ey[2][4];           // factor of the column's P truncation term
        int sx[2][4];             // y = H * 2^sx
        u32x4 xcur[2][2][2];
#pragma unroll
        for (int T = 0; T < 2; ++T)
#pragma unroll
          for (int ks = 0; ks < 2; ++ks) {
            xcur[T][ks][0] = xnext[T][ks][0];
            xcur[T][ks][1] = xnext[T][ks][1];
          }
        load_x(tp ? blk + 1 : blk, tp ^ 1, xnext);
#pragma unroll
        for (int T = 0; T < 2; ++T) {
          const u32x4 (&xv)[2][2] = xcur[T];
          // the row's largest magnitude (fp16 bits), the sum of its magnitudes
          // and the smallest |x| - 1 (as 16-bit integers, so that 0 wraps to
          // the largest), two elements per instruction
          u16x2 mx2 = {0, 0}, tm2 = {0xFFFF, 0xFFFF};
          float l1 = 0.f;
#pragma unroll
          for (int ks = 0; ks < 2; ++ks)
#pragma unroll
            for (int c = 0; c < 2; ++c)
#pragma unroll
              for (int q = 0; q < 4; ++q) {
                const uint32_t wa = xv[ks][c][q] & 0x7FFF7FFFu;
                const u16x2 a2 = __builtin_bit_cast(u16x2, wa);
                mx2 = __builtin_elementwise_max(mx2, a2);
                tm2 = __builtin_elementwise_min(tm2, a2 - (u16x2){1, 1});
                l1 = __builtin_amdgcn_fdot2(__builtin_bit_cast(f16x2, wa), (f16x2){1, 1}, l1, false);
              }
          uint32_t mx = max((uint32_t)mx2.x, (uint32_t)mx2.y);
          uint32_t tm = min((uint32_t)tm2.x, (uint32_t)tm2.y);
          mx = max(mx, (uint32_t)__shfl_xor((int)mx, 16));
          mx = max(mx, (uint32_t)__shfl_xor((int)mx, 32));
          tm = min(tm, (uint32_t)__shfl_xor((int)tm, 16));
          tm = min(tm, (uint32_t)__shfl_xor((int)tm, 32));
          l1 += __shfl_xor(l1, 16);
          l1 += __shfl_xor(l1, 32);
          // max|x| < 2^e
          const int e = mx == 0u ? 0
                        : (mx >> 10) ? (int)(mx >> 10) - 14
                                     : 8 - __builtin_clz(mx);  // (32 - clz) - 24
          const int shift = kXFix - e;
          // |x| >= 2^(e - 20) is exact in 30 bits below 2^e; each smaller nonzero
          // element is truncated by less than 2^(e - 30): count them (rare: only
          // when the smallest nonzero |x| is below thr).  thr: the fp16 bits of
          // 2^(e - 20), or 0 below the fp16 range (none truncated)
          const int te = e - kXFix + 10;
          const uint32_t thr = te >= -14 ? (uint32_t)(te + 15) << 10
                               : te >= -24 ? 1u << (te + 24) : 0u;
          int ntr = 0;
          if (__ballot(thr != 0u && tm < thr - 1u) != 0ull) {
#pragma unroll
            for (int ks = 0; ks < 2; ++ks)
#pragma unroll
              for (int c = 0; c < 2; ++c)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                  const uint32_t wv = xv[ks][c][q];
                  ntr += ((wv & 0x7FFFu) - 1u < thr - 1u) ? 1 : 0;  // 0 < |x| < 2^(e - 20)
                  ntr += (((wv >> 16) & 0x7FFFu) - 1u < thr - 1u) ? 1 : 0;
                }
            ntr += __shfl_xor(ntr, 16);
            ntr += __shfl_xor(ntr, 32);
          }
#pragma unroll
          for (int ks = 0; ks < 2; ++ks) {
            uint32_t dg[kXDigits][4];
#pragma unroll
            for (int c = 0; c < 2; ++c)
#pragma unroll
              for (int q2 = 0; q2 < 2; ++q2) {
                // values 8 c + 4 q2 .. + 3
                const uint32_t w0 = xv[ks][c][2 * q2], w1 = xv[ks][c][2 * q2 + 1];
                uint32_t wd[kXDigits];
                digit_words(fixed_biased(w0 & 0xFFFFu, shift), fixed_biased(w0 >> 16, shift),
                            fixed_biased(w1 & 0xFFFFu, shift), fixed_biased(w1 >> 16, shift), wd);
#pragma unroll
                for (int s = 0; s < kXDigits; ++s) dg[s][2 * c + q2] = wd[s];
              }
#pragma unroll
            for (int s = 0; s < kXDigits; ++s)
              A[T][ks][s] = i32x4{(int)dg[s][0], (int)dg[s][1], (int)dg[s][2], (int)dg[s][3]};
          }
          // the bound's row terms, for the result lanes: token tok's scale,
          // dropped-pair bound and truncated-x bound
          // (float32, rounded up: the factors 1 + 2^-15 leave room for that
          // rounding, for the float32 additions of l1 (128 terms) and for the
          // rounding of the float32 fma that combines them per element)
          const int sxe = 16 + e - kXFix - G;
          const float eb = (float)(kDroppedUnits * __builtin_ldexp(1.0, e - kXFix - G) +
                                   (double)ntr * (double)pmax * __builtin_ldexp(1.0, e - kXFix)) *
                           (1.0f + 0x1p-15f);
          // sum |x_i|
          const float ey = l1 * (1.0f + 0x1p-14f);
          // move them to the lanes holding the token's results: row r = 4 g + v
          // of the tile is token m16 = r of the tile
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const int src_lane = 4 * g4 + v;  // lane (m16 = 4 g4 + v, g4 = 0) has token 4 g4 + v
            sx[T][v] = __shfl(sxe, src_lane);
            Eb[T][v] = __shfl(eb, src_lane);
            Ey[T][v] = __shfl(ey, src_lane);
          }
        }
        // ---- MFMA per 16 output dims, then certified fp16 values to the rows;
        //      the results of tile o are turned into fp16 while the MFMAs of
        //      tile o + 1 run (the loop is unrolled so that one scheduling
        //      region holds both) ----
        // step j = 2 o + ks: output tile o, k step ks.  The P digits of a step
        // are read from LDS into registers one step ahead of their MFMAs.
        auto load_b = [&](int j, i32x4 (&B)[kPDigits]) {
#pragma unroll
          for (int t = 0; t < kPDigits; ++t)
            B[t] = *(const i32x4*)(bdig + (j * kPDigits + t) * 1024 + lane * 16);
        };
        // the 17 digit pairs (s, t), s + t <= 5, of one tile in s-major order;
        // a step issues them for tile 0 then tile 1, in four parts of 9, 8, 9
        // and 8 MFMAs (part q: tile q / 2, pairs 9 (q % 2) ..)
        auto mfma_part = [&](int j, i32x4 (&acc)[2][kLevels], const i32x4 (&B)[kPDigits],
                             int q) {
          const int ks = j & 1, T = q >> 1;
          int n = 0;
#pragma unroll
          for (int s = 0; s < kXDigits; ++s)
#pragma unroll
            for (int t = 0; t < kPDigits; ++t)
              if (s + t <= kTopLevel) {
                if ((n < 9) == ((q & 1) == 0))
                  acc[T][s + t] = __builtin_amdgcn_mfma_i32_16x16x64_i8(A[T][ks][s], B[t],
                                                                        acc[T][s + t], 0, 0, 0);
                ++n;
              }
        };
        auto zero_acc = [&](i32x4 (&acc)[2][kLevels]) {
#pragma unroll
          for (int T = 0; T < 2; ++T)
#pragma unroll
            for (int l = 0; l < kLevels; ++l) acc[T][l] = i32x4{0, 0, 0, 0};
        };
        // result layout: register v of lane l is row 4 (l / 16) + v (token),
        // column l % 16 (output dim 16 o + l % 16).
        // H = sum_l C_l 256^(5 - l), combined as ((t01 2^16 + t23) 2^16 + t45)
        // with t01 = C_0 256 + C_1 etc. exact in int32: a top digit of x or P
        // lies in [-64, 64], so over 128 products |C_0| <= 2^19, |C_1| <= 2^21,
        // |C_2| <= 2^22, |C_3| <= 3 * 2^21, |C_4| <= 7 * 2^20, |C_5| <= 3 * 2^21.
        // The float64 sums are exact below 2^53, else within 2^-53 |H|.
        auto result = [&](const i32x4 (&acc)[2][kLevels], int T, int v) {
          const int t01 = acc[T][0][v] * 256 + acc[T][1][v];
          const int t23 = acc[T][2][v] * 256 + acc[T][3][v];
          const int t45 = acc[T][4][v] * 256 + acc[T][5][v];
          const double H = fma(fma((double)t01, 65536.0, (double)t23), 65536.0, (double)t45);
          return __builtin_ldexp(H, sx[T][v]);
        };
        // Fast check: both ends of [y - E1, y + E1], E1 = E + 2^-22 |y|,
        // rounded to fp16 through float32.  The margin 2^-22 |y| covers the
        // float64 and float32 roundings of the ends, so the two conversions
        // bracket every value within E of y; rounding is monotone, so when
        // they agree that is the fp16 rounding of x_hat.  Elements whose ends
        // disagree (about 1 in 10^3) get the exact certification.  One half
        // (4 tokens) of tile o per call; returns the open elements as bits.
        // (one element: register v of a lane's half tile, dyc the P truncation
        // bound of its column; true when open)
        auto to_row = [&](int o, int T, const i32x4 (&acc)[2][kLevels], int v, float dyc) {
          const int col = 16 * o + m16;
          const double y = result(acc, T, v);
          const double E1 = fma(fabs(y), 0x1p-22, (double)fmaf(dyc, Ey[T][v], Eb[T][v]));
          const uint32_t lo = f16_via_f32(y - E1), hi = f16_via_f32(y + E1);
          const int tok = 16 * (2 * tp + T) + 4 * g4 + v;
          ((uint16_t*)rows)[tok * kRowHalves + col] = (uint16_t)lo;
          return lo != hi;
        };
        // the exact certification of the elements the fast check left open
        auto fix_rows = [&](int o, int T, const i32x4 (&acc)[2][kLevels], const bool (&need)[4]) {
          const int col = 16 * o + m16;
          const float dyc = colDY[col];
#pragma unroll
          for (int v = 0; v < 4; ++v)
            if (need[v]) {
              const double y = result(acc, T, v);
              const double E = (double)fmaf(dyc, Ey[T][v], Eb[T][v]);
              const uint32_t hb = certified_f16(y, E);
              uncertain |= hb == kUncertain;
              const int tok = 16 * (2 * tp + T) + 4 * g4 + v;
              ((uint16_t*)rows)[tok * kRowHalves + col] = (uint16_t)hb;
            }
        };
        // 16 steps j = 2 o + ks (+ two to drain): step j reads the P bound of
        // the column it converts, issues the LDS reads of step j + 1's P
        // digits, then its 34 MFMAs in four parts, each part
        // followed by one element of half a tile of tile o - 1's conversion;
        // the scheduling barriers interleave a part's MFMAs with that
        // element's VALU work (4 instructions after each MFMA) and keep the
        // parts apart, so the conversion runs while the MFMAs do.
        i32x4 acc[2][2][kLevels];
        i32x4 Bq[2][kPDigits];
        load_b(0, Bq[0]);
#pragma unroll
        for (int j = 0; j < 18; ++j) {
          const int o = j >> 1, ks = j & 1;
          const float dyc = j >= 2 ? colDY[16 * (o - 1) + m16] : 0.f;
          if (j + 1 < 16) load_b(j + 1, Bq[(j + 1) & 1]);
          if (j < 16 && ks == 0) zero_acc(acc[o & 1]);
          bool need[4] = {false, false, false, false};
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            if (j < 16) mfma_part(j, acc[o & 1], Bq[j & 1], q);
            if (j >= 2) need[q] = to_row(o - 1, ks, acc[(o - 1) & 1], q, dyc);
            if (q == 0) {  // DS reads: the column bound, then the next step's P digits
              if (j >= 2 && j + 1 < 16)
                __builtin_amdgcn_sched_group_barrier(0x100, kPDigits + 1, 0);
              else if (j + 1 < 16)
                __builtin_amdgcn_sched_group_barrier(0x100, kPDigits, 0);
              else
                __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
            }
            if (j < 16) {
#pragma unroll
              for (int i = 0; i < 9 - (q & 1); ++i) {
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
                __builtin_amdgcn_sched_group_barrier(0x002, 4, 0);  // VALU
              }
            }
            __builtin_amdgcn_sched_barrier(0);
          }
          if (j >= 2 && __ballot(need[0] | need[1] | need[2] | need[3]) != 0u)
            fix_rows(o - 1, ks, acc[(o - 1) & 1], need);
        }
      }
    } else {
      // values given in the rotated basis: the rows are the input
      const int t = pos0 + lane - len_old;
      u32x4* dst = (u32x4*)(rows + lane * kRowHalves);
      if (t >= 0 && t < nnew) {
        const u32x4* src = (const u32x4*)(x + (int64_t)t * kD);
#pragma unroll
        for (int c = 0; c < 16; ++c) dst[c] = src[c];
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();
    if (__ballot(uncertain) != 0) {
      // The rare uncertain elements: x_hat in float64 over the input row and P,
      // rounded once.  The wave takes them one at a time, each lane summing the
      // products of two input dims.
      const int t = pos0 + lane - len_old;
      uint16_t* myrow = (uint16_t*)(rows + lane * kRowHalves);
      uint32_t um[4] = {0u, 0u, 0u, 0u};  // this lane's uncertain dims
      if (t >= 0 && t < nnew)
        for (int j = 0; j < kD; ++j)
          if (myrow[j] == kUncertain) um[j >> 5] |= 1u << (j & 31);
      for (uint64_t act = __ballot((um[0] | um[1] | um[2] | um[3]) != 0u); act != 0u;
           act = __ballot((um[0] | um[1] | um[2] | um[3]) != 0u)) {
        const int L = __builtin_ctzll(act);
        const int jl = um[0] ? __builtin_ctz(um[0])
                       : um[1] ? 32 + __builtin_ctz(um[1])
                       : um[2] ? 64 + __builtin_ctz(um[2])
                       : um[3] ? 96 + __builtin_ctz(um[3]) : 0;
        const int j = __shfl(jl, L);
        const int tl = __shfl(t, L);
        const uint32_t xw = *(const uint32_t*)(x + (int64_t)tl * kD + 2 * lane);
        double part = (double)f16_bits_to_f32(xw & 0xFFFFu) * (double)P[(2 * lane) * kD + j];
        part = fma((double)f16_bits_to_f32(xw >> 16), (double)P[(2 * lane + 1) * kD + j], part);
        part = wave_sum_f64(part);
        if (lane == L) {
          myrow[j] = f64_to_f16_bits(part);
          um[j >> 5] &= ~(1u << (j & 31));
        }
      }
      __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
      __builtin_amdgcn_wave_barrier();
    }

    // ---- one token per lane ----
    const int pos = pos0 + lane;
    const int t = pos - len_old;
    const bool mine = t >= 0 && t < nnew;
    const bool dense = pos >= len_new - a.bb;
    const uint16_t* row = (const uint16_t*)(rows + lane * kRowHalves);
    if (mine && dense) {  // stays in the buffer: ring slot pos % b
      u32x4* dst = (u32x4*)(ring + (int64_t)(pos % a.bb) * kD);
#pragma unroll
      for (int c = 0; c < 16; ++c) dst[c] = ((const u32x4*)row)[c];
    } else if (mine) {
      uint32_t v[64];
#pragma unroll
      for (int c = 0; c < 16; ++c) {
        const u32x4 c4 = ((const u32x4*)row)[c];
        v[4 * c] = c4.x;
        v[4 * c + 1] = c4.y;
        v[4 * c + 2] = c4.z;
        v[4 * c + 3] = c4.w;
      }
      uint32_t kept[4];
      kept_dims(v, k, kept);
      store_slot<F>(row, kept, k, kp, pages + (int64_t)blk * pbytes, lane);
    }
    // the rows are rewritten by the next block
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();
  }
}

int prefill_groups(int max_new_tokens, int min_len_old) {
  (void)min_len_old;
  const int max_blocks = (max_new_tokens + kPage - 1) / kPage + 1;
  const int per_wg = kPrefillBlocksPerWave * kPrefillWaves;
  return (max_blocks + per_wg - 1) / per_wg;
}

template <typename F>
static hipError_t launch_prefill_f(const CompressLaunch& a, dim3 grid) {
  const hipError_t e = hipFuncSetAttribute((const void*)prefill_kernel<F>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, kPrefillLds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(prefill_kernel<F>, grid, dim3(64 * kPrefillWaves), kPrefillLds, a.stream, a);
  return hipGetLastError();
}

hipError_t launch_prefill(const CompressLaunch& a) {
  const int pairs = (2 * a.Hkv + kXcds - 1) / kXcds * kXcds;  // (head, role), padded
  const dim3 grid((int64_t)pairs * a.B * a.prefill_groups);
  if (a.dtype == SWAN_F16_E4M3) return launch_prefill_f<E4M3V>(a, grid);
  return launch_prefill_f<_Float16>(a, grid);
}

}  // namespace swan
