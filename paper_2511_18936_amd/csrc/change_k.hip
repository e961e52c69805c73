// Run-time change of k for running sequences.  Algorithm 1 takes k_active as
// an input at every step; this lays the sparse cache of each (sequence, KV
// head, role) out again for a new k, so that a sequence can continue with it:
//   lowering (k' < k): each stored token keeps the k' largest of its k stored
//     values, ties to the lower index.  For values stored in T this is the
//     token's own top-k' (the top-k' of a top-k set, under one tie rule); for
//     8-bit values it ranks the stored codes.
//   raising (k' > k): the k pairs are kept (the tokens were pruned with the k
//     of their step) and slots k..k'-1 take value 0 at the lowest dims not kept.
//   equal: the pairs are copied.
// Slots past k' up to k'_pad are the usual padding: value 0 at the next lowest
// dims not kept.
//
// One wave per (sequence, KV head, page) and one launch per role and source
// k_pad; lane t owns token t of the page.  The kernel is specialised on the
// source k_pad, so a lane holds its token's k_pad values and indices in
// registers, loaded with one coalesced 16-byte (8-byte for E4M3) load per
// chunk.  Raising and copying store those chunks back in place, then the new
// padding, straight from registers.  Lowering finds the k'-th largest
// magnitude key (binary16: a radix select on bit planes of the keys; the other
// formats: a bitwise search counting the keys at or above a candidate several
// at a time with packed integer arithmetic), marks the kept dims in a 128-bit
// mask (ties at the k'-th magnitude to the lower index) while putting each
// stored value in an LDS row of the lane indexed by dim, then walks the mask
// in ascending order and stores the destination slot 8 entries at a time.
#include <utility>

#include "swan_device.h"
#include "swan_internal.h"

namespace swan {

// Per format: magnitude keys (larger key = larger magnitude) of the values
// packed in a 32-bit word, and the number of them >= a candidate.
template <typename F>
struct MagKey;

// binary16: two keys of 15 bits per word.  (key | 0x8000) - cand keeps bit 15
// set exactly when key >= cand, and never borrows out of its half; the count
// is the population of bits 15 and 31.
template <>
struct MagKey<_Float16> {
  static constexpr int kBits = 15;
  static constexpr uint32_t kMax = 0x7FFFu;
  __device__ static uint32_t prep(uint32_t w) { return (w & 0x7FFF7FFFu) | 0x80008000u; }
  __device__ static uint32_t count_ge(uint32_t p, uint32_t cand) {
    return (uint32_t)__builtin_popcount((p - cand * 0x10001u) & 0x80008000u);
  }
  __device__ static uint32_t total(uint32_t acc) { return acc; }
  __device__ static uint32_t key(uint32_t v) { return v & 0x7FFFu; }
};
// E4M3 codes: four keys of 7 bits per word, the same trick per byte (the
// codes saturate at 448, so no key is the NaN code)
template <>
struct MagKey<E4M3V> {
  static constexpr int kBits = 7;
  static constexpr uint32_t kMax = 0x7Fu;
  __device__ static uint32_t prep(uint32_t w) { return (w & 0x7F7F7F7Fu) | 0x80808080u; }
  __device__ static uint32_t count_ge(uint32_t p, uint32_t cand) {
    return (uint32_t)__builtin_popcount((p - cand * 0x01010101u) & 0x80808080u);
  }
  __device__ static uint32_t total(uint32_t acc) { return acc; }
  __device__ static uint32_t key(uint32_t v) { return v & 0x7Fu; }
};
// float32: one key of 31 bits per word
template <>
struct MagKey<float> {
  static constexpr int kBits = 31;
  static constexpr uint32_t kMax = 0x7FFFFFFFu;
  __device__ static uint32_t prep(uint32_t w) { return w & 0x7FFFFFFFu; }
  __device__ static uint32_t count_ge(uint32_t p, uint32_t cand) { return p >= cand ? 1u : 0u; }
  __device__ static uint32_t total(uint32_t acc) { return acc; }
  __device__ static uint32_t key(uint32_t v) { return v & 0x7FFFFFFFu; }
};

// One step of a 16x16 bit-matrix transpose applied to both 16-bit halves of
// 16 words at once (row i of each matrix = half of w[i], column b = bit b):
// the K x K off-diagonal blocks of every 2K x 2K block trade places.
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

// Bits 0-15 of a bit-plane word stand for a group's even entries, bits 16-31
// for its odd ones; this puts them in entry order (bit i = entry 32 c + i).
__device__ __forceinline__ uint32_t spread16(uint32_t x) {
  x = (x | (x << 8)) & 0x00FF00FFu;
  x = (x | (x << 4)) & 0x0F0F0F0Fu;
  x = (x | (x << 2)) & 0x33333333u;
  return (x | (x << 1)) & 0x55555555u;
}
__device__ __forceinline__ uint32_t entry_order(uint32_t w) {
  return spread16(w & 0xFFFFu) | (spread16(w >> 16) << 1);
}

// binary16 pages: the kd-th largest tau of the 15-bit magnitude keys of
// entries 0..kv-1 (two per word of w), by a radix select on bit planes.  Each
// group of 16 words (32 entries) is transposed so that plane b holds bit b of
// every key (bits 0-15: the group's even entries, 16-31: its odd ones); from
// the top bit down, the entries still equal to the threshold's prefix are
// split by the next bit, and those above it collected.  Out: tau, and the
// entries above it (gt) and equal to it (eq) as masks in entry order, word c
// for entries 32 c .. 32 c + 31.
template <int NW>
__device__ __forceinline__ void kth_key_f16(const uint32_t* w, int kv, int kd, uint32_t& tau,
                                            uint32_t* gt_out, uint32_t* eq_out) {
  constexpr int NC = (NW + 15) / 16;
  uint32_t pl[15][NC], eq[NC], gt[NC];
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    uint32_t t[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) t[i] = 16 * c + i < NW ? w[16 * c + i] & 0x7FFF7FFFu : 0u;
    transpose_step<8>(t, 0x00FF00FFu);
    transpose_step<4>(t, 0x0F0F0F0Fu);
    transpose_step<2>(t, 0x33333333u);
    transpose_step<1>(t, 0x55555555u);
#pragma unroll
    for (int b = 0; b < 15; ++b) pl[b][c] = t[b];
    // entries 32 c + 2 i (bit i) and 32 c + 2 i + 1 (bit 16 + i) below kv
    const int ne = min(max((kv - 32 * c + 1) / 2, 0), 16);
    const int no = min(max((kv - 32 * c) / 2, 0), 16);
    eq[c] = (uint32_t)((1ull << ne) - 1ull) | ((uint32_t)((1ull << no) - 1ull) << 16);
    gt[c] = 0u;
  }
  uint32_t th = 0u;
  int ngt = 0;
#pragma unroll
  for (int b = 14; b >= 0; --b) {
    uint32_t hi[NC];
    int cnt = 0;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      hi[c] = eq[c] & pl[b][c];
      cnt += __popc(hi[c]);
    }
    const bool one = ngt + cnt >= kd;  // the kd-th largest has this bit set
    th |= one ? 1u << b : 0u;
    ngt += one ? 0 : cnt;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      gt[c] |= one ? 0u : hi[c];
      eq[c] = one ? hi[c] : (eq[c] & ~pl[b][c]);
    }
  }
  tau = th;
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    gt_out[c] = entry_order(gt[c]);
    eq_out[c] = entry_order(eq[c]);
  }
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

// bit d (< 128) of a 128-bit mask, set when on (0 or 1).  Flags stay 0/1
// integers in vector registers: as lane masks they would pile up in scalar
// registers over an unrolled loop.
__device__ __forceinline__ void set_dim(uint64_t& lo, uint64_t& hi, uint32_t d, uint32_t on) {
  const uint32_t up = d >> 6;  // 0: dims 0-63, 1: dims 64-127
  lo |= (uint64_t)(on & (up ^ 1u)) << (d & 63u);
  hi |= (uint64_t)(on & up) << (d & 63u);
}
// The compiler is made to forget what it knows of the n words in r (an empty
// asm per word), so that values derived from them in one phase are derived
// again in the next instead of being kept live across it.
template <int N>
__device__ __forceinline__ void launder(uint32_t* r) {
#pragma unroll
  for (int i = 0; i < N; ++i) asm volatile("" : "+v"(r[i]));
}

// 1 when a > b, 1 when a == b (values below 2^31), as integers
__device__ __forceinline__ uint32_t gt01(uint32_t a, uint32_t b) { return (b - a) >> 31; }
__device__ __forceinline__ uint32_t eq01(uint32_t a, uint32_t b) { return ((a ^ b) - 1u) >> 31; }

// byte offsets of entry e of slot t in a page of k_pad kp (include/swan.h)
template <typename F>
__device__ __forceinline__ int val_off(int e, int t) {
  constexpr int VB = Fmt<F>::kValBytes, CB = Fmt<F>::kChunkBytes, GV = CB / VB;
  return (e / GV) * 64 * CB + t * CB + (e % GV) * VB;
}
__device__ __forceinline__ int idx_off(int e, int t, int kp, int vb) {
  return 64 * kp * vb + (e / 8) * 512 + t * 8 + (e % 8);
}

template <typename F>
__device__ __forceinline__ void write_val(char* page, int off, uint32_t v) {
  constexpr int VB = Fmt<F>::kValBytes;
  if constexpr (VB == 1) *(uint8_t*)(page + off) = (uint8_t)v;
  else if constexpr (VB == 2) *(uint16_t*)(page + off) = (uint16_t)v;
  else *(uint32_t*)(page + off) = v;
}

// A lane's LDS row in the lowering kernel, source k_pad KPS: its KPS indices,
// then (16-byte aligned) its KPS values of VB bytes; padded by 16 bytes.
template <int KPS>
constexpr int ck_vals_off() {
  return (KPS + 15) / 16 * 16;
}
template <int KPS, int VB>
constexpr int ck_row_bytes() {
  return ck_vals_off<KPS>() + (KPS * VB + 15) / 16 * 16 + 16;
}

// entries 8 c .. 8 c + 7 of a lane's destination slot: values vw (VB bytes
// each, packed), indices iw (one byte each)
template <int VB>
__device__ __forceinline__ void store_chunk(char* dp, char* di, int c, int lane,
                                            const uint32_t* vw, const uint32_t* iw) {
  if constexpr (VB == 2) {
    *(u32x4*)(dp + c * 1024 + lane * 16) = u32x4{vw[0], vw[1], vw[2], vw[3]};
  } else if constexpr (VB == 1) {
    *(u32x2*)(dp + c * 512 + lane * 8) = u32x2{vw[0], vw[1]};
  } else {
    *(u32x4*)(dp + (2 * c) * 1024 + lane * 16) = u32x4{vw[0], vw[1], vw[2], vw[3]};
    *(u32x4*)(dp + (2 * c + 1) * 1024 + lane * 16) = u32x4{vw[4], vw[5], vw[6], vw[7]};
  }
  *(u32x2*)(di + c * 512 + lane * 8) = u32x2{iw[0], iw[1]};
}

// Grid: nsel * Hkv * max_pages waves over the selected sequences, whose source
// k_pad is KPS8 * 8 and whose k is raised or kept (kRaise) or lowered.  Dynamic
// LDS (lowering): the rows of the 64 lanes, ck_row_bytes each.
template <typename F, int KPS8, bool kRaise>
__global__ __launch_bounds__(64) void change_k_kernel(ChangeKLaunch a) {
  extern __shared__ __attribute__((aligned(16))) char lds[];
  using MK = MagKey<F>;
  constexpr int VB = Fmt<F>::kValBytes, CB = Fmt<F>::kChunkBytes;
  constexpr int KPS = KPS8 * 8;
  constexpr int NW = KPS * VB / 4;   // value words per token
  constexpr int NVC = KPS * VB / CB; // value chunks per token
  constexpr int WPC = CB / 4;        // words per chunk
  constexpr int EPW = 4 / VB;        // entries per word
  constexpr uint32_t VMASK = VB == 4 ? 0xFFFFFFFFu : VB == 2 ? 0xFFFFu : 0xFFu;
  const int lane = threadIdx.x;
  const int p = blockIdx.x % a.max_pages;
  const int sh = blockIdx.x / a.max_pages;
  const int b = a.sel[sh / a.Hkv], h = sh % a.Hkv;
  const int L = a.len[b];
  const int S = L > a.bb ? L - a.bb : 0;
  if (p >= pages_for(S)) return;
  const int ks = a.k_src[b], kd = a.k_dst[b];
  const int kpd = kpad_of(kd);
  constexpr int64_t pbs = (int64_t)64 * KPS * (VB + 1);
  const int64_t pbd = page_bytes_of(VB, kd);
  const char* sp = a.src + a.off_src[b] + ((int64_t)h * a.npc_src + p) * pbs;
  char* dp = a.dst + a.off_dst[b] + ((int64_t)h * a.npc_dst + p) * pbd;

  // the lane's values and indices
  uint32_t w[NW], ix[KPS / 4];
#pragma unroll
  for (int c = 0; c < NVC; ++c) {
    if constexpr (CB == 16) {
      const u32x4 v = __builtin_nontemporal_load((const u32x4*)(sp + c * 64 * CB + lane * CB));
      w[c * WPC + 0] = v.x;
      w[c * WPC + 1] = v.y;
      w[c * WPC + 2] = v.z;
      w[c * WPC + 3] = v.w;
    } else {
      const u32x2 v = __builtin_nontemporal_load((const u32x2*)(sp + c * 64 * CB + lane * CB));
      w[c * WPC + 0] = v.x;
      w[c * WPC + 1] = v.y;
    }
  }
#pragma unroll
  for (int g = 0; g < KPS8; ++g) {
    const u32x2 v =
        __builtin_nontemporal_load((const u32x2*)(sp + 64 * KPS * VB + g * 512 + lane * 8));
    ix[2 * g] = v.x;
    ix[2 * g + 1] = v.y;
  }
  const bool valid = p * kPage + lane < S;

  if constexpr (kRaise) {
    // Raising or copying keeps every pair in place.  The source's padding already
    // holds the lowest dims not kept, in ascending order, and so do the
    // destination's first padding slots, so the destination starts with the
    // source page's entries; slots from the source k_pad on take value 0 at the
    // next lowest dims not among the source's indices.  Each lane writes its own
    // chunks, so no page is staged.
    const int nvc_dst = kpd * VB / CB;
#pragma unroll
    for (int c = 0; c < NVC; ++c) {
      char* o = dp + c * 64 * CB + lane * CB;
      if constexpr (CB == 16) {
        const u32x4 v = valid ? u32x4{w[c * WPC], w[c * WPC + 1], w[c * WPC + 2], w[c * WPC + 3]}
                              : u32x4{0u, 0u, 0u, 0u};
        *(u32x4*)o = v;
      } else {
        *(u32x2*)o = valid ? u32x2{w[c * WPC], w[c * WPC + 1]} : u32x2{0u, 0u};
      }
    }
    for (int c = NVC; c < nvc_dst; ++c) {
      char* o = dp + c * 64 * CB + lane * CB;
      if constexpr (CB == 16) *(u32x4*)o = u32x4{0u, 0u, 0u, 0u};
      else *(u32x2*)o = u32x2{0u, 0u};
    }
    char* di = dp + 64 * kpd * VB;
#pragma unroll
    for (int g = 0; g < KPS8; ++g)
      *(u32x2*)(di + g * 512 + lane * 8) = valid ? u32x2{ix[2 * g], ix[2 * g + 1]} : u32x2{0u, 0u};
    if (kpd > KPS) {  // uniform
      // the source's dims (indices are < 128 and distinct in a valid cache, so at
      // least kpd - KPS dims are free)
      uint64_t m0 = 0, m1 = 0;
#pragma unroll
      for (int e = 0; e < KPS; ++e) {
        const uint32_t d = (ix[e / 4] >> ((e % 4) * 8)) & 0x7Fu;
        const uint64_t bit = 1ull << (d & 63);
        m0 |= d < 64 ? bit : 0ull;
        m1 |= d < 64 ? 0ull : bit;
      }
      uint64_t f0 = ~m0, f1 = ~m1;
      for (int g = KPS8; g < kpd / 8; ++g) {
        uint32_t lo = 0u, hi = 0u;
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          uint32_t d;
          if (f0 != 0ull) {
            d = (uint32_t)__builtin_ctzll(f0);
            f0 &= f0 - 1ull;
          } else {
            d = 64u + (uint32_t)__builtin_ctzll(f1);
            f1 &= f1 - 1ull;
          }
          if (u < 4) lo |= d << (8 * u);
          else hi |= d << (8 * (u - 4));
        }
        *(u32x2*)(di + g * 512 + lane * 8) = valid ? u32x2{lo, hi} : u32x2{0u, 0u};
      }
    }
    return;
  } else {
  // the k'-th largest key tau among the token's kv stored values, the number of
  // keys above it and of keys equal to it
  const int kv = valid ? ks : 0;
  uint32_t tau = 0;
  int greater = 0, ties = 0;
  constexpr int NG = (KPS + 31) / 32;  // 32-entry groups
  uint32_t gtm[NG], eqm[NG];           // (binary16) entries above / at tau, entry order
  if constexpr (std::is_same<F, _Float16>::value) {
    kth_key_f16<NW>(w, kv, kd, tau, gtm, eqm);
#pragma unroll
    for (int c = 0; c < NG; ++c) {
      greater += __popc(gtm[c]);
      ties += __popc(eqm[c]);
    }
  } else {
    // the largest tau with at least kd keys >= tau (the padding entries hold +0,
    // key 0, and every candidate is >= 1, so they never count)
    uint32_t pk[NW];
#pragma unroll
    for (int i = 0; i < NW; ++i) pk[i] = MK::prep(w[i]);
#pragma unroll 1
    for (int bit = MK::kBits - 1; bit >= 0; --bit) {
      const uint32_t cand = tau | (1u << bit);
      uint32_t acc = 0;
#pragma unroll
      for (int i = 0; i < NW; ++i) acc += MK::count_ge(pk[i], cand);
      if ((int)MK::total(acc) >= kd) tau = cand;
    }
#pragma unroll
    for (int e = 0; e < KPS; ++e) {
      const uint32_t key = MK::key((w[e / EPW] >> ((e % EPW) * VB * 8)) & VMASK);
      greater += e < kv && key > tau ? 1 : 0;
      ties += e < kv && key == tau ? 1 : 0;
    }
  }
  const int need_eq = kd - greater;  // ties at tau to keep, lowest index first

  // The pairs are staged in an LDS row of the lane, indices at byte e and
  // values at byte VO + e VB (wide writes from registers).
  constexpr int VO = ck_vals_off<KPS>();
  char* lrow = lds + lane * ck_row_bytes<KPS, VB>();
  using VT = typename std::conditional<VB == 4, uint32_t,
                                       typename std::conditional<VB == 2, uint16_t, uint8_t>::type>::type;
#pragma unroll
  for (int c = 0; c < KPS / 16; ++c)
    *(u32x4*)(lrow + 16 * c) = u32x4{ix[4 * c], ix[4 * c + 1], ix[4 * c + 2], ix[4 * c + 3]};
  if constexpr (KPS % 16 != 0)
    *(u32x2*)(lrow + KPS / 16 * 16) = u32x2{ix[KPS / 16 * 4], ix[KPS / 16 * 4 + 1]};
#pragma unroll
  for (int c = 0; c < NW / 4; ++c)
    *(u32x4*)(lrow + VO + 16 * c) = u32x4{w[4 * c], w[4 * c + 1], w[4 * c + 2], w[4 * c + 3]};
  if constexpr (NW % 4 != 0)
#pragma unroll
    for (int i = NW / 4 * 4; i < NW; ++i) *(uint32_t*)(lrow + VO + 4 * i) = w[i];

  // bit e: entry e is one of the token's kv stored pairs
  const uint64_t emask_lo = kv >= 64 ? ~0ull : (1ull << kv) - 1ull;
  const uint64_t emask_hi = kv >= 128 ? ~0ull : kv > 64 ? (1ull << (kv - 64)) - 1ull : 0ull;
  // Some stored pair's index is not above the one before: 4 entries per word.
  // x = entries 4 i .. 4 i + 3, y = entries 4 i + 1 .. 4 i + 4 (bytes below
  // 128); byte j of (y | 0x80 each) - x - 1 (each) keeps its top bit exactly
  // when y_j > x_j, without borrowing from the next byte.
  uint32_t unordered = 0u;
  launder<KPS / 4>(ix);
#pragma unroll
  for (int i = 0; i < KPS / 4; ++i) {
    const uint32_t x = ix[i] & 0x7F7F7F7Fu;
    const uint32_t y = (x >> 8) | (i + 1 < KPS / 4 ? (ix[i + 1] & 0x7Fu) << 24 : 0x7F000000u);
    const uint32_t up = ((y | 0x80808080u) - x - 0x01010101u) & 0x80808080u;
    // pairs (4 i + j, 4 i + j + 1) with both entries below kv
    const int s0 = 4 * i + 1;  // the pairs' second entries: s0 .. s0 + 3
    const uint32_t in2 = (uint32_t)((s0 + 4 <= 64 ? emask_lo >> (s0 & 63)
                                     : s0 >= 64   ? emask_hi >> (s0 & 63)
                                                  : (emask_lo >> (s0 & 63)) | (emask_hi << ((64 - s0) & 63))) &
                                    0xFull);
    const uint32_t inb = ((in2 & 1u) << 7) | ((in2 & 2u) << 14) | ((in2 & 4u) << 21) |
                         ((in2 & 8u) << 28);
    unordered |= inb & ~up;
  }
  char* di = dp + 64 * kpd * VB;

  if (__ballot(unordered != 0u) == 0ull) {
    // Fast path (uniform): every lane's pairs are stored in ascending index
    // order, so the kept pairs are those with key > tau and the first need_eq
    // of those with key == tau, in stored order: a keep mask over the entries,
    // and each kept pair read back from the staged row by entry.
    uint64_t klo = 0ull, khi = 0ull, tlo = 0ull, thi = 0ull;
    if constexpr (std::is_same<F, _Float16>::value) {
      klo = gtm[0] | (NG > 1 ? (uint64_t)gtm[NG > 1 ? 1 : 0] << 32 : 0ull);
      tlo = eqm[0] | (NG > 1 ? (uint64_t)eqm[NG > 1 ? 1 : 0] << 32 : 0ull);
      khi = NG > 2 ? gtm[NG > 2 ? 2 : 0] | (NG > 3 ? (uint64_t)gtm[NG > 3 ? 3 : 0] << 32 : 0ull) : 0ull;
      thi = NG > 2 ? eqm[NG > 2 ? 2 : 0] | (NG > 3 ? (uint64_t)eqm[NG > 3 ? 3 : 0] << 32 : 0ull) : 0ull;
    } else {
    launder<NW>(w);
#pragma unroll
    for (int e = 0; e < KPS; ++e) {
      const uint32_t key = MK::key((w[e / EPW] >> ((e % EPW) * VB * 8)) & VMASK);
      const uint64_t in = ((e < 64 ? emask_lo : emask_hi) >> (e & 63)) & 1ull;
      const uint64_t gb = (in & (uint64_t)gt01(key, tau)) << (e & 63);
      const uint64_t tb = (in & (uint64_t)eq01(key, tau)) << (e & 63);
      if (e < 64) {
        klo |= gb;
        tlo |= tb;
      } else {
        khi |= gb;
        thi |= tb;
      }
    }
    }
    for (int i = 0; i < need_eq; ++i) {  // need_eq >= 1, most often 1
      const uint32_t e = pop_lowest(tlo, thi);
      if (e < 64u) klo |= 1ull << e;
      else khi |= 1ull << (e - 64u);
    }
    uint64_t ulo = 0ull, uhi = 0ull;  // kept dims, for the padding
    if (kpd > kd) {  // uniform
      launder<KPS / 4>(ix);
#pragma unroll
      for (int e = 0; e < KPS; ++e) {
        const uint32_t d = (ix[e / 4] >> ((e % 4) * 8)) & 0x7Fu;
        set_dim(ulo, uhi, d, (uint32_t)(((e < 64 ? klo : khi) >> (e & 63)) & 1ull));
      }
    }
    // the destination slot 8 entries at a time: the kept pairs, then value 0 at
    // the lowest dims not kept; slots of tokens past the end get value 0 and
    // index 0.  Each lane stores its own chunks (a wave's store is contiguous).
    uint64_t flo = ~ulo, fhi = ~uhi;
    for (int c = 0; c < kpd / 8; ++c) {
      const int nk = min(kd - 8 * c, 8);  // kept entries in this chunk (uniform)
      uint32_t d[8], v[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        if (q < nk) {
          uint32_t e;
          if constexpr (KPS <= 64) {  // the keep mask is klo alone
            e = (uint32_t)__builtin_ctzll(klo) & 63u;
            klo &= klo - 1ull;
          } else {
            e = pop_lowest(klo, khi) & 127u;
          }
          v[q] = (uint32_t)*(const VT*)(lrow + VO + e * VB);
          d[q] = (uint32_t)*(const uint8_t*)(lrow + e);
        } else {
          d[q] = pop_lowest(flo, fhi) & 127u;
          v[q] = 0u;
        }
      }
      uint32_t iw[2] = {0u, 0u}, vw[8] = {0u, 0u, 0u, 0u, 0u, 0u, 0u, 0u};
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        iw[q >> 2] |= d[q] << (8 * (q & 3));
        vw[q * VB / 4] |= v[q] << (8 * ((q * VB) & 3));
      }
      const uint32_t keepw = valid ? ~0u : 0u;  // slots of tokens past the end: 0
#pragma unroll
      for (int i = 0; i < 8; ++i) vw[i] &= keepw;
      iw[0] &= keepw;
      iw[1] &= keepw;
      store_chunk<VB>(dp, di, c, lane, vw, iw);
    }
    return;
  }

  // General path: pairs in any order (after a raise) or more ties at tau than
  // are kept.  The kept dims as a 128-bit mask (the ties: the need_eq lowest
  // tied dims), from the staged row in a rolled loop; then each kept pair goes
  // to the slot of its rank in the mask, and value 0 at the lowest dims not
  // kept fills the rest.  Stores are per entry: this path is rare.
  const uint32_t tau1 = ties > need_eq ? tau + 1u : tau;  // keys >= tau1 kept outright
  uint64_t ulo = 0ull, uhi = 0ull, tlo = 0ull, thi = 0ull;
#pragma unroll 1
  for (int e = 0; e < kv; ++e) {
    const uint32_t d = (uint32_t)*(const uint8_t*)(lrow + e) & 0x7Fu;
    const uint32_t key = MK::key((uint32_t)*(const VT*)(lrow + VO + e * VB));
    set_dim(ulo, uhi, d, gt01(key, tau1) | eq01(key, tau1));
    set_dim(tlo, thi, d, ties > need_eq ? eq01(key, tau) : 0u);
  }
  if (ties > need_eq)
    for (int i = 0; i < need_eq; ++i) set_dim(ulo, uhi, pop_lowest(tlo, thi), 1u);
  if (!valid) ulo = uhi = 0ull;
  const int nlo = __popcll(ulo);
#pragma unroll 1
  for (int e = 0; e < kv; ++e) {
    const uint32_t d = (uint32_t)*(const uint8_t*)(lrow + e) & 0x7Fu;
    const uint32_t v = (uint32_t)*(const VT*)(lrow + VO + e * VB);
    const uint64_t m = d < 64u ? ulo : uhi;
    if ((m >> (d & 63u)) & 1ull) {
      const int slot = (d < 64u ? 0 : nlo) + __popcll(m & ((1ull << (d & 63u)) - 1ull));
      write_val<F>(dp, val_off<F>(slot, lane), v);
      di[idx_off(slot, lane, 0, 0)] = (char)d;
    }
  }
  uint64_t flo = ~ulo, fhi = ~uhi;
#pragma unroll 1
  for (int j = valid ? kd : 0; j < kpd; ++j) {
    const uint32_t d = valid ? pop_lowest(flo, fhi) : 0u;
    write_val<F>(dp, val_off<F>(j, lane), 0u);
    di[idx_off(j, lane, 0, 0)] = (char)d;
  }
  }
}

template <typename F, int KPS8, bool kRaise>
static hipError_t launch_sel(const ChangeKLaunch& a) {
  const size_t lds_bytes = kRaise ? 16 : 64 * (size_t)ck_row_bytes<KPS8 * 8, Fmt<F>::kValBytes>();
  hipError_t e = hipFuncSetAttribute((const void*)change_k_kernel<F, KPS8, kRaise>,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds_bytes);
  if (e != hipSuccess) return e;
  const dim3 grid(a.nsel * a.Hkv * a.max_pages);
  hipLaunchKernelGGL((change_k_kernel<F, KPS8, kRaise>), grid, dim3(64), lds_bytes, a.stream, a);
  return hipGetLastError();
}

template <typename F, int... Is>
static hipError_t dispatch_kps8(int kps8, bool raise, const ChangeKLaunch& a,
                                std::integer_sequence<int, Is...>) {
  hipError_t e = hipErrorInvalidValue;
  ((kps8 == Is + 1 ? (e = raise ? launch_sel<F, Is + 1, true>(a)
                                : launch_sel<F, Is + 1, false>(a),
                      0)
                   : 0),
   ...);
  return e;
}

// One launch per source k_pad and direction (raised or kept, lowered) among the
// sequences.
hipError_t launch_change_k(const ChangeKLaunch& in) {
  uint32_t present = 0;
  for (int b = 0; b < in.B; ++b) present |= 1u << (kpad_of(in.k_src[b]) / 8 - 1);
  for (int kps8 = 1; kps8 <= 16; ++kps8) {
    if (!(present & (1u << (kps8 - 1)))) continue;
    for (int raise = 0; raise < 2; ++raise) {
      ChangeKLaunch a = in;
      a.nsel = 0;
      a.max_pages = 0;
      for (int b = 0; b < in.B; ++b) {
        if (kpad_of(in.k_src[b]) / 8 != kps8 || (in.k_dst[b] >= in.k_src[b]) != (raise != 0))
          continue;
        a.sel[a.nsel++] = b;
        const int S = in.len[b] > in.bb ? in.len[b] - in.bb : 0;
        if (pages_for(S) > a.max_pages) a.max_pages = pages_for(S);
      }
      if (a.max_pages == 0) continue;
      hipError_t e;
      if (in.dtype == SWAN_F16)
        e = dispatch_kps8<_Float16>(kps8, raise, a, std::make_integer_sequence<int, 16>{});
      else if (in.dtype == SWAN_F16_E4M3)
        e = dispatch_kps8<E4M3V>(kps8, raise, a, std::make_integer_sequence<int, 16>{});
      else
        e = dispatch_kps8<float>(kps8, raise, a, std::make_integer_sequence<int, 16>{});
      if (e != hipSuccess) return e;
    }
  }
  return hipSuccess;
}

}  // namespace swan
