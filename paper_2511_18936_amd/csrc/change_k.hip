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
// magnitude key by a bitwise search, counting the keys at or above a candidate
// several at a time with packed integer arithmetic on the stored words; the
// kept pairs then go to the destination page in ascending index order (ties at
// the k'-th magnitude to the lower index), assembled in LDS and written with
// 16-byte stores.
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

// Grid: nsel * Hkv * max_pages waves over the selected sequences, whose source
// k_pad is KPS8 * 8 and whose k is raised or kept (kRaise) or lowered.  Dynamic
// LDS (lowering): the largest destination page of the launch.
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
  // the k'-th largest key: the largest tau with at least kd keys >= tau.  The
  // padding entries hold +0 (key 0) and every candidate is >= 1, so they never
  // count.
  uint32_t tau = 0;
  int need_eq;
  {
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
    uint32_t greater = 0;
    if (tau < MK::kMax) {
      uint32_t acc = 0;
#pragma unroll
      for (int i = 0; i < NW; ++i) acc += MK::count_ge(pk[i], tau + 1u);
      greater = MK::total(acc);
    }
    need_eq = kd - (int)greater;
  }

  // The stored pairs are in ascending index order, except after a raise: its
  // zero-valued pairs then follow the pairs kept at pruning.  In the first case
  // the stored order is the index order, so ties at tau go to the lower index by
  // taking them in stored order and the kept pairs are written in that order;
  // otherwise the kept dims are first collected in a 128-bit mask (ties: the
  // need_eq lowest tied dims) and each kept pair goes to its rank in the mask.
  const bool pad = kpd > kd;
  const int kv = valid ? ks : 0;
  bool asc = true;
  {
    uint32_t prev = 0u;
#pragma unroll
    for (int e = 0; e < KPS; ++e) {
      const uint32_t d = (ix[e / 4] >> ((e % 4) * 8)) & 0xFFu;
      asc = asc && (e == 0 || e >= kv || d > prev);
      prev = d;
    }
  }
  uint32_t u0 = 0u, u1 = 0u, u2 = 0u, u3 = 0u;  // the kept dims (for the padding)
  int j = 0;
  if (__ballot(!asc) == 0) {  // uniform: every lane's pairs are in index order
#pragma unroll
    for (int e = 0; e < KPS; ++e) {
      const uint32_t v = (w[e / EPW] >> ((e % EPW) * VB * 8)) & VMASK;
      const uint32_t key = MK::key(v);
      const bool tie = key == tau;
      const bool keep = e < kv && (key > tau || (tie && need_eq > 0));
      if (keep) {
        need_eq -= tie ? 1 : 0;
        const uint32_t d = (ix[e / 4] >> ((e % 4) * 8)) & 0xFFu;
        write_val<F>(lds, val_off<F>(j, lane), v);
        lds[idx_off(j, lane, kpd, VB)] = (char)d;
        if (pad) {  // uniform
          const uint32_t bit = 1u << (d & 31);
          const uint32_t wd = d >> 5;  // indices are < 128 in a valid cache
          u0 |= wd == 0u ? bit : 0u;
          u1 |= wd == 1u ? bit : 0u;
          u2 |= wd == 2u ? bit : 0u;
          u3 |= wd == 3u ? bit : 0u;
        }
        ++j;
      }
    }
  } else {
    // dims above tau and dims at tau
    uint32_t g0 = 0u, g1 = 0u, g2 = 0u, g3 = 0u, t0 = 0u, t1 = 0u, t2 = 0u, t3 = 0u;
#pragma unroll
    for (int e = 0; e < KPS; ++e) {
      const uint32_t v = (w[e / EPW] >> ((e % EPW) * VB * 8)) & VMASK;
      const uint32_t key = MK::key(v);
      const uint32_t d = (ix[e / 4] >> ((e % 4) * 8)) & 0x7Fu;
      const uint32_t bit = 1u << (d & 31);
      const uint32_t wd = d >> 5;
      const uint32_t gb = e < kv && key > tau ? bit : 0u;
      const uint32_t tb = e < kv && key == tau ? bit : 0u;
      g0 |= wd == 0u ? gb : 0u;
      g1 |= wd == 1u ? gb : 0u;
      g2 |= wd == 2u ? gb : 0u;
      g3 |= wd == 3u ? gb : 0u;
      t0 |= wd == 0u ? tb : 0u;
      t1 |= wd == 1u ? tb : 0u;
      t2 |= wd == 2u ? tb : 0u;
      t3 |= wd == 3u ? tb : 0u;
    }
    // keep the need_eq lowest tied dims
    uint32_t tw[4] = {t0, t1, t2, t3};
    int need = need_eq;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int c = __builtin_popcount(tw[q]);
      if (c <= need) {
        need -= c;
      } else {
        uint32_t rest = tw[q], keep = 0u;
        for (int i = 0; i < need; ++i) {
          keep |= rest & (0u - rest);
          rest &= rest - 1u;
        }
        tw[q] = keep;
        need = 0;
      }
    }
    u0 = g0 | tw[0];
    u1 = g1 | tw[1];
    u2 = g2 | tw[2];
    u3 = g3 | tw[3];
    const int c0 = __builtin_popcount(u0), c1 = c0 + __builtin_popcount(u1),
              c2 = c1 + __builtin_popcount(u2);
    j = c2 + __builtin_popcount(u3);
#pragma unroll
    for (int e = 0; e < KPS; ++e) {
      const uint32_t v = (w[e / EPW] >> ((e % EPW) * VB * 8)) & VMASK;
      const uint32_t d = (ix[e / 4] >> ((e % 4) * 8)) & 0x7Fu;
      const uint32_t wd = d >> 5;
      const uint32_t m = wd == 0u ? u0 : wd == 1u ? u1 : wd == 2u ? u2 : u3;
      const int before = wd == 0u ? 0 : wd == 1u ? c0 : wd == 2u ? c1 : c2;
      if (e < kv && ((m >> (d & 31)) & 1u)) {
        const int slot = before + __builtin_popcount(m & ((1u << (d & 31)) - 1u));
        write_val<F>(lds, val_off<F>(slot, lane), v);
        lds[idx_off(slot, lane, kpd, VB)] = (char)d;
      }
    }
  }
  // value 0 at the lowest free dims (at most 128 - j dims are used, so they never
  // run out before kpd); slots of tokens past the end get value 0 and index 0
  int word = 0;
  uint32_t fr = ~u0;
  for (; j < kpd; ++j) {
    while (fr == 0u && word < 3) {
      ++word;
      fr = word == 1 ? ~u1 : word == 2 ? ~u2 : ~u3;
    }
    const int d = valid ? word * 32 + __builtin_ctz(fr) : 0;
    fr &= fr - 1u;
    write_val<F>(lds, val_off<F>(j, lane), 0u);
    lds[idx_off(j, lane, kpd, VB)] = (char)d;
  }
  __syncthreads();
  for (int64_t off = lane * 16; off < pbd; off += 64 * 16)
    *(u32x4*)(dp + off) = *(const u32x4*)(lds + off);
  }
}

template <typename F, int KPS8, bool kRaise>
static hipError_t launch_sel(const ChangeKLaunch& a, size_t lds_bytes) {
  hipError_t e = hipFuncSetAttribute((const void*)change_k_kernel<F, KPS8, kRaise>,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds_bytes);
  if (e != hipSuccess) return e;
  const dim3 grid(a.nsel * a.Hkv * a.max_pages);
  hipLaunchKernelGGL((change_k_kernel<F, KPS8, kRaise>), grid, dim3(64), lds_bytes, a.stream, a);
  return hipGetLastError();
}

template <typename F, int... Is>
static hipError_t dispatch_kps8(int kps8, bool raise, const ChangeKLaunch& a, size_t lds,
                                std::integer_sequence<int, Is...>) {
  hipError_t e = hipErrorInvalidValue;
  ((kps8 == Is + 1 ? (e = raise ? launch_sel<F, Is + 1, true>(a, lds)
                                : launch_sel<F, Is + 1, false>(a, lds),
                      0)
                   : 0),
   ...);
  return e;
}

// One launch per source k_pad and direction (raised or kept, lowered) among the
// sequences.
hipError_t launch_change_k(const ChangeKLaunch& in) {
  const int vb = in.dtype == SWAN_F32 ? 4 : in.dtype == SWAN_F16 ? 2 : 1;
  uint32_t present = 0;
  for (int b = 0; b < in.B; ++b) present |= 1u << (kpad_of(in.k_src[b]) / 8 - 1);
  for (int kps8 = 1; kps8 <= 16; ++kps8) {
    if (!(present & (1u << (kps8 - 1)))) continue;
    for (int raise = 0; raise < 2; ++raise) {
      ChangeKLaunch a = in;
      a.nsel = 0;
      a.max_pages = 0;
      size_t lds = 16;
      for (int b = 0; b < in.B; ++b) {
        if (kpad_of(in.k_src[b]) / 8 != kps8 || (in.k_dst[b] >= in.k_src[b]) != (raise != 0))
          continue;
        a.sel[a.nsel++] = b;
        const int S = in.len[b] > in.bb ? in.len[b] - in.bb : 0;
        if (pages_for(S) > a.max_pages) a.max_pages = pages_for(S);
        const size_t n = raise ? 0 : (size_t)page_bytes_of(vb, in.k_dst[b]);
        if (n > lds) lds = n;
      }
      if (a.max_pages == 0) continue;
      hipError_t e;
      if (in.dtype == SWAN_F16)
        e = dispatch_kps8<_Float16>(kps8, raise, a, lds, std::make_integer_sequence<int, 16>{});
      else if (in.dtype == SWAN_F16_E4M3)
        e = dispatch_kps8<E4M3V>(kps8, raise, a, lds, std::make_integer_sequence<int, 16>{});
      else
        e = dispatch_kps8<float>(kps8, raise, a, lds, std::make_integer_sequence<int, 16>{});
      if (e != hipSuccess) return e;
    }
  }
  return hipSuccess;
}

}  // namespace swan
