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
// One wave per (sequence, KV head, page) and one launch per role; lane t owns
// token t of the page.  The source page is staged in LDS with 16-byte loads,
// the destination page is assembled in LDS and written with 16-byte stores.
// Lowering finds the k'-th largest magnitude key of the lane's k entries by a
// bitwise search (one pass over the entries per key bit), then walks the
// entries in index order keeping those above it and the first ties.
#include "swan_device.h"
#include "swan_internal.h"

namespace swan {

// magnitude key of a stored value (larger key = larger magnitude) and its bits
template <typename F>
struct MagKey;
template <>
struct MagKey<_Float16> {
  static constexpr int kBits = 15;
  __device__ static uint32_t get(uint32_t v) { return v & 0x7FFFu; }
};
template <>
struct MagKey<float> {
  static constexpr int kBits = 31;
  __device__ static uint32_t get(uint32_t v) { return v & 0x7FFFFFFFu; }
};
template <>
struct MagKey<E4M3V> {
  static constexpr int kBits = 7;
  __device__ static uint32_t get(uint32_t v) { return v & 0x7Fu; }
};

// byte offsets of entry e of slot t in a page of k_pad kp (include/swan.h)
template <typename F>
__device__ __forceinline__ int val_off(int e, int t) {
  constexpr int VB = Fmt<F>::kValBytes, CB = Fmt<F>::kChunkBytes, GV = CB / VB;
  return (e / GV) * 64 * CB + t * CB + (e % GV) * VB;
}
template <typename F>
__device__ __forceinline__ int idx_off(int e, int t, int kp) {
  return 64 * kp * Fmt<F>::kValBytes + (e / 8) * 512 + t * 8 + (e % 8);
}

template <typename F>
__device__ __forceinline__ uint32_t read_val(const char* page, int off) {
  constexpr int VB = Fmt<F>::kValBytes;
  if constexpr (VB == 1) return *(const uint8_t*)(page + off);
  else if constexpr (VB == 2) return *(const uint16_t*)(page + off);
  else return *(const uint32_t*)(page + off);
}
template <typename F>
__device__ __forceinline__ void write_val(char* page, int off, uint32_t v) {
  constexpr int VB = Fmt<F>::kValBytes;
  if constexpr (VB == 1) *(uint8_t*)(page + off) = (uint8_t)v;
  else if constexpr (VB == 2) *(uint16_t*)(page + off) = (uint16_t)v;
  else *(uint32_t*)(page + off) = v;
}

// Grid: B * Hkv * max_pages waves.  Dynamic LDS: the largest source page
// (rounded to 16 bytes) plus the largest destination page of the launch.
template <typename F>
__global__ __launch_bounds__(64) void change_k_kernel(ChangeKLaunch a) {
  extern __shared__ __attribute__((aligned(16))) char lds[];
  using MK = MagKey<F>;
  const int lane = threadIdx.x;
  const int p = blockIdx.x % a.max_pages;
  const int bh = blockIdx.x / a.max_pages;
  const int b = bh / a.Hkv, h = bh % a.Hkv;
  const int L = a.len[b];
  const int S = L > a.bb ? L - a.bb : 0;
  if (p >= pages_for(S)) return;
  const int ks = a.k_src[b], kd = a.k_dst[b];
  const int kps = kpad_of(ks), kpd = kpad_of(kd);
  const int64_t pbs = page_bytes_of(Fmt<F>::kValBytes, ks);
  const int64_t pbd = page_bytes_of(Fmt<F>::kValBytes, kd);
  const char* sp = a.src + a.off_src[b] + ((int64_t)h * a.npc_src + p) * pbs;
  char* dp = a.dst + a.off_dst[b] + ((int64_t)h * a.npc_dst + p) * pbd;
  char* ls = lds;                                  // source page
  char* ld = lds + ((pbs + 15) & ~(int64_t)15);    // destination page

  for (int64_t off = lane * 16; off < pbs; off += 64 * 16)
    *(u32x4*)(ls + off) = __builtin_nontemporal_load((const u32x4*)(sp + off));
  for (int64_t off = lane * 16; off < pbd; off += 64 * 16)
    *(u32x4*)(ld + off) = u32x4{0u, 0u, 0u, 0u};
  __syncthreads();

  if (p * kPage + lane < S) {
    // k'-th largest key (lowering only): the largest tau with at least kd keys >= tau
    uint32_t tau = 0;
    int need_eq = 0;
    if (kd < ks) {
      for (int bit = MK::kBits - 1; bit >= 0; --bit) {
        const uint32_t cand = tau | (1u << bit);
        int cnt = 0;
        for (int e = 0; e < ks; ++e)
          cnt += MK::get(read_val<F>(ls, val_off<F>(e, lane))) >= cand ? 1 : 0;
        if (cnt >= kd) tau = cand;
      }
      int greater = 0;
      for (int e = 0; e < ks; ++e)
        greater += MK::get(read_val<F>(ls, val_off<F>(e, lane))) > tau ? 1 : 0;
      need_eq = kd - greater;
    }
    // kept entries in index order, then zero-valued slots at the lowest free dims;
    // u0..u3: the dims used so far, as a 128-bit mask
    uint32_t u0 = 0u, u1 = 0u, u2 = 0u, u3 = 0u;
    int j = 0;
    for (int e = 0; e < ks; ++e) {
      const uint32_t v = read_val<F>(ls, val_off<F>(e, lane));
      bool keep = true;
      if (kd < ks) {
        const uint32_t key = MK::get(v);
        keep = key > tau || (key == tau && need_eq > 0);
        if (keep && key == tau) --need_eq;
      }
      if (!keep) continue;
      const uint32_t d = (uint8_t)ls[idx_off<F>(e, lane, kps)];
      write_val<F>(ld, val_off<F>(j, lane), v);
      ld[idx_off<F>(j, lane, kpd)] = (char)d;
      const uint32_t bit = 1u << (d & 31);
      const uint32_t w = (d >> 5) & 3u;  // indices are < 128 in a valid cache
      u0 |= w == 0u ? bit : 0u;
      u1 |= w == 1u ? bit : 0u;
      u2 |= w == 2u ? bit : 0u;
      u3 |= w == 3u ? bit : 0u;
      ++j;
    }
    // at most 128 - j dims are used, so the free ones never run out before kpd
    int word = 0;
    uint32_t fr = ~u0;
    for (; j < kpd; ++j) {  // values are already 0
      while (fr == 0u && word < 3) {
        ++word;
        fr = word == 1 ? ~u1 : word == 2 ? ~u2 : ~u3;
      }
      const int d = word * 32 + __builtin_ctz(fr);
      fr &= fr - 1u;
      ld[idx_off<F>(j, lane, kpd)] = (char)d;
    }
  }
  __syncthreads();
  for (int64_t off = lane * 16; off < pbd; off += 64 * 16)
    *(u32x4*)(dp + off) = *(const u32x4*)(ld + off);
}

template <typename F>
static hipError_t launch_change_k_t(const ChangeKLaunch& a, size_t lds_bytes) {
  hipError_t e = hipFuncSetAttribute((const void*)change_k_kernel<F>,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds_bytes);
  if (e != hipSuccess) return e;
  const dim3 grid(a.B * a.Hkv * a.max_pages);
  hipLaunchKernelGGL(change_k_kernel<F>, grid, dim3(64), lds_bytes, a.stream, a);
  return hipGetLastError();
}

hipError_t launch_change_k(const ChangeKLaunch& a) {
  if (a.max_pages <= 0) return hipSuccess;
  size_t lds = 0;
  const int vb = a.dtype == SWAN_F32 ? 4 : a.dtype == SWAN_F16 ? 2 : 1;
  for (int b = 0; b < a.B; ++b) {
    const size_t n = (size_t)((page_bytes_of(vb, a.k_src[b]) + 15) & ~(int64_t)15) +
                     (size_t)page_bytes_of(vb, a.k_dst[b]);
    if (n > lds) lds = n;
  }
  if (a.dtype == SWAN_F16) return launch_change_k_t<_Float16>(a, lds);
  if (a.dtype == SWAN_F16_E4M3) return launch_change_k_t<E4M3V>(a, lds);
  return launch_change_k_t<float>(a, lds);
}

}  // namespace swan
