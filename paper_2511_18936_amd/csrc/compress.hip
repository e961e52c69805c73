// Compress-append (Algorithm 1, the steps that project, append, evict and
// prune).
//
// Several new tokens per sequence: two launches on the caller's stream, so
// that every vector leaving the ring is read before a new token overwrites its
// slot.  One new token (a decode step): one launch, insert_kernel<F, 1>, whose
// wave evicts the slot's old vector before it writes the new one.
//   evict_kernel   one wave per ring vector that leaves the buffer: top-k of
//                  its stored values, packed into its page slot
//   insert_kernel  one wave per group of TPW new tokens of one (sequence, kv
//                  head, role) (TPW = 1 for a decode step, which also does
//                  that step's eviction, else 8): rotation
//                  x . P accumulated in float64 and rounded once to the storage
//                  type; tokens still inside the buffer go to their ring slot,
//                  the others are pruned and packed at once.  In a
//                  decode step (swan_decode_step) the key wave of (sequence,
//                  kv head) also rotates the step's queries of that head's
//                  QG query heads with the same rows of P_QK: q_hat for the
//                  attention that follows, with the summation order of the
//                  separate query rotation (qrot_kernel), so the same bits
//
// Top-k (Sec. 4.3, ranking the stored values, ties to the lower index): each
// lane holds dims 2l and 2l+1; the key (|x| bits << 8) | (255 - dim) is unique
// and orders by magnitude, then by lower index.  A binary search over the key
// bits with wave ballots finds the k-th largest key; the selected entries are
// then numbered in ascending dim order with mbcnt and written to the page.
#include <type_traits>

#include "swan_device.h"
#include "swan_internal.h"

namespace swan {

constexpr int kTPW = 8;  // new tokens per insert wave (several new tokens per sequence)

// Write the top-k of a 128-vector of stored values (lane holds elements 2l,
// 2l+1) into page slot `slot` of the page at `page`, in page format F (the
// values as stored, or rounded to E4M3; the selection ranks the stored values).
template <typename F>
__device__ __forceinline__ void select_and_pack(typename Store<typename Fmt<F>::Elem>::Bits x0,
                                                typename Store<typename Fmt<F>::Elem>::Bits x1,
                                                int k, char* page, int slot, int lane) {
  using St = Store<typename Fmt<F>::Elem>;
  using Key = typename std::conditional<(St::kMagBits + 8 > 32), uint64_t, uint32_t>::type;
  constexpr int kKeyBits = St::kMagBits + 8;
  const Key key0 = ((Key)St::mag(x0) << 8) | (Key)(255 - 2 * lane);
  const Key key1 = ((Key)St::mag(x1) << 8) | (Key)(255 - (2 * lane + 1));
  Key thr = 0;
  for (int bit = kKeyBits - 1; bit >= 0; --bit) {
    const Key cand = thr | ((Key)1 << bit);
    const int cnt = __popcll(__ballot(key0 >= cand)) + __popcll(__ballot(key1 >= cand));
    if (cnt >= k) thr = cand;
  }
  const bool s0 = key0 >= thr;
  const bool s1 = key1 >= thr;
  const uint64_t m0 = __ballot(s0);
  const uint64_t m1 = __ballot(s1);
  const int e0 = popc_below(m0) + popc_below(m1);
  const int e1 = e0 + (s0 ? 1 : 0);
  constexpr int VB = Fmt<F>::kValBytes, CB = Fmt<F>::kChunkBytes, GV = CB / VB;
  const int kp = kpad_of(k);
  char* vals = page + slot * CB;
  char* idxs = page + (int64_t)kPage * kp * VB + slot * 8;
  auto put = [&](int e, typename St::Bits x) {
    char* dst = vals + (e / GV) * (kPage * CB) + (e % GV) * VB;
    if constexpr (std::is_same<F, E4M3V>::value)
      *(uint8_t*)dst = (uint8_t)f16_bits_to_e4m3(x);
    else
      *(typename St::Bits*)dst = x;
  };
  if (s0) {
    put(e0, x0);
    idxs[(e0 / 8) * 512 + (e0 % 8)] = (char)(2 * lane);
  }
  if (s1) {
    put(e1, x1);
    idxs[(e1 / 8) * 512 + (e1 % 8)] = (char)(2 * lane + 1);
  }
  // padding entries k .. kp-1: value +0 at the lowest unselected dims, so that
  // the indices of a token stay distinct
  const int npad = kp - k;
  if (npad > 0) {
    const uint64_t n0 = __ballot(!s0);
    const uint64_t n1 = __ballot(!s1);
    const int r0 = popc_below(n0) + popc_below(n1);
    const int r1 = r0 + (s0 ? 0 : 1);
    if (!s0 && r0 < npad) {
      const int e = k + r0;
      put(e, 0);
      idxs[(e / 8) * 512 + (e % 8)] = (char)(2 * lane);
    }
    if (!s1 && r1 < npad) {
      const int e = k + r1;
      put(e, 0);
      idxs[(e / 8) * 512 + (e % 8)] = (char)(2 * lane + 1);
    }
  }
}

__device__ __forceinline__ int evict_begin(int len_old, int bb) {
  return len_old > bb ? len_old - bb : 0;
}

// tokens that leave the ring in this call: positions [begin, end)
__device__ __forceinline__ int evict_end(int len_old, int n_new, int bb) {
  const int lim = len_old + n_new - bb;
  return len_old < lim ? len_old : lim;
}

template <typename F>
__global__ __launch_bounds__(64) void evict_kernel(CompressLaunch a) {
  using St = Store<typename Fmt<F>::Elem>;
  const int lane = threadIdx.x;
  int w = blockIdx.x;
  const int e = w % a.max_evict;
  w /= a.max_evict;
  const int role = w & 1;
  w >>= 1;
  const int h = w % a.Hkv;
  const int b = w / a.Hkv;
  const int len_old = a.tab.len[b];
  const int p0 = evict_begin(len_old, a.bb);
  const int p1 = evict_end(len_old, a.tab.nnew[b], a.bb);
  const int p = p0 + e;
  if (p >= p1) return;
  const typename St::Bits* ring =
      (const typename St::Bits*)(role ? a.v_ring : a.k_ring) +
      (((int64_t)b * a.Hkv + h) * a.bb + (p % a.bb)) * kD;
  const typename St::Bits x0 = ring[2 * lane];
  const typename St::Bits x1 = ring[2 * lane + 1];
  const int k = a.tab.kact[role][b];
  const int64_t pbytes = page_bytes_of(Fmt<F>::kValBytes, k);
  char* page = (char*)(role ? a.v_pages : a.k_pages) + a.tab.page_off[role][b] +
               ((int64_t)h * a.n_pages_cap + p / kPage) * pbytes;
  select_and_pack<F>(x0, x1, k, page, p % kPage, lane);
}

// QG > 0 (decode steps): the key wave also rotates QG query rows, q_hat = q .
// P_QK[h] * qmult in float32.  Each output sums 4 quarters of 32 rows, each
// quarter in two accumulators (even and odd rows) that are added, and the
// quarters meet as (q0 + q1) + (q2 + q3): the order of qrot_kernel.
template <typename F, int TPW, int QG>
__global__ __launch_bounds__(64) void insert_kernel(CompressLaunch a) {
  using T = typename Fmt<F>::Elem;
  using St = Store<T>;
  static_assert(QG == 0 || TPW == 1, "query rotation: decode steps only");
  __shared__ __attribute__((aligned(16))) double xs[kD][TPW];
  __shared__ float qs[QG > 0 ? QG : 1][kD];
  const int lane = threadIdx.x;
  const int ngroups = (a.n_new + TPW - 1) / TPW;
  int w = blockIdx.x;
  const int grp = w % ngroups;
  w /= ngroups;
  const int role = w & 1;
  w >>= 1;
  const int h = w % a.Hkv;
  const int b = w / a.Hkv;
  const int t0 = grp * TPW;
  const int nnew = a.tab.nnew[b];
  if (t0 >= nnew) return;
  const int nt = (nnew - t0) < TPW ? (nnew - t0) : TPW;
  const T* x = (const T*)(role ? a.v_new : a.k_new) +
               (((int64_t)b * a.Hkv + h) * a.n_new + t0) * kD;
  for (int t = 0; t < TPW; ++t) {
    double v0 = 0.0, v1 = 0.0;
    if (t < nt) {
      v0 = (double)(float)x[(int64_t)t * kD + 2 * lane];
      v1 = (double)(float)x[(int64_t)t * kD + 2 * lane + 1];
    }
    xs[2 * lane][t] = v0;
    xs[2 * lane + 1][t] = v1;
  }
  const bool with_q = QG > 0 && role == 0;  // uniform
  const int64_t q0 = ((int64_t)b * a.Hq + (int64_t)h * QG) * kD;  // first query row
  if (with_q) {
#pragma unroll
    for (int g = 0; g < QG; ++g) {
      qs[g][2 * lane] = (float)((const T*)a.q)[q0 + g * kD + 2 * lane];
      qs[g][2 * lane + 1] = (float)((const T*)a.q)[q0 + g * kD + 2 * lane + 1];
    }
  }
  __syncthreads();
  double acc0[TPW], acc1[TPW];
  const float* Prole = role ? a.P_vo : a.P_qk;
  if (!Prole) {  // values already in the rotated basis (P_VO absorbed into W_V)
#pragma unroll
    for (int t = 0; t < TPW; ++t) {
      acc0[t] = xs[2 * lane][t];
      acc1[t] = xs[2 * lane + 1][t];
    }
  } else {
    const float2* P = (const float2*)(Prole + (int64_t)h * kD * kD) + lane;
#pragma unroll
    for (int t = 0; t < TPW; ++t) acc0[t] = acc1[t] = 0.0;
    // 32 rows of P in flight per batch: the loads are the latency of this kernel
    auto rows = [&](auto wq) {
      constexpr bool kQ = decltype(wq)::value && QG > 0;
      constexpr int NQ = kQ ? QG : 1;
      float qa[NQ][2][8];  // [query head][output dim 2 lane + o][2 quarter + row parity]
#pragma unroll
      for (int g = 0; g < NQ; ++g)
#pragma unroll
        for (int c = 0; c < 8; ++c) qa[g][0][c] = qa[g][1][c] = 0.f;
#pragma unroll
      for (int qt = 0; qt < 4; ++qt) {
#pragma unroll 32
        for (int u = 0; u < 32; ++u) {
          const int i = 32 * qt + u;
          const float2 pr = P[i * (kD / 2)];
          const double p0 = (double)pr.x, p1 = (double)pr.y;
#pragma unroll
          for (int t = 0; t < TPW; ++t) {
            const double xv = xs[i][t];
            acc0[t] = fma(xv, p0, acc0[t]);
            acc1[t] = fma(xv, p1, acc1[t]);
          }
          if constexpr (kQ) {
#pragma unroll
            for (int g = 0; g < QG; ++g) {
              const float qv = qs[g][i];
              qa[g][0][2 * qt + (u & 1)] = fmaf(qv, pr.x, qa[g][0][2 * qt + (u & 1)]);
              qa[g][1][2 * qt + (u & 1)] = fmaf(qv, pr.y, qa[g][1][2 * qt + (u & 1)]);
            }
          }
        }
      }
      if constexpr (kQ) {
#pragma unroll
        for (int g = 0; g < QG; ++g)
#pragma unroll
          for (int o = 0; o < 2; ++o) {
            const float s0 = qa[g][o][0] + qa[g][o][1], s1 = qa[g][o][2] + qa[g][o][3];
            const float s2 = qa[g][o][4] + qa[g][o][5], s3 = qa[g][o][6] + qa[g][o][7];
            a.qhat[q0 + g * kD + 2 * lane + o] = ((s0 + s1) + (s2 + s3)) * a.qmult;
          }
      }
    };
    if (with_q)
      rows(std::true_type{});
    else
      rows(std::false_type{});
  }
  const int len_old = a.tab.len[b];
  const int len_new = len_old + nnew;
  const int k = a.tab.kact[role][b];
  const int64_t pbytes = page_bytes_of(Fmt<F>::kValBytes, k);
  char* pages = (char*)(role ? a.v_pages : a.k_pages) + a.tab.page_off[role][b] +
                (int64_t)h * a.n_pages_cap * pbytes;
  typename St::Bits* ring = (typename St::Bits*)(role ? a.v_ring : a.k_ring) +
                            ((int64_t)b * a.Hkv + h) * a.bb * kD;
  if constexpr (TPW == 1) {
    // one new token: the vector that leaves the buffer (if any) sits in the
    // ring slot the new token takes; prune and pack it first (each lane reads
    // the two elements it overwrites below)
    const int p0 = evict_begin(len_old, a.bb);
    if (p0 < evict_end(len_old, nnew, a.bb)) {
      const typename St::Bits* old = ring + (int64_t)(p0 % a.bb) * kD;
      const typename St::Bits o0 = old[2 * lane];
      const typename St::Bits o1 = old[2 * lane + 1];
      select_and_pack<F>(o0, o1, k, pages + (int64_t)(p0 / kPage) * pbytes, p0 % kPage, lane);
    }
  }
#pragma unroll
  for (int t = 0; t < TPW; ++t) {
    if (t >= nt) break;
    const typename St::Bits y0 = St::from_f64(acc0[t]);
    const typename St::Bits y1 = St::from_f64(acc1[t]);
    const int pos = len_old + t0 + t;
    if (pos >= len_new - a.bb) {  // stays dense: ring slot pos % b
      typename St::Bits* r = ring + (int64_t)(pos % a.bb) * kD;
      r[2 * lane] = y0;
      r[2 * lane + 1] = y1;
    } else {  // pruned on arrival
      select_and_pack<F>(y0, y1, k, pages + (int64_t)(pos / kPage) * pbytes, pos % kPage, lane);
    }
  }
}

template <typename F>
static hipError_t launch_compress_t(const CompressLaunch& a) {
  const int units = a.B * a.Hkv * 2;
  if (a.n_new == 1) {  // a decode step: eviction and insertion in one launch
    switch (a.q ? a.Hq / a.Hkv : 0) {
      case 0:
        hipLaunchKernelGGL((insert_kernel<F, 1, 0>), dim3(units), dim3(64), 0, a.stream, a);
        break;
      case 1:
        hipLaunchKernelGGL((insert_kernel<F, 1, 1>), dim3(units), dim3(64), 0, a.stream, a);
        break;
      case 2:
        hipLaunchKernelGGL((insert_kernel<F, 1, 2>), dim3(units), dim3(64), 0, a.stream, a);
        break;
      case 3:
        hipLaunchKernelGGL((insert_kernel<F, 1, 3>), dim3(units), dim3(64), 0, a.stream, a);
        break;
      case 4:
        hipLaunchKernelGGL((insert_kernel<F, 1, 4>), dim3(units), dim3(64), 0, a.stream, a);
        break;
      default:
        return hipErrorInvalidValue;  // the caller rotates more query heads per kv head itself
    }
    return hipGetLastError();
  }
  if (a.max_evict > 0) {
    hipLaunchKernelGGL(evict_kernel<F>, dim3(units * a.max_evict), dim3(64), 0, a.stream, a);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (a.n_new >= kPrefillMinTokens && sizeof(typename Fmt<F>::Elem) == 2) return launch_prefill(a);
  if (a.n_new > 0) {
    const int ngroups = (a.n_new + kTPW - 1) / kTPW;
    hipLaunchKernelGGL((insert_kernel<F, kTPW, 0>), dim3((int64_t)units * ngroups), dim3(64), 0,
                       a.stream, a);
    return hipGetLastError();
  }
  return hipSuccess;
}

hipError_t launch_compress(const CompressLaunch& a) {
  if (a.dtype == SWAN_F16) return launch_compress_t<_Float16>(a);
  if (a.dtype == SWAN_F16_E4M3) return launch_compress_t<E4M3V>(a);
  return launch_compress_t<float>(a);
}

}  // namespace swan
