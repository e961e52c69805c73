// Compress-append (Algorithm 1, the steps that project, append, evict and
// prune).
//
// Several new tokens per sequence: two launches on the caller's stream, so
// that every vector leaving the ring is read before a new token overwrites its
// slot.  One new token (a decode step): one launch, step_kernel, which evicts
// the slot's old vector before it writes the new one.
//   evict_kernel   one wave per ring vector that leaves the buffer: top-k of
//                  its stored values, packed into its page slot
//   insert_kernel  one wave per group of kTPW new tokens of one (sequence, kv
//                  head, role): rotation x . P accumulated in float64 and
//                  rounded once to the storage type; tokens still inside the
//                  buffer go to their ring slot, the others are pruned and
//                  packed at once
//   step_kernel    a decode step: one workgroup of four waves per (sequence,
//                  kv head, role), each wave a quarter of P's rows; the same
//                  rounding, ring write or pruning, and the eviction.  In
//                  swan_decode_step the key workgroup also rotates the step's
//                  queries of its kv head (q_hat for the attention that
//                  follows) with the same rows of P_QK
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

template <typename F, int TPW>
__global__ __launch_bounds__(64) void insert_kernel(CompressLaunch a) {
  using T = typename Fmt<F>::Elem;
  using St = Store<T>;
  __shared__ __attribute__((aligned(16))) double xs[kD][TPW];
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
#pragma unroll 32
    for (int i = 0; i < kD; ++i) {
      const float2 pr = P[i * (kD / 2)];
      const double p0 = (double)pr.x, p1 = (double)pr.y;
#pragma unroll
      for (int t = 0; t < TPW; ++t) {
        const double xv = xs[i][t];
        acc0[t] = fma(xv, p0, acc0[t]);
        acc1[t] = fma(xv, p1, acc1[t]);
      }
    }
  }
  const int len_old = a.tab.len[b];
  const int len_new = len_old + nnew;
  const int k = a.tab.kact[role][b];
  const int64_t pbytes = page_bytes_of(Fmt<F>::kValBytes, k);
  char* pages = (char*)(role ? a.v_pages : a.k_pages) + a.tab.page_off[role][b] +
                (int64_t)h * a.n_pages_cap * pbytes;
  typename St::Bits* ring = (typename St::Bits*)(role ? a.v_ring : a.k_ring) +
                            ((int64_t)b * a.Hkv + h) * a.bb * kD;
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

// A decode step's append, one new token per sequence: one workgroup of four
// waves per (sequence, kv head, role).  Wave s rotates with rows 32 s .. 32 s
// + 31 of P, its 32 row loads issued together, so the rotation costs one
// memory latency rather than a wave's walk over all 128 rows; the four
// float64 partials meet in LDS as (s0 + s1) + (s2 + s3), and wave 0 rounds the
// sum once and writes the ring slot (or, with no buffer, prunes and packs the
// token), after it has pruned and packed the vector that leaves the buffer
// from that same slot.  QG > 0 (swan_decode_step): the key workgroup also
// rotates the QG query rows of its kv head, q_hat = q . P_QK[h] * qmult in
// float32, quarter s in wave s with even and odd rows in two accumulators
// that are added, the quarters meeting as (q0 + q1) + (q2 + q3): the order of
// qrot_kernel, so q_hat has the same bits as from that kernel.
template <typename F, int QG>
__global__ __launch_bounds__(256) void step_kernel(CompressLaunch a) {
  using T = typename Fmt<F>::Elem;
  using St = Store<T>;
  constexpr int NQ = QG > 0 ? QG : 1;
  __shared__ double xs[kD];
  __shared__ double part[4][kD];
  __shared__ float qs[NQ][kD];
  __shared__ float qpart[NQ][4][kD];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  int w = blockIdx.x;
  const int role = w & 1;
  w >>= 1;
  const int h = w % a.Hkv;
  const int b = w / a.Hkv;
  if (a.tab.nnew[b] == 0) return;  // uniform over the workgroup
  const bool with_q = QG > 0 && role == 0;
  const T* x = (const T*)(role ? a.v_new : a.k_new) + ((int64_t)b * a.Hkv + h) * a.n_new * kD;
  const int64_t q0 = ((int64_t)b * a.Hq + (int64_t)h * NQ) * kD;  // first query row
  if (tid < kD) xs[tid] = (double)(float)x[tid];
  if (with_q)
    for (int i = tid; i < NQ * kD; i += 256) qs[i / kD][i % kD] = (float)((const T*)a.q)[q0 + i];
  const int len_old = a.tab.len[b];
  const int k = a.tab.kact[role][b];
  const int64_t pbytes = page_bytes_of(Fmt<F>::kValBytes, k);
  char* pages = (char*)(role ? a.v_pages : a.k_pages) + a.tab.page_off[role][b] +
                (int64_t)h * a.n_pages_cap * pbytes;
  typename St::Bits* ring = (typename St::Bits*)(role ? a.v_ring : a.k_ring) +
                            ((int64_t)b * a.Hkv + h) * a.bb * kD;
  const float* Prole = role ? a.P_vo : a.P_qk;
  float2 pr[32];
  if (Prole) {  // this wave's quarter of P: 32 rows in flight
    const float2* P = (const float2*)(Prole + (int64_t)h * kD * kD + (int64_t)(32 * wave) * kD) +
                      lane;
#pragma unroll
    for (int u = 0; u < 32; ++u) pr[u] = P[u * (kD / 2)];
  }
  // the vector that leaves the buffer (if any) sits in the ring slot the new
  // token takes: wave 0 prunes and packs it first (each lane reads the two
  // elements it overwrites below)
  const int p0 = evict_begin(len_old, a.bb);
  if (wave == 0 && p0 < evict_end(len_old, 1, a.bb)) {
    const typename St::Bits* old = ring + (int64_t)(p0 % a.bb) * kD;
    const typename St::Bits o0 = old[2 * lane];
    const typename St::Bits o1 = old[2 * lane + 1];
    select_and_pack<F>(o0, o1, k, pages + (int64_t)(p0 / kPage) * pbytes, p0 % kPage, lane);
  }
  __syncthreads();  // xs and qs
  if (Prole) {
    double acc0 = 0.0, acc1 = 0.0;
#pragma unroll
    for (int u = 0; u < 32; ++u) {
      const double xv = xs[32 * wave + u];
      acc0 = fma(xv, (double)pr[u].x, acc0);
      acc1 = fma(xv, (double)pr[u].y, acc1);
    }
    part[wave][2 * lane] = acc0;
    part[wave][2 * lane + 1] = acc1;
    if (with_q) {
#pragma unroll
      for (int g = 0; g < NQ; ++g) {
        float e0 = 0.f, o0 = 0.f, e1 = 0.f, o1 = 0.f;  // [even / odd rows][output 2 lane + 0 / 1]
#pragma unroll
        for (int u = 0; u < 32; u += 2) {
          e0 = fmaf(qs[g][32 * wave + u], pr[u].x, e0);
          o0 = fmaf(qs[g][32 * wave + u + 1], pr[u + 1].x, o0);
          e1 = fmaf(qs[g][32 * wave + u], pr[u].y, e1);
          o1 = fmaf(qs[g][32 * wave + u + 1], pr[u + 1].y, o1);
        }
        qpart[g][wave][2 * lane] = e0 + o0;
        qpart[g][wave][2 * lane + 1] = e1 + o1;
      }
    }
  }
  __syncthreads();  // the partials
  if (wave == 0) {
    double y0 = xs[2 * lane], y1 = xs[2 * lane + 1];  // values already rotated (P_VO absorbed)
    if (Prole) {
      y0 = (part[0][2 * lane] + part[1][2 * lane]) + (part[2][2 * lane] + part[3][2 * lane]);
      y1 = (part[0][2 * lane + 1] + part[1][2 * lane + 1]) +
           (part[2][2 * lane + 1] + part[3][2 * lane + 1]);
    }
    const typename St::Bits v0 = St::from_f64(y0);
    const typename St::Bits v1 = St::from_f64(y1);
    const int pos = len_old;
    if (a.bb > 0) {  // stays dense: ring slot pos % b
      typename St::Bits* r = ring + (int64_t)(pos % a.bb) * kD;
      r[2 * lane] = v0;
      r[2 * lane + 1] = v1;
    } else {  // no buffer: pruned on arrival
      select_and_pack<F>(v0, v1, k, pages + (int64_t)(pos / kPage) * pbytes, pos % kPage, lane);
    }
  } else if (wave == 1 && with_q) {
    for (int i = lane; i < NQ * kD; i += 64) {
      const int g = i / kD, j = i % kD;
      a.qhat[q0 + i] =
          ((qpart[g][0][j] + qpart[g][1][j]) + (qpart[g][2][j] + qpart[g][3][j])) * a.qmult;
    }
  }
}

template <typename F>
static hipError_t launch_compress_t(const CompressLaunch& a) {
  const int units = a.B * a.Hkv * 2;
  if (a.n_new == 1) {  // a decode step: eviction and insertion in one launch
    const dim3 grid(units), block(256);
    switch (a.q ? a.Hq / a.Hkv : 0) {
      case 0:
        hipLaunchKernelGGL((step_kernel<F, 0>), grid, block, 0, a.stream, a);
        break;
      case 1:
        hipLaunchKernelGGL((step_kernel<F, 1>), grid, block, 0, a.stream, a);
        break;
      case 2:
        hipLaunchKernelGGL((step_kernel<F, 2>), grid, block, 0, a.stream, a);
        break;
      case 3:
        hipLaunchKernelGGL((step_kernel<F, 3>), grid, block, 0, a.stream, a);
        break;
      case 4:
        hipLaunchKernelGGL((step_kernel<F, 4>), grid, block, 0, a.stream, a);
        break;
      case 5:
        hipLaunchKernelGGL((step_kernel<F, 5>), grid, block, 0, a.stream, a);
        break;
      case 6:
        hipLaunchKernelGGL((step_kernel<F, 6>), grid, block, 0, a.stream, a);
        break;
      case 7:
        hipLaunchKernelGGL((step_kernel<F, 7>), grid, block, 0, a.stream, a);
        break;
      case 8:
        hipLaunchKernelGGL((step_kernel<F, 8>), grid, block, 0, a.stream, a);
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
    hipLaunchKernelGGL((insert_kernel<F, kTPW>), dim3((int64_t)units * ngroups), dim3(64), 0,
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
