// Decode attention on the hybrid SWAN cache (Algorithm 1, attention part).
//
// Launches, in order on the caller's stream:
//   qrot_kernel    q_hat = q . P_QK[g], pre-multiplied by scale * log2(e)
//   attn_kernel    one wave per (sequence, query head, token split) over the
//                  sparse pages, plus one wave per (sequence, query head) over
//                  the dense buffer; each writes a partial (m, l, acc[128]) in
//                  the rotated space.  On the fp16 formats a batch with
//                  several k_pad takes one launch of attn_fused_kernel
//                  (decode_fused.hip), each wave specialised on its own
//                  sequence's k_pad.  Otherwise one launch per distinct k_pad
//                  of the batch; several run side by side on library-owned
//                  streams of the calling thread, joined back before the
//                  merge.  For fp16 GQA the launch is attn_gqa_kernel
//                  (decode_gqa.h) instead, one workgroup per KV stream for
//                  several query heads.  Sequences whose keys and
//                  values have different k_pad run the same kernels specialised
//                  on the larger k_pad (decode_asym.hip, decode_gqa_asym.hip).
//   merge_kernel   log-sum-exp merge of the partials, then o = o_hat . P_VO^T
//                  (the inverse rotation that Sec. 4.2 absorbs into W_O)
// The sparse attention wave itself is described in decode_mha.h.
#include "decode_mha.h"

namespace swan {

// ---------------------------------------------------------------------------
// q rotation: q_hat[b][h][j] = mult * sum_i q[b][h][i] * P_qk[g][i][j]
// 512 threads per (b, h): thread (j, s) sums rows i = 32 s .. 32 s + 31 (two
// independent accumulators, 32 loads in flight), the four quarters meet in LDS
// ---------------------------------------------------------------------------
constexpr int kRotQuarters = 4;
template <typename T>
__global__ __launch_bounds__(kD * kRotQuarters) void qrot_kernel(const T* __restrict__ q,
                                                                 const float* __restrict__ Pqk,
                                                                 float* __restrict__ qhat, int Hq,
                                                                 int G, float mult) {
  __shared__ float qs[kD];
  __shared__ float part[kRotQuarters][kD];
  const int bh = blockIdx.x;
  const int g = (bh % Hq) / G;
  const int j = threadIdx.x & (kD - 1), sq = threadIdx.x / kD;
  if (sq == 0) qs[j] = (float)q[(int64_t)bh * kD + j];
  __syncthreads();
  const float* P = Pqk + (int64_t)g * kD * kD + (int64_t)(32 * sq) * kD + j;
  float a0 = 0.f, a1 = 0.f;
#pragma unroll
  for (int i = 0; i < 32; i += 2) {
    a0 = fmaf(qs[32 * sq + i], P[i * kD], a0);
    a1 = fmaf(qs[32 * sq + i + 1], P[(i + 1) * kD], a1);
  }
  part[sq][j] = a0 + a1;
  __syncthreads();
  if (sq == 0)
    qhat[(int64_t)bh * kD + j] = ((part[0][j] + part[1][j]) + (part[2][j] + part[3][j])) * mult;
}

// ---------------------------------------------------------------------------
// merge partials (log-sum-exp, fixed order) and rotate back: o = o_hat . P_vo^T
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(128) void merge_kernel(DecodeLaunch a) {
  __shared__ float oh[kD];
  __shared__ float wts[kMaxSplits + 1];
  __shared__ float red[4];
  const int bhq = blockIdx.x;
  const int b = bhq / a.Hq, hq = bhq % a.Hq, h = hq / (a.Hq / a.Hkv);
  const int t = threadIdx.x;
  const int L = a.tab.len[b];
  const int S = L > a.bb ? L - a.bb : 0;
  const int np = pages_for(S);
  const int nsg = a.tab.nsplit[b];
  const int ns = np < nsg ? np : nsg;
  const bool has_buf = (L < a.bb ? L : a.bb) > 0;
  const float* part = a.part + (int64_t)bhq * (a.n_splits + 1) * kPartFloats;
  // partial i < ns is split i; partial ns stands for the buffer (slot n_splits)
  const int np_all = ns + (has_buf ? 1 : 0);
  auto slot = [&](int i) { return i < ns ? i : a.n_splits; };
  float mloc = -INFINITY;
  for (int i = t; i < np_all; i += 128) mloc = fmaxf(mloc, part[slot(i) * kPartFloats]);
  mloc = wave_max(mloc);
  if ((t & 63) == 0) red[t >> 6] = mloc;
  __syncthreads();
  const float m = fmaxf(red[0], red[1]);
  float lloc = 0.f;
  for (int i = t; i < np_all; i += 128) {
    const float* pi = part + slot(i) * kPartFloats;
    const float wgt = exp2f(pi[0] - m);
    wts[i] = wgt;
    lloc += wgt * pi[1];
  }
  lloc = wave_sum(lloc);
  if ((t & 63) == 0) red[2 + (t >> 6)] = lloc;
  __syncthreads();
  const float inv = 1.f / (red[2] + red[3]);
  float o = 0.f;
  for (int i = 0; i < np_all; ++i) o = fmaf(wts[i], part[slot(i) * kPartFloats + 4 + t], o);
  oh[t] = o * inv;
  if (!a.P_vo) {  // the output stays in the rotated basis (P_VO absorbed into W_O)
    ((T*)a.out)[(int64_t)bhq * kD + t] = (T)oh[t];
    return;
  }
  __syncthreads();
  const float4* P = (const float4*)(a.P_vo + ((int64_t)h * kD + t) * kD);
  float r = 0.f;
#pragma unroll 8
  for (int j4 = 0; j4 < kD / 4; ++j4) {
    const float4 p = P[j4];
    r = fmaf(p.x, oh[4 * j4], r);
    r = fmaf(p.y, oh[4 * j4 + 1], r);
    r = fmaf(p.z, oh[4 * j4 + 2], r);
    r = fmaf(p.w, oh[4 * j4 + 3], r);
  }
  ((T*)a.out)[(int64_t)bhq * kD + t] = (T)r;
}

template <typename T, int KP8>
static hipError_t launch_attn(const DecodeLaunch& a, const SeqGroup& g) {
  const dim3 grid(g.n * a.Hq * (g.n_splits + 1));
  hipLaunchKernelGGL((attn_kernel<T, KP8, false>), grid, dim3(64), 0, a.stream, a, g);
  return hipGetLastError();
}

template <typename T>
static hipError_t launch_group(const DecodeLaunch& a, const SeqGroup& g, int kp8) {
  if (decode_heads_per_wave(a.dtype, a.Hq, a.Hkv) > 1) return launch_attn_gqa(a, g, kp8);
  switch (kp8) {
#define SWAN_KP8_CASE(n) \
  case n:                \
    return launch_attn<T, n>(a, g);
    SWAN_KP8_CASE(1) SWAN_KP8_CASE(2) SWAN_KP8_CASE(3) SWAN_KP8_CASE(4)
    SWAN_KP8_CASE(5) SWAN_KP8_CASE(6) SWAN_KP8_CASE(7) SWAN_KP8_CASE(8)
    SWAN_KP8_CASE(9) SWAN_KP8_CASE(10) SWAN_KP8_CASE(11) SWAN_KP8_CASE(12)
    SWAN_KP8_CASE(13) SWAN_KP8_CASE(14) SWAN_KP8_CASE(15) SWAN_KP8_CASE(16)
#undef SWAN_KP8_CASE
    default:
      return hipErrorInvalidValue;
  }
}

// Side streams of one device and thread for the attention launches of a
// batch that mixes page formats: the launches are independent (disjoint
// sequences), so running them side by side overlaps each one's ramp-up and
// tail.  Default priority.  Each thread has its own, so that callers on other
// threads (and streams) never wait on each other through them.
struct SideStreams {
  bool tried, ok;
  hipStream_t s[kSideStreams];
  hipEvent_t fork, join[kSideStreams];
};

// The calling thread's side streams on the current device, or NULL (launch on
// the caller's stream alone) when they cannot be made or `caller` belongs to
// another device.
static SideStreams* side_streams(hipStream_t caller) {
  static thread_local SideStreams per_device[kMaxDevices];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  if (caller) {
    hipDevice_t sdev = -1;
    if (hipStreamGetDevice(caller, &sdev) != hipSuccess || sdev != dev) return nullptr;
  }
  SideStreams* ss = &per_device[dev];
  if (!ss->tried) {
    ss->tried = true;
    bool ok = hipEventCreateWithFlags(&ss->fork, hipEventDisableTiming) == hipSuccess;
    for (int i = 0; ok && i < kSideStreams; ++i)
      ok = hipStreamCreateWithFlags(&ss->s[i], hipStreamNonBlocking) == hipSuccess &&
           hipEventCreateWithFlags(&ss->join[i], hipEventDisableTiming) == hipSuccess;
    ss->ok = ok;
  }
  return ss->ok ? ss : nullptr;
}

template <typename T>
static hipError_t launch_decode_t(const DecodeLaunch& a) {
  const int BH = a.B * a.Hq;
  using E = typename Fmt<T>::Elem;
  hipError_t e;
  if (!a.qhat_ready) {
    hipLaunchKernelGGL(qrot_kernel<E>, dim3(BH), dim3(kD * kRotQuarters), 0, a.stream,
                       (const E*)a.q, a.P_qk, a.qhat, a.Hq, a.Hq / a.Hkv, a.qmult);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  if (a.prof_start && (e = hipEventRecord(a.prof_start, a.stream)) != hipSuccess) return e;
  // sequences grouped by (k_pad of the keys, k_pad of the values); then, from
  // the largest k_pad down, a group joins the launch before it when its k_pad
  // is at least kMergePct % of that launch's (two thirds: the spare groups then
  // add at most half again the compute of its pages, which the HBM time still
  // covers, and fewer launches share the GPU more evenly).  A launch whose
  // sequences all have its k_pad for both roles runs the kernels specialised
  // on it; any other runs the instances for different k_pad (spare groups) at
  // the launch's largest.
  SeqGroup groups[SWAN_MAX_BATCH];
  int kp8k[SWAN_MAX_BATCH], kp8v[SWAN_MAX_BATCH];
  uint32_t present[kD / 8 + 1] = {};  // bit v of present[k]: some sequence has (k, v)
  for (int b = 0; b < a.B; ++b)
    present[kpad_of(a.tab.kact[0][b]) / 8] |= 1u << (kpad_of(a.tab.kact[1][b]) / 8);
  int ng = 0;
  for (int pk = kD / 8; pk >= 1; --pk)
    for (int pv = kD / 8; pv >= 1; --pv) {
      if (!((present[pk] >> pv) & 1u)) continue;
      SeqGroup& g = groups[ng];
      g.n = 0;
      g.n_splits = 0;
      for (int b = 0; b < a.B; ++b)
        if (kpad_of(a.tab.kact[0][b]) / 8 == pk && kpad_of(a.tab.kact[1][b]) / 8 == pv) {
          g.seq[g.n++] = b;
          g.n_splits = a.tab.nsplit[b] > g.n_splits ? a.tab.nsplit[b] : g.n_splits;
        }
      kp8k[ng] = pk;
      kp8v[ng] = pv;
      ++ng;
    }
  if (ng > 1 && decode_heads_per_wave(a.dtype, a.Hq, a.Hkv) == 1 &&
      (a.dtype == SWAN_F16 || a.dtype == SWAN_F16_E4M3)) {
    // MHA, fp16 storage: one launch over every group, each sequence's waves
    // specialised on its own k_pad tier, larger k_pad first
    FusedSeqs f;
    f.n = 0;
    f.n_splits = 0;
    bool taken[SWAN_MAX_BATCH] = {};
    for (int done = 0; done < ng; ++done) {
      int best = -1, bkp = 0;
      for (int i = 0; i < ng; ++i) {
        const int kp = kp8k[i] > kp8v[i] ? kp8k[i] : kp8v[i];
        if (!taken[i] && kp > bkp) {
          best = i;
          bkp = kp;
        }
      }
      taken[best] = true;
      for (int j = 0; j < groups[best].n; ++j) {
        f.seq[f.n] = groups[best].seq[j];
        f.kp8[f.n] = (int8_t)fused_tier(bkp);
        ++f.n;
      }
      if (groups[best].n_splits > f.n_splits) f.n_splits = groups[best].n_splits;
    }
    if ((e = launch_attn_fused(a, f)) != hipSuccess) return e;
    if (a.prof_stop && (e = hipEventRecord(a.prof_stop, a.stream)) != hipSuccess) return e;
    hipLaunchKernelGGL(merge_kernel<E>, dim3(BH), dim3(128), 0, a.stream, a);
    return hipGetLastError();
  }
  struct Launch {
    SeqGroup g;
    int kp8;
    bool sym;  // every sequence has k_pad 8 kp8 for keys and values
  };
  Launch ls[SWAN_MAX_BATCH];
  bool used[SWAN_MAX_BATCH] = {};
  int nl = 0;
  for (int done = 0; done < ng; ++done) {
    int best = -1, bkp = 0;  // the largest k_pad left (ties: first in group order)
    for (int i = 0; i < ng; ++i) {
      const int kp = kp8k[i] > kp8v[i] ? kp8k[i] : kp8v[i];
      if (!used[i] && kp > bkp) {
        best = i;
        bkp = kp;
      }
    }
    used[best] = true;
    const bool sym = kp8k[best] == kp8v[best];
    if (nl > 0 && a.merge_pct > 0 && bkp * 100 >= ls[nl - 1].kp8 * a.merge_pct) {
      Launch& l = ls[nl - 1];
      for (int j = 0; j < groups[best].n; ++j) l.g.seq[l.g.n++] = groups[best].seq[j];
      if (groups[best].n_splits > l.g.n_splits) l.g.n_splits = groups[best].n_splits;
      l.sym = false;
    } else {
      ls[nl].g = groups[best];
      ls[nl].kp8 = bkp;
      ls[nl].sym = sym;
      ++nl;
    }
  }
  auto launch_one = [&](const DecodeLaunch& ai, int i) {
    if (ls[i].sym) return launch_group<T>(ai, ls[i].g, ls[i].kp8);
    return decode_heads_per_wave(ai.dtype, ai.Hq, ai.Hkv) > 1
               ? launch_attn_gqa_asym(ai, ls[i].g, ls[i].kp8)
               : launch_attn_asym(ai, ls[i].g, ls[i].kp8);
  };
  SideStreams* ss = nl > 1 && a.side_streams > 0 ? side_streams(a.stream) : nullptr;
  if (!ss) {  // one launch, or no side streams: back to back on the caller's stream
    for (int i = 0; i < nl; ++i)
      if ((e = launch_one(a, i)) != hipSuccess) return e;
  } else {
    const int nmax = a.side_streams < kSideStreams ? a.side_streams : kSideStreams;
    const int nside = nl - 1 < nmax ? nl - 1 : nmax;
    if ((e = hipEventRecord(ss->fork, a.stream)) != hipSuccess) return e;
    for (int j = 0; j < nside; ++j)
      if ((e = hipStreamWaitEvent(ss->s[j], ss->fork, 0)) != hipSuccess) return e;
    for (int i = 0; i < nl; ++i) {
      DecodeLaunch ai = a;
      const int lane = i % (nside + 1);  // 0: the caller's stream
      if (lane > 0) ai.stream = ss->s[lane - 1];
      if ((e = launch_one(ai, i)) != hipSuccess) return e;
    }
    for (int j = 0; j < nside; ++j) {
      if ((e = hipEventRecord(ss->join[j], ss->s[j])) != hipSuccess) return e;
      if ((e = hipStreamWaitEvent(a.stream, ss->join[j], 0)) != hipSuccess) return e;
    }
  }
  if (a.prof_stop && (e = hipEventRecord(a.prof_stop, a.stream)) != hipSuccess) return e;
  hipLaunchKernelGGL(merge_kernel<E>, dim3(BH), dim3(128), 0, a.stream, a);
  return hipGetLastError();
}

hipError_t launch_decode(const DecodeLaunch& a) {
  if (a.dtype == SWAN_F16) return launch_decode_t<_Float16>(a);
  if (a.dtype == SWAN_F16_E4M3) return launch_decode_t<E4M3V>(a);
  return launch_decode_t<float>(a);
}

}  // namespace swan
