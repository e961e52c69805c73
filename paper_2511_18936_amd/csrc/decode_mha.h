// The MHA sparse attention wave and its kernel (Algorithm 1, attention part),
// shared by the launches for equal and for different key / value k_pad.
//
// Sparse wave: one token per lane.  The rotated query is replicated 8 times in
// LDS (q_rep[dim][8]) so that the gathers q_hat[idx] of 8 consecutive lanes
// fall on distinct banks; the value accumulator is lane-private, acc[dim][64]
// in LDS: a token's indices are distinct, so each page's update is a plain
// read-modify-write with all reads issued before the writes.  Pages of keys
// and values are streamed with coalesced nontemporal loads, the page after
// next in flight while the current one is consumed.  The softmax reference m
// is the first page's maximum and is only raised (with a rescale of acc) when
// a score exceeds it by more than kTau in log2 units (one ballot per page), so
// exponentials stay bounded by 2^kTau while rescales are rare.
#pragma once

#include "decode_common.h"

namespace swan {

template <typename T, int KP8>
__device__ __forceinline__ void process_page(const PageRegs<T, KP8>& kr, const PageRegs<T, KP8>& vr,
                                             bool valid, const float* qrep_l, float* acc_l,
                                             float* acc, int lane, SoftmaxState& st) {
  const float s = valid ? page_score<T, KP8>(kr, qrep_l) : -INFINITY;
  // the reference m only moves when a score passes m + kTau: one ballot per
  // page, a wave max only on the first page and on the rare raise
  if (st.first) {
    st.m = wave_max(s);
    st.first = false;
  } else if (__ballot(s > st.m + kTau) != 0) {
    const float pm = wave_max(s);
    const float f = exp2f(st.m - pm);
    rescale_acc(acc, lane, f);
    st.l *= f;
    st.m = pm;
  }
  const float p = valid ? exp2f(s - st.m) : 0.f;
  st.l += p;
  page_accumulate<T, KP8>(vr, acc_l, p, valid);
}

// The key and value pages of one (sequence, kv head): first page, page bytes
// and active groups of each role.
struct UnitPages {
  const char* kbase;
  const char* vbase;
  int64_t kbytes, vbytes;
  int nk8, nv8;
};

// One wave: pages [pbeg, pend) of one (sequence, kv head), for one query head.
// The next page is always loaded so that no load sits under a branch and the
// compiler can keep one page in flight; past the split's last page that load
// reads the small resident spare arrays instead (n8 = 0: value 0, index
// kSpareRow), which stay in cache, and its registers are never used.
// pipeline depth by the register footprint of a page (16-byte chunks per lane):
// two register sets (one page in flight while one is consumed) up to 12
template <typename T, int KP8>
constexpr bool two_page_sets() {
  return KP8 * PageRegs<T, KP8>::VCH <= 12;
}

// sparse_split's first key and value page, loaded before the caller fills its
// LDS (q replicas, zeroed accumulators) so that the load latency overlaps that
template <typename T, int KP8>
struct FirstPage {
  PageRegs<T, KP8> k, v;
};

template <typename T, int KP8>
__device__ void sparse_split(const UnitPages& u, int pbeg, int pend, int S, float* qrep,
                             float* acc, int lane, float* __restrict__ part,
                             FirstPage<T, KP8>& first) {
  const float* qrep_l = qrep + (lane & (kQRep - 1));
  float* acc_l = acc + (lane & (kAccCols - 1));
  SoftmaxState st{0.f, 0.f, true};
  if constexpr (two_page_sets<T, KP8>()) {
    PageRegs<T, KP8>& ka = first.k;
    PageRegs<T, KP8>& va = first.v;
    PageRegs<T, KP8> kb, vb;
    const int plast = pend - 1;
    for (int p = pbeg; p < pend; p += 2) {
      const bool in1 = p + 1 <= plast;  // uniform
      const int p1 = in1 ? p + 1 : plast;
      load_page<T, KP8>(kb, u.kbase + p1 * u.kbytes, lane, in1 ? u.nk8 : 0);
      load_page<T, KP8>(vb, u.vbase + p1 * u.vbytes, lane, in1 ? u.nv8 : 0);
      process_page<T, KP8>(ka, va, p * kPage + lane < S, qrep_l, acc_l, acc, lane, st);
      const bool in2 = p + 2 <= plast;
      const int p2 = in2 ? p + 2 : plast;
      load_page<T, KP8>(ka, u.kbase + p2 * u.kbytes, lane, in2 ? u.nk8 : 0);
      load_page<T, KP8>(va, u.vbase + p2 * u.vbytes, lane, in2 ? u.nv8 : 0);
      if (p + 1 < pend)
        process_page<T, KP8>(kb, vb, (p + 1) * kPage + lane < S, qrep_l, acc_l, acc, lane, st);
    }
  } else {  // large pages: one page at a time (the first one already loaded)
    PageRegs<T, KP8>& ka = first.k;
    PageRegs<T, KP8>& va = first.v;
    for (int p = pbeg; p < pend; ++p) {
      if (p > pbeg) {
        load_page<T, KP8>(ka, u.kbase + p * u.kbytes, lane, u.nk8);
        load_page<T, KP8>(va, u.vbase + p * u.vbytes, lane, u.nv8);
      }
      process_page<T, KP8>(ka, va, p * kPage + lane < S, qrep_l, acc_l, acc, lane, st);
    }
  }
  const float ltot = wave_sum(st.l);
  wave_lds_fence();
  reduce_acc(acc, lane, part);
  if (lane == 0) {
    part[0] = st.m;
    part[1] = ltot;
  }
}

// The dense-buffer wave of (sequence b, query head hq): its partial over the
// ring's tokens (slot n_splits).
template <typename T>
__device__ __forceinline__ void buffer_wave(const DecodeLaunch& a, int b, int hq, float* qrep,
                                            float* acc, int lane) {
  const int h = hq / (a.Hq / a.Hkv);
  const int bhq = b * a.Hq + hq;
  const int L = a.tab.len[b];
  const int nb = L < a.bb ? L : a.bb;
  if (nb == 0) return;
  const int64_t ring_off = ((int64_t)b * a.Hkv + h) * a.bb * kD;
  float* part = a.part + ((int64_t)bhq * (a.n_splits + 1) + a.n_splits) * kPartFloats;
  using E = typename Fmt<T>::Elem;
  buffer_part<E>((const E*)a.k_ring + ring_off, (const E*)a.v_ring + ring_off, nb,
                 a.qhat + (int64_t)bhq * kD, qrep, acc, lane, part);
}

// The sparse wave of (sequence b, query head hq, token split `split`) on pages
// of k_pad 8 KP8.  kAsym: keys and values may have a smaller k_pad than 8 KP8;
// each role's own k_pad then sets its page size and loaded groups at run time,
// the rest being spare groups (load_page), for which q_rep and acc have a
// spare row kSpareRow (qrep and acc hold kD + 1 rows).
template <typename T, int KP8, bool kAsym>
__device__ __forceinline__ void sparse_wave(const DecodeLaunch& a, int b, int hq, int split,
                                            float* qrep, float* acc, int lane) {
  const int h = hq / (a.Hq / a.Hkv);
  const int bhq = b * a.Hq + hq;
  const int L = a.tab.len[b];
  const int S = L > a.bb ? L - a.bb : 0;
  const int np = pages_for(S);
  const int nsb = a.tab.nsplit[b];
  const int ns = np < nsb ? np : nsb;
  if (split >= ns) return;
  const int pbeg = split_begin(split, ns, np, a.tab.flat[b] != 0);
  const int pend = split_begin(split + 1, ns, np, a.tab.flat[b] != 0);
  UnitPages u;
  u.kbytes = page_bytes_of(Fmt<T>::kValBytes, a.tab.kact[0][b]);
  u.vbytes = kAsym ? page_bytes_of(Fmt<T>::kValBytes, a.tab.kact[1][b]) : u.kbytes;
  u.nk8 = kAsym ? kpad_of(a.tab.kact[0][b]) / 8 : KP8;
  u.nv8 = kAsym ? kpad_of(a.tab.kact[1][b]) / 8 : KP8;
  u.kbase = (const char*)a.k_pages + a.tab.page_off[0][b] + (int64_t)h * a.n_pages_cap * u.kbytes;
  u.vbase = (const char*)a.v_pages + a.tab.page_off[1][b] + (int64_t)h * a.n_pages_cap * u.vbytes;
  float* part = a.part + ((int64_t)bhq * (a.n_splits + 1) + split) * kPartFloats;
  FirstPage<T, KP8> first;
  load_page<T, KP8>(first.k, u.kbase + pbeg * u.kbytes, lane, u.nk8);
  load_page<T, KP8>(first.v, u.vbase + pbeg * u.vbytes, lane, u.nv8);

  // replicate q_hat: q_rep[dim][8]; lane writes dims lane and lane + 64
  const float* qh = a.qhat + (int64_t)bhq * kD;
#pragma unroll
  for (int hh = 0; hh < 2; ++hh) {
    const int r = lane + 64 * hh;
    const float v = qh[r];
    float4* row = (float4*)(qrep + r * kQRep);
    row[0] = make_float4(v, v, v, v);
    row[1] = make_float4(v, v, v, v);
  }
  if (kAsym && lane < 2)  // the spare row's q is 0
    ((float4*)(qrep + kSpareRow * kQRep))[lane] = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll 8
  for (int c = 0; c < kAccCols / 2; ++c)
    ((float4*)acc)[c * 64 + lane] = make_float4(0.f, 0.f, 0.f, 0.f);
  wave_lds_fence();
  sparse_split<T, KP8>(u, pbeg, pend, S, qrep, acc, lane, part, first);
}

// One launch per distinct k_pad of the batch (KP8 = k_pad / 8), over the
// sequences g.seq[0..g.n) that use it (kAsym as in sparse_wave).
// Grid: n * Hq dense-buffer waves first, then n * Hq * g.n_splits sparse waves.
template <typename T, int KP8, bool kAsym>
__global__ __launch_bounds__(64) void attn_kernel(DecodeLaunch a, SeqGroup g) {
  constexpr int kRows = kAsym ? kD + 1 : kD;
  __shared__ __attribute__((aligned(16))) float qrep[kRows * kQRep];
  __shared__ __attribute__((aligned(16))) float acc[kRows * kAccCols];
  const int lane = threadIdx.x;
  const int GH = g.n * a.Hq;
  int w = blockIdx.x;
  if (w < GH) {  // dense-buffer wave
    buffer_wave<T>(a, g.seq[w / a.Hq], w % a.Hq, qrep, acc, lane);
    return;
  }
  w -= GH;
  const int gi = w % GH;
  sparse_wave<T, KP8, kAsym>(a, g.seq[gi / a.Hq], gi % a.Hq, w / GH, qrep, acc, lane);
}

}  // namespace swan
