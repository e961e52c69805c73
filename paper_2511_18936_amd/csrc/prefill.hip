// Compress-append of many tokens at once (prefill), fp16 storage (sparse
// values fp16 or E4M3).
//
// Same result as token-by-token Algorithm 1 (and as insert_kernel): each new
// key/value is rotated exactly (float64 products and sums) and rounded once
// to fp16; tokens that stay in the buffer go to their ring slot, the others
// are pruned to their top-k magnitudes (ties: lower index) and packed.
//
// One wave handles 64-position blocks of one (sequence, kv head, role):
//   rotation   on MFMA in float64 (v_mfma_f64_16x16x4f64): 16 tokens x 32
//              output dims per pass, the contraction dim permuted so that a
//              lane reads 32 contiguous input values of its token row; the
//              lane's B operands (its 2 x 32 entries of P for one quarter of
//              the output dims) are held in registers across the block's 4
//              passes of 16 tokens
//   selection  one token per lane on its 128 stored values: a radix select
//              on bit planes of the magnitudes finds the k-th largest, then
//              one in-order pass emits the kept pairs (and the padding) into
//              an LDS copy of the page
//   output     each lane stores its own 16-byte slot chunks of the page (a
//              wave store is 1 KiB contiguous), or its dense row to the ring
#include <type_traits>

#include "swan_device.h"
#include "swan_internal.h"

namespace swan {

typedef double d4 __attribute__((ext_vector_type(4)));

constexpr int kRowHalves = 136;                // LDS row of one token's 128 fp16 values (+ pad)
constexpr int kPrefillBlocksPerWave = 4;       // 64-position blocks per wave
constexpr int kXcds = 8;                       // MI355X: 8 XCDs, each with its own L2
constexpr int kStageBytes = 64 * kRowHalves * 2;  // the rows, then the page copy
// a page (64 * k_pad * 3 bytes) fits the copy up to k_pad 88; above, values and
// indices are emitted and stored in two rounds

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

// k-th largest of the 128 fp16 magnitudes in v (two per dword), and how many
// elements equal to it are kept (the rest of the k are strictly larger).
// Radix select on bit planes: the magnitudes of each 32-element chunk c are
// transposed so that pl[b][c] holds bit b of each element (bits 0-15: the
// chunk's even elements, 16-31: its odd ones); from the top bit down, the
// candidates still equal to the threshold prefix are split by the next bit.
__device__ __forceinline__ void kth_magnitude(const uint32_t* v, int k, uint32_t& tau,
                                              int& need_eq) {
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
  uint32_t eq[4] = {~0u, ~0u, ~0u, ~0u};
  int gt = 0;
  uint32_t t = 0;
#pragma unroll
  for (int b = 14; b >= 0; --b) {
    uint32_t hi[4];
    int cnt = 0;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      hi[c] = eq[c] & pl[b][c];
      cnt += __popc(hi[c]);
    }
    const bool one = gt + cnt >= k;  // the k-th largest has this bit set
    t |= one ? (1u << b) : 0u;
    gt += one ? 0 : cnt;
#pragma unroll
    for (int c = 0; c < 4; ++c) eq[c] = one ? hi[c] : (eq[c] & ~pl[b][c]);
  }
  tau = t;
  need_eq = k - gt;
}

// One token per lane: its kept (value, index) pairs in ascending index
// order, then the padding (value +0 at the lowest unselected dims), written
// into the LDS page copy at the lane's offsets: values [kp/8][64][CB] at sv
// (fp16 bits, or their E4M3 codes), indices [kp/8][64][8 B] at si.
template <typename F, bool kVals, bool kIdx>
__device__ __forceinline__ void emit_slots(const uint32_t* v, uint32_t tau, int need_eq, int k,
                                           int npad, char* sv, uint8_t* si) {
  constexpr bool kE4M3 = std::is_same<F, E4M3V>::value;
  auto put = [&](int e, uint32_t hb) {
    if constexpr (kE4M3)
      ((uint8_t*)sv)[(e >> 3) * 512 + (e & 7)] = (uint8_t)f16_bits_to_e4m3(hb);
    else
      ((uint16_t*)sv)[(e >> 3) * 512 + (e & 7)] = (uint16_t)hb;
  };
  int e = 0, eq = 0, pad = 0;
#pragma unroll
  for (int j = 0; j < kD; ++j) {
    const uint32_t hb = (v[j >> 1] >> ((j & 1) * 16)) & 0xFFFFu;
    const uint32_t m = hb & 0x7FFFu;
    const bool tie = m == tau;
    const bool sel = m > tau || (tie && eq < need_eq);
    eq += tie ? 1 : 0;
    if (sel) {
      if (kVals) put(e, hb);
      if (kIdx) si[(e >> 3) * 512 + (e & 7)] = (uint8_t)j;
      ++e;
    } else if (pad < npad) {
      const int ep = k + pad;
      if (kVals) put(ep, 0u);
      if (kIdx) si[(ep >> 3) * 512 + (ep & 7)] = (uint8_t)j;
      ++pad;
    }
  }
}

template <typename F>
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(2, 2)))
void prefill_kernel(CompressLaunch a) {
  constexpr int VB = Fmt<F>::kValBytes, CB = Fmt<F>::kChunkBytes;
  __shared__ __attribute__((aligned(16))) char lds[kStageBytes];
  _Float16* rows = (_Float16*)lds;  // [64 tokens][kRowHalves], then reused as the page copy
  const int lane = threadIdx.x;
  const int q = lane >> 4, r16 = lane & 15;
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
  const int bbeg = blk0 + grp * kPrefillBlocksPerWave;
  if (bbeg > blk1) return;
  const int bend = min(bbeg + kPrefillBlocksPerWave, blk1 + 1);

  const _Float16* x = (const _Float16*)(role ? a.v_new : a.k_new) +
                      ((int64_t)b * a.Hkv + h) * a.n_new * kD;
  // NULL P_vo: values already in the rotated basis; the rotation is then by I
  const float* Prole = role ? a.P_vo : a.P_qk;
  const float* P = Prole ? Prole + (int64_t)h * kD * kD : nullptr;

  const int k = a.tab.kact[role][b];
  const int kp = kpad_of(k);
  const int64_t pbytes = page_bytes_of(VB, k);
  char* pages = (char*)(role ? a.v_pages : a.k_pages) + a.tab.page_off[role][b] +
                (int64_t)h * a.n_pages_cap * pbytes;
  uint16_t* ring = (uint16_t*)(role ? a.v_ring : a.k_ring) + ((int64_t)b * a.Hkv + h) * a.bb * kD;

  for (int blk = bbeg; blk < bend; ++blk) {
    const int pos0 = blk * kPage;
    // ---- rotation: 4 quarters of the output dims x 4 passes of 16 tokens,
    //      results rounded to fp16 into LDS rows ----
#pragma unroll 1
    for (int nh = 0; nh < 4; ++nh) {
      // B operands of this quarter: pb[nt][ks] = P[32 q + ks][32 nh + 16 nt + r16]
      float pb[2][32];
#pragma unroll
      for (int ks = 0; ks < 32; ++ks)
#pragma unroll
        for (int nt = 0; nt < 2; ++nt)
          pb[nt][ks] = P ? P[(32 * q + ks) * kD + 32 * nh + 16 * nt + r16]
                         : (32 * q + ks == 32 * nh + 16 * nt + r16 ? 1.f : 0.f);
#pragma unroll 1
      for (int mt = 0; mt < 4; ++mt) {
        const int tp0 = pos0 + 16 * mt - len_old;  // token index of the pass's first row
        if (tp0 + 15 < 0 || tp0 >= nnew) continue;  // no new token in this pass (uniform)
        // A operands: lane (q, r16) holds x[token 16 mt + r16][32 q .. 32 q + 31]
        u32x4 xv[4];
        {
          const int t = tp0 + r16;
          if (t >= 0 && t < nnew) {
            const u32x4* src = (const u32x4*)(x + (int64_t)t * kD + 32 * q);
#pragma unroll
            for (int c = 0; c < 4; ++c) xv[c] = src[c];
          } else {
#pragma unroll
            for (int c = 0; c < 4; ++c) xv[c] = u32x4{0u, 0u, 0u, 0u};
          }
        }
        d4 acc[2];
#pragma unroll
        for (int nt = 0; nt < 2; ++nt) acc[nt] = d4{0.0, 0.0, 0.0, 0.0};
#pragma unroll
        for (int ks = 0; ks < 32; ++ks) {
          const uint32_t wv = xv[ks >> 3][(ks >> 1) & 3];
          const double av = (double)f16_bits_to_f32((ks & 1) ? (wv >> 16) : (wv & 0xFFFFu));
#pragma unroll
          for (int nt = 0; nt < 2; ++nt)
          {
            float pv = pb[nt][ks];
            asm volatile("" : "+v"(pv));  // convert per use: as doubles pb would not fit
            acc[nt] = __builtin_amdgcn_mfma_f64_16x16x4f64(av, (double)pv, acc[nt], 0, 0, 0);
          }
        }
        // f64 MFMA result layout: register v of lane l holds D[l / 16 + 4 v][l % 16],
        // i.e. token row q + 4 v of the pass, output dim 32 nh + 16 nt + r16
#pragma unroll
        for (int nt = 0; nt < 2; ++nt)
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const uint16_t hb = f64_to_f16_bits_fast(acc[nt][v]);
            ((uint16_t*)rows)[(16 * mt + q + 4 * v) * kRowHalves + 32 * nh + 16 * nt + r16] = hb;
          }
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();

    // ---- one token per lane ----
    const int pos = pos0 + lane;
    const int t = pos - len_old;
    const bool mine = t >= 0 && t < nnew;
    const bool dense = pos >= len_new - a.bb;
    uint32_t v[64];
    if (mine) {
      const u32x4* rp = (const u32x4*)(rows + lane * kRowHalves);
#pragma unroll
      for (int c = 0; c < 16; ++c) {
        const u32x4 c4 = rp[c];
        v[4 * c] = c4.x;
        v[4 * c + 1] = c4.y;
        v[4 * c + 2] = c4.z;
        v[4 * c + 3] = c4.w;
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();
    if (mine && dense) {  // stays in the buffer: ring slot pos % b
      u32x4* dst = (u32x4*)(ring + (int64_t)(pos % a.bb) * kD);
#pragma unroll
      for (int c = 0; c < 16; ++c) dst[c] = u32x4{v[4 * c], v[4 * c + 1], v[4 * c + 2], v[4 * c + 3]};
    }
    const bool sparse = mine && !dense;
    // uniform; never for one-byte values (64 * 128 * 2 bytes fit)
    const bool two_rounds = VB > 1 && 64 * kp * (VB + 1) > kStageBytes;
    const int vregion = 64 * kp * VB;                            // value bytes of a page
    uint32_t tau_keep = 0;
    int need_keep = 0, npad = 0;
    if (sparse) {
      // k-th largest magnitude; ties at it are taken lowest dim first
      uint32_t tau;
      int need_eq;
      kth_magnitude(v, k, tau, need_eq);
      npad = kp - k;
      if (!two_rounds)
        emit_slots<F, true, true>(v, tau, need_eq, k, npad, lds + lane * CB,
                                  (uint8_t*)lds + vregion + lane * 8);
      else
        emit_slots<F, true, false>(v, tau, need_eq, k, npad, lds + lane * CB, nullptr);
      tau_keep = tau;
      need_keep = need_eq;
    }
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();
    char* page = pages + (int64_t)blk * pbytes;
    const int nch = kp >> 3;
    if (sparse) {  // this lane's slot chunks of the page
      for (int c = 0; c < nch; ++c) {
        if constexpr (CB == 16)
          *(u32x4*)(page + c * 1024 + lane * 16) = *(const u32x4*)(lds + c * 1024 + lane * 16);
        else
          *(u32x2*)(page + c * 512 + lane * 8) = *(const u32x2*)(lds + c * 512 + lane * 8);
      }
      if (!two_rounds)
        for (int c = 0; c < nch; ++c)
          *(u32x2*)(page + vregion + c * 512 + lane * 8) =
              *(const u32x2*)(lds + vregion + c * 512 + lane * 8);
    }
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();
    if (two_rounds) {  // indices: the same selection again, then their chunks
      if (sparse)
        emit_slots<F, false, true>(v, tau_keep, need_keep, k, npad, nullptr,
                                   (uint8_t*)lds + lane * 8);
      __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
      __builtin_amdgcn_wave_barrier();
      if (sparse)
        for (int c = 0; c < nch; ++c)
          *(u32x2*)(page + vregion + c * 512 + lane * 8) =
              *(const u32x2*)(lds + c * 512 + lane * 8);
      __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
      __builtin_amdgcn_wave_barrier();
    }
  }
}

int prefill_groups(int max_new_tokens, int min_len_old) {
  (void)min_len_old;
  const int max_blocks = (max_new_tokens + kPage - 1) / kPage + 1;
  return (max_blocks + kPrefillBlocksPerWave - 1) / kPrefillBlocksPerWave;
}

hipError_t launch_prefill(const CompressLaunch& a) {
  const int pairs = (2 * a.Hkv + kXcds - 1) / kXcds * kXcds;  // (head, role), padded
  const dim3 grid((int64_t)pairs * a.B * a.prefill_groups);
  if (a.dtype == SWAN_F16_E4M3)
    hipLaunchKernelGGL(prefill_kernel<E4M3V>, grid, dim3(64), 0, a.stream, a);
  else
    hipLaunchKernelGGL(prefill_kernel<_Float16>, grid, dim3(64), 0, a.stream, a);
  return hipGetLastError();
}

}  // namespace swan
