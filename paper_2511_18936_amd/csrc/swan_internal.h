// Internal declarations shared by the libswan translation units (host + device).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "swan.h"

namespace swan {

constexpr int kD = 128;        // head dimension of the GPU path
constexpr int kPage = 64;      // tokens per page (one token per lane of a wave64)
constexpr int kMaxSplits = 256;
constexpr int kMaxRing = 4096; // largest dense buffer the decode kernel stages in LDS
constexpr int kPartFloats = 132;  // m, l, 2 pad, acc[128]

// Per-sequence parameters passed by value to every kernel (batch <= 64).
// Role 0 is the keys, role 1 the values: each has its own k and page layout.
struct SeqTab {
  int32_t len[SWAN_MAX_BATCH];          // tokens cached (compress: before the call; decode: L)
  int32_t kact[2][SWAN_MAX_BATCH];      // k of the keys / of the values
  int64_t page_off[2][SWAN_MAX_BATCH];  // byte offset of the sequence's first key / value page
  int32_t nnew[SWAN_MAX_BATCH];         // compress: tokens appended to the sequence
  int32_t nsplit[SWAN_MAX_BATCH];       // decode: token splits of the sequence's launch
  int8_t flat[SWAN_MAX_BATCH];          // decode: 1 = splits of equal size (short sequences)
};

__host__ __device__ inline int kpad_of(int k) { return (k + 7) & ~7; }

// First page of split s when a sequence's np pages are cut into ns splits of
// shrinking size (weights ns, ns - 1, ..., 1): the grids are split-major, so
// the longest splits are dispatched first and the last ones are short, which
// shortens the tail.  Every split has at least one page when
// ns (ns + 1) / 2 <= np (the planner keeps to that).  A short sequence, whose
// pages that rule would leave in a few long splits, is cut into ns equal splits
// instead (flat; every split has a page when ns <= np).
__host__ __device__ inline int split_begin(int s, int ns, int np, bool flat = false) {
  if (flat) return (int)((int64_t)s * np / ns);
  const int64_t before = (int64_t)s * ns - (int64_t)s * (s - 1) / 2;  // sum_{i<s} (ns - i)
  const int64_t total = (int64_t)ns * (ns + 1) / 2;
  return (int)(before * np / total);
}

__host__ __device__ inline int64_t page_bytes_of(int elem_bytes, int k) {
  return int64_t(kPage) * kpad_of(k) * (elem_bytes + 1);
}

__host__ __device__ inline int pages_for(int tokens) { return (tokens + kPage - 1) / kPage; }

// Host-side launchers (defined in the .hip files).  All return hipSuccess or the
// error of the launch.
struct DecodeLaunch {
  const void* q;
  const float* P_qk;
  const float* P_vo;
  void* out;
  const void* k_pages;
  const void* v_pages;
  const void* k_ring;
  const void* v_ring;
  float* qhat;   // [B][Hq][128] workspace
  float* part;   // [B][Hq][NS + 1][kPartFloats] workspace
  int B, Hq, Hkv, bb, n_pages_cap;
  int n_splits;  // NS: largest split count of any launch (slot NS holds the buffer partial)
  float qmult;   // scale * log2(e)
  int dtype;
  SeqTab tab;
  hipStream_t stream;
  hipEvent_t prof_start;  // optional events around the attention launches
  hipEvent_t prof_stop;
  int merge_pct;          // launch grouping of a mixed-k batch (<= 0: none)
  int side_streams;       // library streams for those launches, 0..kSideStreams
  int qhat_ready = 0;     // 1: qhat already holds the rotated queries (decode steps)
};
hipError_t launch_decode(const DecodeLaunch& a);
constexpr int kSideStreams = 3;  // extra streams for the launches of a mixed-k batch
constexpr int kMaxDevices = 16;

// sequences of one attention launch (those sharing a page format)
struct SeqGroup {
  int32_t n;
  int32_t n_splits;
  int32_t seq[SWAN_MAX_BATCH];
};

// sequences of a batch with several k_pad, in one MHA attention launch: each
// sparse wave runs the kernel body specialised on its own sequence's k_pad
struct FusedSeqs {
  int32_t n;                    // sequences
  int32_t n_splits;             // the largest split count among them
  int32_t seq[SWAN_MAX_BATCH];  // batch indices, larger k_pad first
  int8_t kp8[SWAN_MAX_BATCH];   // fused_tier of the larger of its key and value k_pad / 8
};
int fused_tier(int kp8);  // the kernel body serving k_pad 8 kp8: 2, 4, ..., 12 or 16
hipError_t launch_attn_fused(const DecodeLaunch& a, const FusedSeqs& f);

// GQA path (fp16 storage, G = n_q / n_kv > 1): query heads served by one wave,
// 1 when the GQA kernel does not apply
int gqa_heads_per_wave(int G);
inline int decode_heads_per_wave(int dtype, int n_q, int n_kv) {
  const int G = n_q / n_kv;
  return ((dtype == SWAN_F16 || dtype == SWAN_F16_E4M3) && G > 1) ? gqa_heads_per_wave(G) : 1;
}
hipError_t launch_attn_gqa(const DecodeLaunch& a, const SeqGroup& g, int kp8);
// sequences whose keys and values have different k_pad; kp8 = the larger / 8
hipError_t launch_attn_asym(const DecodeLaunch& a, const SeqGroup& g, int kp8);
hipError_t launch_attn_gqa_asym(const DecodeLaunch& a, const SeqGroup& g, int kp8);


struct CompressLaunch {
  const void* k_new;
  const void* v_new;
  const float* P_qk;
  const float* P_vo;
  void* k_pages;
  void* v_pages;
  void* k_ring;
  void* v_ring;
  int B, Hkv, bb, n_pages_cap, n_new;  // n_new: token stride of k_new / v_new
  int max_evict;  // largest per-sequence eviction count
  int prefill_groups;  // waves per (sequence, head, role) of the prefill kernel
  int dtype;
  SeqTab tab;     // len = tokens cached before the call
  hipStream_t stream;
  // decode steps (n_new == 1) only: q != nullptr makes the key waves also
  // write q_hat = q . P_qk * qmult for the Hq / Hkv (at most kStepQG) query
  // heads of their kv head, q [B][Hq][128] storage type, qhat [B][Hq][128]
  const void* q = nullptr;
  float* qhat = nullptr;
  int Hq = 0;
  float qmult = 0.f;
};
constexpr int kStepQG = 8;
hipError_t launch_compress(const CompressLaunch& a);
// prefill path (fp16, many tokens): float64 MFMA rotation + lane-per-token top-k
constexpr int kPrefillMinTokens = 64;
int prefill_groups(int max_new_tokens, int min_len_old);
hipError_t launch_prefill(const CompressLaunch& a);

// run-time change of k: one launch per role, over the role's page arrays
// (change_k.hip)
struct ChangeKLaunch {
  const char* src;  // the role's pages in the source cache
  char* dst;        // the role's pages in the destination cache
  int B, Hkv, bb, npc_src, npc_dst, max_pages, dtype;
  int32_t len[SWAN_MAX_BATCH];      // tokens cached
  int32_t k_src[SWAN_MAX_BATCH];    // the role's k in the source layout
  int32_t k_dst[SWAN_MAX_BATCH];    // the role's k in the destination layout
  int64_t off_src[SWAN_MAX_BATCH];  // byte offset of the sequence's first source page
  int64_t off_dst[SWAN_MAX_BATCH];  // byte offset of the sequence's first destination page
  int nsel;                         // set by launch_change_k: the sequences of one launch
  int32_t sel[SWAN_MAX_BATCH];
  hipStream_t stream;
};
hipError_t launch_change_k(const ChangeKLaunch& a);

// RoPE of query / key rows before the rotation (rope.hip)
struct RopeLaunch {
  const void* x;
  void* y;
  int B, H, n, dtype;
  int32_t pos0[SWAN_MAX_BATCH];  // position of each sequence's first row
  double base;
  hipStream_t stream;
};
hipError_t launch_rope(const RopeLaunch& a);

struct CalibLaunch {
  const float* rows;
  int64_t n_rows;
  float* P_out;
  float* sigma_out;
  double* gram;    // [128][128]
  double* vecs;    // [128][128]
  int32_t* status; // [4]: converged flag, sweeps
  hipStream_t stream;
};
hipError_t launch_calibrate(const CalibLaunch& a);
constexpr size_t kCalibWorkspace = 2 * sizeof(double) * kD * kD + 256;
constexpr int kJacobiMaxSweeps = 40;

}  // namespace swan
