// Host side of the C ABI declared in include/swan.h: argument validation
// (always before anything is enqueued), workspace sizing, split planning and
// kernel launches.  No allocation, no host arithmetic on the data path.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <mutex>
#include <string>

#include "swan.h"
#include "swan_internal.h"

// ---------------------------------------------------------------------------
// Scratch of swan_decode_attention_noalloc: the decode workspace (q_hat, then
// the partials) in a device array of fixed size, one copy per GPU, held until
// the process ends.  Host code only ever uses the address that
// hipGetSymbolAddress returns for the current device: the array's name is a
// host-side stand-in, not a device address.
// ---------------------------------------------------------------------------
constexpr size_t kScratchBytes = SWAN_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) char scratch[kScratchBytes];

namespace {

thread_local std::string g_last_error;
thread_local hipEvent_t g_prof_start = nullptr;
thread_local hipEvent_t g_prof_stop = nullptr;

// Decode tuning of this thread (swan_set_decode_tuning), with the defaults
// resolved: about two sparse waves per wave slot of the GPU (measured best for
// long contexts), short sequences in 4-page splits, launch merging at two
// thirds of the k_pad, three side streams.
struct Tuning {
  int64_t target_waves = 256 * 4 * 2;
  int short_split_pages = 3;  // 0: never
  int merge_pct = 66;         // 0: never
  int side_streams = swan::kSideStreams;
};
thread_local Tuning g_tuning;

swan_status fail(swan_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

swan_status ok() {
  g_last_error.clear();
  return SWAN_OK;
}

// bytes of one element of queries, outputs, new keys / values and the ring
int elem_bytes(int32_t dtype) { return dtype == SWAN_F32 ? 4 : 2; }
// bytes of one sparse value
int value_bytes(int32_t dtype) { return dtype == SWAN_F32 ? 4 : dtype == SWAN_F16 ? 2 : 1; }
bool dtype_ok(int32_t dtype) {
  return dtype == SWAN_F32 || dtype == SWAN_F16 || dtype == SWAN_F16_E4M3;
}

swan_status check_cache_shape(const swan_cache* c) {
  if (!c) return fail(SWAN_ERR_INVALID_ARG, "cache descriptor is NULL");
  if (c->batch < 1 || c->batch > SWAN_MAX_BATCH)
    return fail(SWAN_ERR_INVALID_ARG, "batch %d outside 1..%d", c->batch, SWAN_MAX_BATCH);
  if (c->n_kv_heads < 1 || c->n_q_heads < 1)
    return fail(SWAN_ERR_INVALID_ARG, "head counts must be >= 1 (q %d, kv %d)", c->n_q_heads,
                c->n_kv_heads);
  if (c->n_q_heads % c->n_kv_heads != 0)
    return fail(SWAN_ERR_INVALID_ARG, "n_q_heads %d is not a multiple of n_kv_heads %d",
                c->n_q_heads, c->n_kv_heads);
  if (c->head_dim != SWAN_HEAD_DIM)
    return fail(SWAN_ERR_UNSUPPORTED, "head_dim %d: the GPU path supports %d only", c->head_dim,
                SWAN_HEAD_DIM);
  if (c->buffer_tokens < 0)
    return fail(SWAN_ERR_INVALID_ARG, "buffer_tokens %d < 0", c->buffer_tokens);
  if (c->buffer_tokens > swan::kMaxRing)
    return fail(SWAN_ERR_UNSUPPORTED, "buffer_tokens %d above %d", c->buffer_tokens,
                swan::kMaxRing);
  if (c->sparse_capacity < 0)
    return fail(SWAN_ERR_INVALID_ARG, "sparse_capacity %d < 0", c->sparse_capacity);
  if (!dtype_ok(c->dtype)) return fail(SWAN_ERR_UNSUPPORTED, "dtype %d not supported", c->dtype);
  if (c->reserved != 0) return fail(SWAN_ERR_INVALID_ARG, "reserved field must be 0");
  return SWAN_OK;
}

// k of the keys (k_active_host) and, if not NULL, of the values (k_value_host)
swan_status check_k(const swan_cache* c, const int32_t* k_active_host,
                    const int32_t* k_value_host) {
  if (!k_active_host) return fail(SWAN_ERR_INVALID_ARG, "k_active_host is NULL");
  for (int b = 0; b < c->batch; ++b) {
    const int k = k_active_host[b];
    if (k < 1 || k > c->head_dim)
      return fail(SWAN_ERR_INVALID_ARG, "k_active[%d] = %d outside 1..%d", b, k, c->head_dim);
    if (!k_value_host) continue;
    const int kv = k_value_host[b];
    if (kv < 1 || kv > c->head_dim)
      return fail(SWAN_ERR_INVALID_ARG, "k_value[%d] = %d outside 1..%d", b, kv, c->head_dim);
  }
  return SWAN_OK;
}

// k of role r (0 keys, 1 values) of sequence b
inline int k_of(const int32_t* k_active_host, const int32_t* k_value_host, int r, int b) {
  return (r == 1 && k_value_host) ? k_value_host[b] : k_active_host[b];
}

swan_status check_cache_ptrs(const swan_cache* c) {
  if (c->sparse_capacity > 0 && (!c->k_pages || !c->v_pages))
    return fail(SWAN_ERR_INVALID_ARG, "k_pages / v_pages is NULL");
  if (c->buffer_tokens > 0 && (!c->k_ring || !c->v_ring))
    return fail(SWAN_ERR_INVALID_ARG, "k_ring / v_ring is NULL");
  const void* ptrs[4] = {c->k_pages, c->v_pages, c->k_ring, c->v_ring};
  for (const void* p : ptrs)
    if (((uintptr_t)p & 15) != 0)
      return fail(SWAN_ERR_INVALID_ARG, "cache arrays must be 16-byte aligned");
  return SWAN_OK;
}

// fills tab.kact and tab.page_off of both roles; bytes[r] = total page bytes of role r
void fill_layout(const swan_cache* c, const int32_t* k_active_host, const int32_t* k_value_host,
                 swan::SeqTab& tab, int64_t bytes[2]) {
  const int npc = swan::pages_for(c->sparse_capacity);
  for (int b = 0; b < SWAN_MAX_BATCH; ++b) {
    for (int r = 0; r < 2; ++r) {
      tab.kact[r][b] = 0;
      tab.page_off[r][b] = 0;
    }
    tab.len[b] = 0;
    tab.nnew[b] = 0;
    tab.nsplit[b] = 1;
    tab.flat[b] = 0;
  }
  for (int r = 0; r < 2; ++r) {
    int64_t off = 0;
    for (int b = 0; b < c->batch; ++b) {
      const int k = k_of(k_active_host, k_value_host, r, b);
      tab.kact[r][b] = k;
      tab.page_off[r][b] = off;
      off += (int64_t)c->n_kv_heads * npc * swan::page_bytes_of(value_bytes(c->dtype), k);
    }
    bytes[r] = off;
  }
}

// Token splits per (sequence, query head): about the thread's target number of
// waves in total, the split count of each sequence following its bytes (a page
// weighs the k_pad of its keys plus that of its values); the splits themselves
// shrink in size (split_begin), and their count is capped so that every split
// keeps a page.  Fills nsplit[b] (may be NULL); returns the largest.
int plan_splits(const swan_cache* c, const int32_t* seq_len_host, const int32_t* k_active_host,
                const int32_t* k_value_host, int32_t* nsplit, int8_t* flat = nullptr) {
  auto weight = [&](int b) {
    return swan::kpad_of(k_of(k_active_host, k_value_host, 0, b)) +
           swan::kpad_of(k_of(k_active_host, k_value_host, 1, b));
  };
  // waves per sequence and split: one per query head, or one per GH query
  // heads of a KV head on the GQA path
  const int hpw = swan::decode_heads_per_wave(c->dtype, c->n_q_heads, c->n_kv_heads);
  const int waves_per_seq = c->n_q_heads / hpw;
  int64_t total = 0;
  for (int b = 0; b < c->batch; ++b) {
    const int S = seq_len_host[b] > c->buffer_tokens ? seq_len_host[b] - c->buffer_tokens : 0;
    total += (int64_t)swan::pages_for(S) * weight(b) * waves_per_seq;
  }
  // A batch of several k_pad on the fused MHA launch (decode_fused.hip) takes
  // twice the waves: its shorter splits balance the tiers' different costs
  // per page (measured: 16k x 8 with k in {32, 48, 64, 96}, 0.222 -> 0.213 ms;
  // the single-k workloads gain nothing from it and GQA loses 8 %).
  bool several_kpad = false;
  for (int b = 1; b < c->batch; ++b)
    several_kpad |= swan::kpad_of(k_of(k_active_host, k_value_host, 0, b)) !=
                        swan::kpad_of(k_of(k_active_host, k_value_host, 0, 0)) ||
                    swan::kpad_of(k_of(k_active_host, k_value_host, 1, b)) !=
                        swan::kpad_of(k_of(k_active_host, k_value_host, 1, 0));
  const bool fused = several_kpad && hpw == 1 &&
                     (c->dtype == SWAN_F16 || c->dtype == SWAN_F16_E4M3);
  const int64_t target_waves = g_tuning.target_waves * (fused ? 2 : 1);
  // A sequence whose shrinking splits the one-page rule cuts to half the count
  // wanted or fewer is short: its waves would each walk many pages one after
  // another, so it gets equal splits of flat_pages pages instead.
  const int flat_pages = g_tuning.short_split_pages;
  int64_t per_wave = (total + target_waves - 1) / target_waves;
  if (per_wave < 1) per_wave = 1;
  int ns_max = 1;
  for (int b = 0; b < c->batch; ++b) {
    const int S = seq_len_host[b] > c->buffer_tokens ? seq_len_host[b] - c->buffer_tokens : 0;
    const int np = swan::pages_for(S);
    const int64_t work = (int64_t)np * weight(b);
    const int want = (int)((work + per_wave - 1) / per_wave);
    int ns = want;
    while (ns > 1 && (int64_t)ns * (ns + 1) / 2 > np) --ns;  // every split keeps a page
    bool fl = false;
    if (flat_pages > 0 && 2 * ns <= want) {
      // short sequence: equal splits of about flat_pages pages instead
      fl = true;
      ns = np / flat_pages < want ? np / flat_pages : want;
    }
    if (ns > swan::kMaxSplits) ns = swan::kMaxSplits;
    if (ns < 1) ns = 1;
    if (nsplit) nsplit[b] = ns;
    if (flat) flat[b] = fl ? 1 : 0;
    if (ns > ns_max) ns_max = ns;
  }
  return ns_max;
}

size_t round256(size_t x) { return (x + 255) & ~(size_t)255; }

// workspace: q_hat, then the partials
size_t decode_ws_bytes(const swan_cache* c, int ns) {
  const size_t units = (size_t)c->batch * c->n_q_heads;
  const size_t qhat = units * swan::kD * sizeof(float);
  const size_t part = units * (size_t)(ns + 1) * swan::kPartFloats * sizeof(float);
  return round256(qhat) + part;
}

swan_status hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return ok();
  return fail(SWAN_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

std::mutex g_scratch_mu;
void* g_scratch_ptr[swan::kMaxDevices] = {};

// The scratch array's address on the device of `stream` (set up once per
// device, with that device current).
swan_status scratch_for_stream(hipStream_t stream, void** ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_status(e, "hipGetDevice");
  if (dev < 0 || dev >= swan::kMaxDevices)
    return fail(SWAN_ERR_UNSUPPORTED, "device %d: the scratch table holds %d devices", dev,
                swan::kMaxDevices);
  if (stream) {
    hipDevice_t sdev = -1;
    e = hipStreamGetDevice(stream, &sdev);
    if (e != hipSuccess) return hip_status(e, "hipStreamGetDevice");
    if (sdev != dev)
      return fail(SWAN_ERR_INVALID_ARG,
                  "the stream belongs to device %d but device %d is current", (int)sdev, dev);
  }
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_status(e, "hipGetSymbolAddress(scratch)");
    if (!p || ((uintptr_t)p & 255) != 0)
      return fail(SWAN_ERR_HIP, "scratch array at an unusable address");
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return SWAN_OK;
}

// swan_compress_append's validation, into `a` (nothing is enqueued); any_new:
// some sequence appends a token
swan_status compress_prep(const swan_cache* c, const int32_t* seq_len_host,
                          const int32_t* k_active_host, const int32_t* k_value_host,
                          const void* k_new, const void* v_new, int32_t n_new,
                          const int32_t* n_new_host, const float* P_qk, const float* P_vo,
                          void* stream, swan::CompressLaunch& a, bool& any_new) {
  swan_status st = check_cache_shape(c);
  if (st != SWAN_OK) return st;
  if ((st = check_k(c, k_active_host, k_value_host)) != SWAN_OK) return st;
  if ((st = check_cache_ptrs(c)) != SWAN_OK) return st;
  if (!seq_len_host) return fail(SWAN_ERR_INVALID_ARG, "seq_len_host is NULL");
  if (n_new < 0) return fail(SWAN_ERR_INVALID_ARG, "n_new %d < 0", n_new);
  if (n_new > 0 && (!k_new || !v_new)) return fail(SWAN_ERR_INVALID_ARG, "k_new / v_new is NULL");
  if (!P_qk) return fail(SWAN_ERR_INVALID_ARG, "P_qk is NULL");
  if ((((uintptr_t)P_qk | (uintptr_t)P_vo) & 15) != 0)
    return fail(SWAN_ERR_INVALID_ARG, "P_qk / P_vo must be 16-byte aligned");
  if ((((uintptr_t)k_new | (uintptr_t)v_new) & 15) != 0)
    return fail(SWAN_ERR_INVALID_ARG, "k_new / v_new must be 16-byte aligned");
  int max_evict = 0;
  any_new = false;
  for (int b = 0; b < c->batch; ++b) {
    const int64_t L0 = seq_len_host[b];
    if (L0 < 0) return fail(SWAN_ERR_INVALID_ARG, "seq_len[%d] = %lld < 0", b, (long long)L0);
    const int nb_new = n_new_host ? n_new_host[b] : n_new;
    if (nb_new < 0 || nb_new > n_new)
      return fail(SWAN_ERR_INVALID_ARG, "n_new_host[%d] = %d outside 0..%d", b, nb_new, n_new);
    any_new |= nb_new != 0;
    const int64_t L1 = L0 + nb_new;
    if (L1 > INT32_MAX / 2)
      return fail(SWAN_ERR_INVALID_ARG, "seq_len[%d] + n_new too large", b);
    if (L1 - c->buffer_tokens > c->sparse_capacity)
      return fail(SWAN_ERR_CAPACITY, "sequence %d needs %lld sparse tokens, capacity %d", b,
                  (long long)(L1 - c->buffer_tokens), c->sparse_capacity);
    const int64_t p0 = L0 > c->buffer_tokens ? L0 - c->buffer_tokens : 0;
    const int64_t p1 = L0 < L1 - c->buffer_tokens ? L0 : L1 - c->buffer_tokens;
    if (p1 - p0 > max_evict) max_evict = (int)(p1 - p0);
  }
  int64_t role_bytes[2];
  fill_layout(c, k_active_host, k_value_host, a.tab, role_bytes);
  for (int b = 0; b < c->batch; ++b) {
    a.tab.len[b] = seq_len_host[b];
    a.tab.nnew[b] = n_new_host ? n_new_host[b] : n_new;
  }
  a.k_new = k_new;
  a.v_new = v_new;
  a.P_qk = P_qk;
  a.P_vo = P_vo;
  a.k_pages = c->k_pages;
  a.v_pages = c->v_pages;
  a.k_ring = c->k_ring;
  a.v_ring = c->v_ring;
  a.B = c->batch;
  a.Hkv = c->n_kv_heads;
  a.bb = c->buffer_tokens;
  a.n_pages_cap = swan::pages_for(c->sparse_capacity);
  a.n_new = n_new;
  a.max_evict = max_evict;
  a.prefill_groups = swan::prefill_groups(n_new, 0);
  a.dtype = c->dtype;
  a.stream = (hipStream_t)stream;
  return SWAN_OK;
}

// The decode entry points' validation and split plan, into `a` (nothing is
// enqueued).  no_alloc: the workspace is this library's scratch array (looked
// up after every host check has passed), a plan that needs more than the
// array is rejected, and the launches stay on `stream` (creating the side
// streams could allocate).
swan_status decode_prep(const swan_cache* c, const int32_t* seq_len_host,
                        const int32_t* k_active_host, const int32_t* k_value_host, const void* q,
                        const float* P_qk, const float* P_vo, float scale, void* out,
                        void* workspace, size_t workspace_bytes, void* stream, bool no_alloc,
                        swan::DecodeLaunch& a) {
  swan_status st = check_cache_shape(c);
  if (st != SWAN_OK) return st;
  if ((st = check_k(c, k_active_host, k_value_host)) != SWAN_OK) return st;
  if ((st = check_cache_ptrs(c)) != SWAN_OK) return st;
  if (!seq_len_host) return fail(SWAN_ERR_INVALID_ARG, "seq_len_host is NULL");
  if (!q || !out || !P_qk) return fail(SWAN_ERR_INVALID_ARG, "q / out / P_qk is NULL");
  if ((((uintptr_t)P_qk | (uintptr_t)P_vo) & 15) != 0)
    return fail(SWAN_ERR_INVALID_ARG, "P_qk / P_vo must be 16-byte aligned");
  for (int b = 0; b < c->batch; ++b) {
    const int64_t L = seq_len_host[b];
    if (L < 1) return fail(SWAN_ERR_INVALID_ARG, "seq_len[%d] = %lld: need L >= 1", b, (long long)L);
    if (L - c->buffer_tokens > c->sparse_capacity)
      return fail(SWAN_ERR_CAPACITY, "sequence %d has %lld sparse tokens, capacity %d", b,
                  (long long)(L - c->buffer_tokens), c->sparse_capacity);
  }
  if (!(scale == scale) || isinf(scale)) return fail(SWAN_ERR_INVALID_ARG, "scale is not finite");
  int64_t role_bytes[2];
  fill_layout(c, k_active_host, k_value_host, a.tab, role_bytes);
  const int ns = plan_splits(c, seq_len_host, k_active_host, k_value_host, a.tab.nsplit,
                            a.tab.flat);
  const size_t need = decode_ws_bytes(c, ns);
  if (no_alloc) {
    if (need > kScratchBytes)
      return fail(SWAN_ERR_WORKSPACE,
                  "this batch needs %zu bytes of decode scratch; swan_decode_attention_noalloc "
                  "holds %zu (use swan_decode_attention with a workspace)", need, kScratchBytes);
    const swan_status sst = scratch_for_stream((hipStream_t)stream, &workspace);
    if (sst != SWAN_OK) return sst;
    workspace_bytes = kScratchBytes;
  }
  if (!workspace || workspace_bytes < need)
    return fail(SWAN_ERR_WORKSPACE, "workspace of %zu bytes, need %zu", workspace_bytes, need);
  if (((uintptr_t)workspace & 255) != 0)
    return fail(SWAN_ERR_INVALID_ARG, "workspace must be 256-byte aligned");
  for (int b = 0; b < c->batch; ++b) a.tab.len[b] = seq_len_host[b];
  const float sc = scale > 0.f ? scale : 1.0f / sqrtf((float)c->head_dim);
  a.q = q;
  a.P_qk = P_qk;
  a.P_vo = P_vo;
  a.out = out;
  a.k_pages = c->k_pages;
  a.v_pages = c->v_pages;
  a.k_ring = c->k_ring;
  a.v_ring = c->v_ring;
  const size_t units = (size_t)c->batch * c->n_q_heads;
  a.qhat = (float*)workspace;
  a.part = (float*)((char*)workspace + round256(units * swan::kD * sizeof(float)));
  a.B = c->batch;
  a.Hq = c->n_q_heads;
  a.Hkv = c->n_kv_heads;
  a.bb = c->buffer_tokens;
  a.n_pages_cap = swan::pages_for(c->sparse_capacity);
  a.n_splits = ns;
  a.qmult = sc * 1.4426950408889634f;
  a.dtype = c->dtype;
  a.stream = (hipStream_t)stream;
  a.prof_start = g_prof_start;
  a.prof_stop = g_prof_stop;
  a.merge_pct = g_tuning.merge_pct;
  a.side_streams = no_alloc ? 0 : g_tuning.side_streams;
  return SWAN_OK;
}

// Both decode entry points: validation, split plan, launches.
swan_status decode_impl(const swan_cache* c, const int32_t* seq_len_host,
                        const int32_t* k_active_host, const int32_t* k_value_host, const void* q,
                        const float* P_qk, const float* P_vo, float scale, void* out,
                        void* workspace, size_t workspace_bytes, void* stream, bool no_alloc) {
  swan::DecodeLaunch a;
  const swan_status st = decode_prep(c, seq_len_host, k_active_host, k_value_host, q, P_qk,
                                     P_vo, scale, out, workspace, workspace_bytes, stream,
                                     no_alloc, a);
  if (st != SWAN_OK) return st;
  return hip_status(swan::launch_decode(a), "decode launch");
}

}  // namespace

extern "C" {

const char* swan_last_error(void) { return g_last_error.c_str(); }

int32_t swan_version(void) { return 205; }

swan_status swan_page_bytes(int32_t dtype, int32_t k_active, size_t* bytes) {
  if (!bytes) return fail(SWAN_ERR_INVALID_ARG, "bytes is NULL");
  if (!dtype_ok(dtype)) return fail(SWAN_ERR_UNSUPPORTED, "dtype %d not supported", dtype);
  if (k_active < 1 || k_active > SWAN_HEAD_DIM)
    return fail(SWAN_ERR_INVALID_ARG, "k_active %d outside 1..%d", k_active, SWAN_HEAD_DIM);
  *bytes = (size_t)swan::page_bytes_of(value_bytes(dtype), k_active);
  return ok();
}

swan_status swan_cache_bytes(const swan_cache* c, const int32_t* k_active_host,
                             const int32_t* k_value_host, size_t* k_page_bytes,
                             size_t* v_page_bytes, size_t* ring_bytes) {
  swan_status st = check_cache_shape(c);
  if (st != SWAN_OK) return st;
  if ((st = check_k(c, k_active_host, k_value_host)) != SWAN_OK) return st;
  if (!k_page_bytes || !v_page_bytes || !ring_bytes)
    return fail(SWAN_ERR_INVALID_ARG, "output pointer is NULL");
  swan::SeqTab tab;
  int64_t bytes[2];
  fill_layout(c, k_active_host, k_value_host, tab, bytes);
  *k_page_bytes = (size_t)bytes[0];
  *v_page_bytes = (size_t)bytes[1];
  *ring_bytes = (size_t)c->batch * c->n_kv_heads * c->buffer_tokens * c->head_dim *
                elem_bytes(c->dtype);
  return ok();
}

swan_status swan_calibrate_workspace_bytes(int32_t d, size_t* bytes) {
  if (!bytes) return fail(SWAN_ERR_INVALID_ARG, "bytes is NULL");
  if (d != SWAN_HEAD_DIM)
    return fail(SWAN_ERR_UNSUPPORTED, "d %d: the GPU path supports %d only", d, SWAN_HEAD_DIM);
  *bytes = swan::kCalibWorkspace;
  return ok();
}

swan_status swan_calibrate_rotation(const float* rows, int64_t n_rows, int32_t d, float* P_out,
                                    float* sigma_out, void* workspace, size_t workspace_bytes,
                                    void* stream) {
  if (d != SWAN_HEAD_DIM)
    return fail(SWAN_ERR_UNSUPPORTED, "d %d: the GPU path supports %d only", d, SWAN_HEAD_DIM);
  if (!rows || !P_out) return fail(SWAN_ERR_INVALID_ARG, "rows / P_out is NULL");
  if (n_rows < 1) return fail(SWAN_ERR_INVALID_ARG, "n_rows %lld < 1", (long long)n_rows);
  if (!workspace || workspace_bytes < swan::kCalibWorkspace)
    return fail(SWAN_ERR_WORKSPACE, "workspace of %zu bytes, need %zu", workspace_bytes,
                swan::kCalibWorkspace);
  if (((uintptr_t)workspace & 15) != 0)
    return fail(SWAN_ERR_INVALID_ARG, "workspace must be 16-byte aligned");
  char* ws = (char*)workspace;
  swan::CalibLaunch a;
  a.rows = rows;
  a.n_rows = n_rows;
  a.P_out = P_out;
  a.sigma_out = sigma_out;
  a.gram = (double*)ws;
  a.vecs = (double*)(ws + sizeof(double) * swan::kD * swan::kD);
  a.status = (int32_t*)(ws + 2 * sizeof(double) * swan::kD * swan::kD);
  a.stream = (hipStream_t)stream;
  hipError_t e = swan::launch_calibrate(a);
  if (e != hipSuccess) return hip_status(e, "calibrate launch");
  int32_t st_host[2] = {0, 0};
  e = hipMemcpyAsync(st_host, a.status, sizeof(st_host), hipMemcpyDeviceToHost, a.stream);
  if (e != hipSuccess) return hip_status(e, "calibrate status copy");
  e = hipStreamSynchronize(a.stream);
  if (e != hipSuccess) return hip_status(e, "calibrate synchronize");
  if (!st_host[0])
    return fail(SWAN_ERR_NO_CONVERGENCE, "Jacobi eigensolver did not converge in %d sweeps",
                st_host[1]);
  return ok();
}

swan_status swan_compress_append(const swan_cache* c, const int32_t* seq_len_host,
                                 const int32_t* k_active_host, const int32_t* k_value_host,
                                 const void* k_new, const void* v_new, int32_t n_new,
                                 const int32_t* n_new_host, const float* P_qk, const float* P_vo,
                                 void* stream) {
  swan::CompressLaunch a;
  bool any_new = false;
  const swan_status st = compress_prep(c, seq_len_host, k_active_host, k_value_host, k_new, v_new,
                                       n_new, n_new_host, P_qk, P_vo, stream, a, any_new);
  if (st != SWAN_OK) return st;
  if (!any_new) return ok();
  return hip_status(swan::launch_compress(a), "compress launch");
}

swan_status swan_decode_workspace_bytes(const swan_cache* c, const int32_t* seq_len_host,
                                        const int32_t* k_active_host,
                                        const int32_t* k_value_host, size_t* bytes) {
  swan_status st = check_cache_shape(c);
  if (st != SWAN_OK) return st;
  if ((st = check_k(c, k_active_host, k_value_host)) != SWAN_OK) return st;
  if (!seq_len_host || !bytes) return fail(SWAN_ERR_INVALID_ARG, "NULL argument");
  *bytes = decode_ws_bytes(c, plan_splits(c, seq_len_host, k_active_host, k_value_host, nullptr));
  return ok();
}

swan_status swan_decode_attention(const swan_cache* c, const int32_t* seq_len_host,
                                  const int32_t* k_active_host, const int32_t* k_value_host,
                                  const void* q, const float* P_qk, const float* P_vo, float scale,
                                  void* out, void* workspace, size_t workspace_bytes,
                                  void* stream) {
  return decode_impl(c, seq_len_host, k_active_host, k_value_host, q, P_qk, P_vo, scale, out,
                     workspace, workspace_bytes, stream, false);
}

swan_status swan_decode_attention_noalloc(const swan_cache* c, const int32_t* seq_len_host,
                                          const int32_t* k_active_host,
                                          const int32_t* k_value_host, const void* q,
                                          const float* P_qk, const float* P_vo, float scale,
                                          void* out, void* stream) {
  return decode_impl(c, seq_len_host, k_active_host, k_value_host, q, P_qk, P_vo, scale, out,
                     nullptr, 0, stream, true);
}

swan_status swan_decode_step(const swan_cache* c, const int32_t* seq_len_host,
                             const int32_t* k_active_host, const int32_t* k_value_host,
                             const void* k_new, const void* v_new, const void* q,
                             const float* P_qk, const float* P_vo, float scale, void* out,
                             void* workspace, size_t workspace_bytes, void* stream) {
  // every check of both halves before anything is enqueued
  swan::CompressLaunch ca;
  bool any_new = false;
  swan_status st = compress_prep(c, seq_len_host, k_active_host, k_value_host, k_new, v_new, 1,
                                 nullptr, P_qk, P_vo, stream, ca, any_new);
  if (st != SWAN_OK) return st;
  int32_t len1[SWAN_MAX_BATCH];
  for (int b = 0; b < c->batch; ++b) len1[b] = seq_len_host[b] + 1;
  swan::DecodeLaunch da;
  st = decode_prep(c, len1, k_active_host, k_value_host, q, P_qk, P_vo, scale, out, workspace,
                   workspace_bytes, stream, false, da);
  if (st != SWAN_OK) return st;
  if (c->n_q_heads / c->n_kv_heads <= swan::kStepQG) {  // the key waves rotate the queries
    ca.q = q;
    ca.qhat = da.qhat;
    ca.Hq = da.Hq;
    ca.qmult = da.qmult;
    da.qhat_ready = 1;
  }
  const hipError_t e = swan::launch_compress(ca);
  if (e != hipSuccess) return hip_status(e, "compress launch");
  return hip_status(swan::launch_decode(da), "decode launch");
}

swan_status swan_change_k(const swan_cache* src, const int32_t* k_active_src,
                          const int32_t* k_value_src, const swan_cache* dst,
                          const int32_t* k_active_dst, const int32_t* k_value_dst,
                          const int32_t* seq_len_host, void* stream) {
  swan_status st = check_cache_shape(src);
  if (st != SWAN_OK) return st;
  if ((st = check_cache_shape(dst)) != SWAN_OK) return st;
  if (src->batch != dst->batch || src->n_q_heads != dst->n_q_heads ||
      src->n_kv_heads != dst->n_kv_heads || src->buffer_tokens != dst->buffer_tokens ||
      src->dtype != dst->dtype)
    return fail(SWAN_ERR_INVALID_ARG,
                "src and dst differ in batch, heads, buffer_tokens or dtype");
  if ((st = check_k(src, k_active_src, k_value_src)) != SWAN_OK) return st;
  if ((st = check_k(dst, k_active_dst, k_value_dst)) != SWAN_OK) return st;
  if ((st = check_cache_ptrs(src)) != SWAN_OK) return st;
  if ((st = check_cache_ptrs(dst)) != SWAN_OK) return st;
  if (src->k_ring != dst->k_ring || src->v_ring != dst->v_ring)
    return fail(SWAN_ERR_INVALID_ARG, "dst must share src's ring arrays (the buffer is unchanged)");
  if (!seq_len_host) return fail(SWAN_ERR_INVALID_ARG, "seq_len_host is NULL");
  int max_pages = 0;
  for (int b = 0; b < src->batch; ++b) {
    const int64_t L = seq_len_host[b];
    if (L < 0) return fail(SWAN_ERR_INVALID_ARG, "seq_len[%d] = %lld < 0", b, (long long)L);
    const int64_t S = L > src->buffer_tokens ? L - src->buffer_tokens : 0;
    if (S > src->sparse_capacity || S > dst->sparse_capacity)
      return fail(SWAN_ERR_CAPACITY, "sequence %d has %lld sparse tokens, capacities %d / %d", b,
                  (long long)S, src->sparse_capacity, dst->sparse_capacity);
    const int np = swan::pages_for((int)S);
    if (np > max_pages) max_pages = np;
  }
  swan::SeqTab ts, td;
  int64_t bytes_src[2], bytes_dst[2];
  fill_layout(src, k_active_src, k_value_src, ts, bytes_src);
  fill_layout(dst, k_active_dst, k_value_dst, td, bytes_dst);
  // no destination page array may overlap a source one
  const char* sa[2] = {(const char*)src->k_pages, (const char*)src->v_pages};
  const char* da[2] = {(const char*)dst->k_pages, (const char*)dst->v_pages};
  for (int i = 0; i < 2; ++i)
    for (int j = 0; j < 2; ++j)
      if (bytes_src[i] > 0 && bytes_dst[j] > 0 && da[j] < sa[i] + bytes_src[i] &&
          sa[i] < da[j] + bytes_dst[j])
        return fail(SWAN_ERR_INVALID_ARG, "dst page arrays overlap src page arrays");
  for (int r = 0; r < 2; ++r) {
    swan::ChangeKLaunch a;
    a.src = sa[r];
    a.dst = (char*)da[r];
    a.B = src->batch;
    a.Hkv = src->n_kv_heads;
    a.bb = src->buffer_tokens;
    a.npc_src = swan::pages_for(src->sparse_capacity);
    a.npc_dst = swan::pages_for(dst->sparse_capacity);
    a.max_pages = max_pages;
    a.dtype = src->dtype;
    for (int b = 0; b < SWAN_MAX_BATCH; ++b) {
      a.len[b] = b < src->batch ? seq_len_host[b] : 0;
      a.k_src[b] = ts.kact[r][b];
      a.k_dst[b] = td.kact[r][b];
      a.off_src[b] = ts.page_off[r][b];
      a.off_dst[b] = td.page_off[r][b];
    }
    a.stream = (hipStream_t)stream;
    const hipError_t e = swan::launch_change_k(a);
    if (e != hipSuccess) return hip_status(e, "change_k launch");
  }
  return ok();
}

swan_status swan_rope(const void* x, void* y, int32_t dtype, int32_t batch, int32_t n_heads,
                      int32_t n, int32_t head_dim, const int32_t* pos0_host, double base,
                      void* stream) {
  if (!dtype_ok(dtype)) return fail(SWAN_ERR_UNSUPPORTED, "dtype %d not supported", dtype);
  if (head_dim != SWAN_HEAD_DIM)
    return fail(SWAN_ERR_UNSUPPORTED, "head_dim %d: the GPU path supports %d only", head_dim,
                SWAN_HEAD_DIM);
  if (batch < 1 || batch > SWAN_MAX_BATCH || n_heads < 1 || n < 0)
    return fail(SWAN_ERR_INVALID_ARG, "batch %d, n_heads %d, n %d", batch, n_heads, n);
  if (!(base > 1.0) || isinf(base)) return fail(SWAN_ERR_INVALID_ARG, "base must be > 1");
  if (!pos0_host) return fail(SWAN_ERR_INVALID_ARG, "pos0_host is NULL");
  if (n == 0) return ok();
  if (!x || !y) return fail(SWAN_ERR_INVALID_ARG, "x / y is NULL");
  if ((((uintptr_t)x | (uintptr_t)y) & 15) != 0)
    return fail(SWAN_ERR_INVALID_ARG, "x / y must be 16-byte aligned");
  swan::RopeLaunch a;
  a.x = x;
  a.y = y;
  a.B = batch;
  a.H = n_heads;
  a.n = n;
  a.dtype = dtype;
  for (int b = 0; b < SWAN_MAX_BATCH; ++b) {
    if (b < batch && (pos0_host[b] < 0 || (int64_t)pos0_host[b] + n > INT32_MAX))
      return fail(SWAN_ERR_INVALID_ARG, "pos0[%d] = %d out of range", b, pos0_host[b]);
    a.pos0[b] = b < batch ? pos0_host[b] : 0;
  }
  a.base = base;
  a.stream = (hipStream_t)stream;
  return hip_status(swan::launch_rope(a), "rope launch");
}

swan_status swan_set_decode_tuning(const swan_decode_tuning* t) {
  Tuning n;
  if (t) {
    if (t->target_waves < 0 || t->target_waves > (1 << 20))
      return fail(SWAN_ERR_INVALID_ARG, "target_waves %d outside 0..%d", t->target_waves, 1 << 20);
    if (t->short_split_pages < -1 || t->short_split_pages > 4096)
      return fail(SWAN_ERR_INVALID_ARG, "short_split_pages %d outside -1..4096",
                  t->short_split_pages);
    if (t->merge_pct < -1 || t->merge_pct > 100)
      return fail(SWAN_ERR_INVALID_ARG, "merge_pct %d outside -1..100", t->merge_pct);
    if (t->side_streams < -1 || t->side_streams > swan::kSideStreams)
      return fail(SWAN_ERR_INVALID_ARG, "side_streams %d outside -1..%d", t->side_streams,
                  swan::kSideStreams);
    if (t->target_waves > 0) n.target_waves = t->target_waves;
    if (t->short_split_pages != 0) n.short_split_pages = t->short_split_pages < 0 ? 0 : t->short_split_pages;
    if (t->merge_pct != 0) n.merge_pct = t->merge_pct < 0 ? 0 : t->merge_pct;
    if (t->side_streams != 0) n.side_streams = t->side_streams < 0 ? 0 : t->side_streams;
  }
  g_tuning = n;
  return ok();
}

swan_status swan_set_profile_events(void* start_event, void* stop_event) {
  if ((start_event == nullptr) != (stop_event == nullptr))
    return fail(SWAN_ERR_INVALID_ARG, "pass both events or neither");
  g_prof_start = (hipEvent_t)start_event;
  g_prof_stop = (hipEvent_t)stop_event;
  return ok();
}

}  // extern "C"
