/*
 * swan.h -- C ABI of libswan, a gfx950 (MI355X) implementation of the decode
 * hot path of SWAN (Sparse Winnowed Attention, arXiv 2511.18936).
 *
 * The method, in the paper's terms: keys and values are rotated by an offline
 * per-head orthogonal matrix obtained from an SVD (Sec. 4.1.2), the most recent
 * b rotated vectors stay dense in a FIFO buffer, and each vector evicted from
 * the buffer is pruned to its k largest-magnitude components, stored as
 * (value, uint8 index) pairs (Algorithm 1; Sec. 4.3; Sec. 5.1).  A decode query
 * is rotated once and scored directly against the sparse pairs and the dense
 * buffer; softmax and the weighted sum of values stay in the rotated space and
 * one inverse rotation per head maps the output back (Sec. 4.2, Lemma 2).
 *
 * Keys and values may keep different numbers of components per sequence
 * (k_active for the keys, k_value for the values), as in the key/value
 * retention ablation of Appendix A.5 (Table 2).  Algorithm 1 itself uses one
 * k_active for both; passing k_value_host = NULL selects that.
 *
 * Conventions for every entry point:
 *  - Pointers are DEVICE pointers unless the name ends in _host.
 *  - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *    Work is enqueued on it and the call returns without waiting, except
 *    swan_calibrate_rotation, which waits for its result.
 *  - The library never allocates memory.  The caller owns every buffer and
 *    sizes it with the *_bytes queries below.  The one resource it keeps: for
 *    a batch whose sequences use different k_pad, swan_decode_attention runs
 *    those attention launches side by side on up to three HIP streams of its
 *    own per calling thread and device (default priority, created on that
 *    thread's first such call with their events, kept until the process
 *    ends), forked from and joined back into `stream` with events, so the
 *    call orders with `stream` like any other and threads never share them.
 *    Calls are made with the stream's device current; otherwise the launches
 *    run one after another on `stream`.  It also holds, per GPU, the fixed
 *    scratch array of swan_decode_attention_noalloc (a device global, not an
 *    allocation).
 *  - The decode split plan and launch grouping follow fixed rules, which
 *    swan_set_decode_tuning can change for the calling thread; no environment
 *    variable is read.
 *  - All arguments are validated on the host before anything is enqueued, so
 *    a non-OK status means nothing was written.  Errors never abort, throw or
 *    exit; swan_last_error() returns a message for the calling thread.
 *  - Faults inside enqueued kernels surface at the caller's next
 *    synchronisation, as for any HIP work.
 *  - The GPU path supports head_dim == 128 only; batch <= SWAN_MAX_BATCH.
 */
#ifndef SWAN_H
#define SWAN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum swan_status {
  SWAN_OK = 0,
  SWAN_ERR_INVALID_ARG = 1,    /* null pointer, bad size, out-of-range k, ... */
  SWAN_ERR_UNSUPPORTED = 2,    /* valid request outside what this build supports */
  SWAN_ERR_CAPACITY = 3,       /* sparse_capacity would be exceeded */
  SWAN_ERR_WORKSPACE = 4,      /* workspace missing or smaller than the query says */
  SWAN_ERR_HIP = 5,            /* a HIP runtime call failed (message has details) */
  SWAN_ERR_NO_CONVERGENCE = 6  /* the eigensolver hit its sweep limit */
} swan_status;

typedef enum swan_dtype {
  SWAN_F32 = 0,      /* float32 storage */
  SWAN_F16 = 1,      /* IEEE binary16 storage */
  SWAN_F16_E4M3 = 2  /* binary16 keys, values, queries, outputs and dense buffer; the
                        sparse values stored as OCP FP8 E4M3 (one byte, no scale): the
                        kept binary16 values rounded to the nearest E4M3 value, ties to
                        the even code, magnitudes above 448 to 448 (Sec. 4.3 and
                        Sec. 5.1 name 8-bit values; the format is this library's
                        reading).  The top-k still ranks the binary16 values. */
} swan_dtype;

#define SWAN_MAX_BATCH 64
#define SWAN_HEAD_DIM 128
#define SWAN_PAGE_TOKENS 64

/*
 * The hybrid KV cache of Algorithm 1 for one attention layer: per (sequence,
 * KV head) a dense FIFO buffer of the last b rotated tokens (the "ring") and a
 * sparse cache of pruned tokens (the "pages").  The caller allocates the four
 * arrays (sizes from swan_cache_bytes) and keeps, on the host, the number of
 * tokens cached per sequence and each sequence's k_active.
 *
 * Ring layout: [batch][n_kv_heads][buffer_tokens][head_dim] of the storage
 * type; the token at position pos (0-based, pos >= L - b) is in slot pos % b.
 *
 * Page layout.  Sparse token p of sequence s and KV head h (p < L - b) is in
 * page p / 64, slot t = p % 64.  With VB the bytes of a sparse value (4 for
 * SWAN_F32, 2 for SWAN_F16, 1 for SWAN_F16_E4M3), CB the value chunk bytes (16,
 * 16, 8), GV = CB / VB values per chunk and k_pad = k rounded up to a multiple
 * of 8, a page is
 *     values : k_pad / GV chunks, each [64 slots][CB bytes]
 *     indices: k_pad / 8  chunks, each [64 slots][8 bytes] (uint8)
 * so entry e of slot t has its value at byte (e / GV) * 64 * CB + t * CB +
 * (e % GV) * VB and its index at byte 64 * k_pad * VB + (e / 8) * 512 + t * 8 +
 * (e % 8).  A page is 64 * k_pad * (VB + 1) bytes.  Entries 0..k-1 are the
 * kept components in ascending index order (after swan_change_k raised k, the
 * components kept at pruning in ascending order, then the raise's zero-valued
 * pairs in ascending order); entries k..k_pad-1 are padding with value +0 at the
 * lowest dims that were not kept, so the k_pad indices of a token are distinct
 * (the decode kernel relies on it).  The keys' pages live in k_pages and use the sequence's k_active; the
 * values' pages live in v_pages and use its k_value (k_active when
 * k_value_host is NULL).  In each array, sequence s owns
 * n_kv_heads * ceil(sparse_capacity / 64) pages of that role's k, stored after
 * those of sequences 0..s-1; within it, head h owns the consecutive pages
 * [h * ceil(sparse_capacity / 64), ...).
 */
typedef struct swan_cache {
  int32_t batch;            /* sequences, 1..SWAN_MAX_BATCH */
  int32_t n_q_heads;        /* query heads; a multiple of n_kv_heads (GQA group G = n_q / n_kv) */
  int32_t n_kv_heads;       /* KV heads */
  int32_t head_dim;         /* d_h; must be 128 */
  int32_t buffer_tokens;    /* b >= 0, dense buffer size of Algorithm 1 */
  int32_t sparse_capacity;  /* max pruned tokens per (sequence, KV head) */
  int32_t dtype;            /* swan_dtype of keys, values, queries and outputs */
  int32_t reserved;         /* must be 0 */
  void* k_pages;            /* sparse keys (see page layout) */
  void* v_pages;            /* sparse values */
  void* k_ring;             /* dense rotated keys, [B][H_kv][b][d] */
  void* v_ring;             /* dense rotated values, same layout */
} swan_cache;

/* Message describing the last non-OK status returned on this thread. */
const char* swan_last_error(void);

/* Library ABI version (major * 100 + minor). */
int32_t swan_version(void);

/*
 * Bytes of one page for storage type `dtype` and `k_active`: the Sec. 5.1 space
 * model of 64 vectors (k values + k uint8 indices each, k padded to 8; the
 * 2-byte row offsets are implicit because k is fixed per sequence).
 */
swan_status swan_page_bytes(int32_t dtype, int32_t k_active, size_t* bytes);

/*
 * Sizes of the cache arrays: *k_page_bytes for k_pages, *v_page_bytes for
 * v_pages and *ring_bytes for each of k_ring / v_ring.  k_active_host[batch] is
 * each sequence's k for its keys (1..head_dim); k_value_host[batch], if not
 * NULL, its k for its values (1..head_dim; NULL: the same as the keys).  They
 * fix the page layout, so every later call on this cache must pass the same
 * values.  The array pointers in `c` are ignored.
 */
swan_status swan_cache_bytes(const swan_cache* c, const int32_t* k_active_host,
                             const int32_t* k_value_host, size_t* k_page_bytes,
                             size_t* v_page_bytes, size_t* ring_bytes);

/* Device workspace needed by swan_calibrate_rotation for head dimension d. */
swan_status swan_calibrate_workspace_bytes(int32_t d, size_t* bytes);

/*
 * Offline calibration, Sec. 4.1.2: P = the right singular matrix of the joint
 * matrix S (`rows`, n_rows x d, row-major float32, device), i.e. the
 * eigenvectors of S^T S, with columns ordered by descending singular value and
 * each column's largest-magnitude entry made positive (ties: lowest row).  No
 * mean is removed.  Writes P_out[i * d + j] = component i of basis vector j
 * (float32, device; x_hat = x . P) and, if sigma_out is not NULL, the singular
 * values sigma_out[j] (float32, device).  The caller forms S, e.g. keys for
 * P_QK and values for P_VO.  Needs d == 128, n_rows >= 1.  Runs on `stream` and
 * waits for it, because convergence is reported through the status
 * (SWAN_ERR_NO_CONVERGENCE).
 */
swan_status swan_calibrate_rotation(const float* rows, int64_t n_rows, int32_t d,
                                    float* P_out, float* sigma_out, void* workspace,
                                    size_t workspace_bytes, void* stream);

/*
 * Algorithm 1, compress part, for up to n_new tokens per sequence.
 *  seq_len_host[batch]  tokens already cached per sequence (before this call);
 *  k_active_host[batch] k of each sequence's keys (1..head_dim), and
 *  k_value_host[batch]  of its values (NULL: as the keys), as in swan_cache_bytes;
 *  k_new, v_new         [batch][n_kv_heads][n_new][head_dim] storage type, the
 *                       un-rotated (post-RoPE) keys and values;
 *  n_new_host[batch]    tokens to append per sequence, 0..n_new (the first ones
 *                       of its rows); NULL means n_new for every sequence;
 *  P_qk, P_vo           [n_kv_heads][head_dim][head_dim] float32 rotations.
 *                       P_vo may be NULL: the values are then already in the
 *                       rotated basis (a model with P_VO absorbed into W_V,
 *                       Sec. 4.2) and are stored as given.
 * Each new token is rotated (k_hat = k . P_qk, v_hat = v . P_vo, accumulated in
 * float64 and rounded once to the storage type) and appended to the buffer;
 * every token that leaves the buffer (position < L_new - b) is pruned to the
 * top-k magnitudes of its stored values (ties: lower index), separately for
 * keys (k_active) and values (k_value), and packed into its page slot.  With b == 0 every token is
 * pruned on arrival.  Appending n tokens at once gives the same bytes as n
 * single appends.  The caller then adds each sequence's count to its seq_len.
 * Errors: SWAN_ERR_CAPACITY if L_new - b > sparse_capacity for a sequence.
 */
swan_status swan_compress_append(const swan_cache* c, const int32_t* seq_len_host,
                                 const int32_t* k_active_host, const int32_t* k_value_host,
                                 const void* k_new, const void* v_new, int32_t n_new,
                                 const int32_t* n_new_host, const float* P_qk,
                                 const float* P_vo, void* stream);

/* Device workspace needed by swan_decode_attention for these lengths and k. */
swan_status swan_decode_workspace_bytes(const swan_cache* c, const int32_t* seq_len_host,
                                        const int32_t* k_active_host,
                                        const int32_t* k_value_host, size_t* bytes);

/*
 * Algorithm 1, attention part, one decode query per (sequence, query head):
 *  seq_len_host[batch]  L >= 1, tokens in the cache with the current one
 *                       already appended by swan_compress_append;
 *  k_active_host, k_value_host  as in swan_compress_append;
 *  q                    [batch][n_q_heads][head_dim] storage type (post-RoPE);
 *  scale                softmax scale; <= 0 means 1 / sqrt(head_dim);
 *  out                  [batch][n_q_heads][head_dim] storage type.
 * Computes q_hat = q . P_qk[g] (g = h_q / G), scores q_hat . k over the sparse
 * pairs and the dense buffer, softmax, o_hat = sum_t p_t v_hat_t, and returns
 * out = o_hat . P_vo[g]^T (the inverse rotation of Sec. 4.2), rounded once to
 * the storage type.  With P_vo NULL it returns o_hat itself, for a model that
 * absorbs P_VO^T into W_O (Sec. 4.2).  Scores, probabilities and accumulators
 * are float32.
 */
swan_status swan_decode_attention(const swan_cache* c, const int32_t* seq_len_host,
                                  const int32_t* k_active_host, const int32_t* k_value_host,
                                  const void* q, const float* P_qk, const float* P_vo,
                                  float scale, void* out, void* workspace,
                                  size_t workspace_bytes, void* stream);

/*
 * swan_decode_attention without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  Arguments, results and errors are those
 * of swan_decode_attention.  The workspace (rotated queries and split
 * partials) is instead a device array inside this library: SWAN_NOALLOC_SCRATCH_BYTES
 * (16 MiB) per GPU, set up on the first call on a device (with the stream's
 * device current) and held until the process ends.  A batch whose
 * swan_decode_workspace_bytes exceeds it is rejected with SWAN_ERR_WORKSPACE
 * before anything is enqueued.  The call allocates nothing: no hipMalloc, no
 * stream or event creation (all launches go to `stream`, also for a batch that
 * mixes k_pad).  Every call on one GPU shares that GPU's array, so calls that
 * can overlap on one GPU (other streams, other threads) race and must be
 * ordered by the caller; calls on one stream are ordered by it.
 * `stream` must belong to the current device (SWAN_ERR_INVALID_ARG otherwise).
 */
#define SWAN_NOALLOC_SCRATCH_BYTES ((size_t)16 << 20)
swan_status swan_decode_attention_noalloc(const swan_cache* c, const int32_t* seq_len_host,
                                          const int32_t* k_active_host,
                                          const int32_t* k_value_host, const void* q,
                                          const float* P_qk, const float* P_vo, float scale,
                                          void* out, void* stream);

/*
 * One decode step of Algorithm 1 (its compress part for one new token per
 * sequence, then its attention part): the same as swan_compress_append with
 * n_new = 1 (n_new_host NULL) followed by swan_decode_attention with lengths
 * seq_len_host[b] + 1, on `stream`, with the same results bit for bit, in one
 * launch fewer: for n_q_heads / n_kv_heads <= 8 the query rotation runs inside
 * the append launch, where the workgroup that rotates a kv head's new key reads
 * the same rows of P_qk (one launch less on a latency-bound step).
 *  seq_len_host[batch]  tokens cached per sequence BEFORE the step (>= 0);
 *  k_new, v_new         [batch][n_kv_heads][1][head_dim] storage type (un-rotated);
 *  q, out               [batch][n_q_heads][head_dim] storage type;
 *  workspace            at least swan_decode_workspace_bytes for the lengths after
 *                       the step (seq_len_host[b] + 1), 256-byte aligned;
 *  k_active_host, k_value_host, P_qk, P_vo, scale  as in the two calls.
 * Every argument of both parts is checked before anything is enqueued, so an
 * error leaves the cache as it was.  The caller then adds 1 to each seq_len.
 * Errors: those of swan_compress_append and swan_decode_attention.
 */
swan_status swan_decode_step(const swan_cache* c, const int32_t* seq_len_host,
                             const int32_t* k_active_host, const int32_t* k_value_host,
                             const void* k_new, const void* v_new, const void* q,
                             const float* P_qk, const float* P_vo, float scale, void* out,
                             void* workspace, size_t workspace_bytes, void* stream);

/*
 * Rotary position embedding, for the query and key rows of a layer before the
 * cache rotates them (the paper rotates post-RoPE queries and keys, Sec. 4.2).
 *  x, y          [batch][n_heads][n][head_dim] rows of the storage type of
 *                `dtype` (binary16 for SWAN_F16 and SWAN_F16_E4M3), device; y may
 *                be x (in place);
 *  pos0_host[b]  position of sequence b's first row (row i sits at pos0 + i);
 *  base          the RoPE base (10000 for Llama-2, 500000 for Llama-3), > 1.
 * Dims j and j + head_dim/2 rotate by the angle pos * base^(-2j/head_dim), in
 * float64, rounded once to the storage type.  Needs head_dim == 128.
 */
swan_status swan_rope(const void* x, void* y, int32_t dtype, int32_t batch, int32_t n_heads,
                      int32_t n, int32_t head_dim, const int32_t* pos0_host, double base,
                      void* stream);

/*
 * Run-time change of k for running sequences (Algorithm 1 takes k_active as an
 * input at every step; Sec. 1 and Sec. 3 present k as tunable at inference
 * time).  Lays the sparse caches of `src` (laid out with k_active_src /
 * k_value_src) out again in `dst` (laid out with k_active_dst / k_value_dst),
 * per sequence and role:
 *  - k' < k: each stored token keeps the k' largest of its k stored values,
 *    ties to the lower index, in ascending index order.  For SWAN_F16 / SWAN_F32 values this is exactly
 *    the token's top-k' (the top-k' of a top-k set, under one tie rule), so the
 *    result equals pruning at k' from the start; for SWAN_F16_E4M3 it ranks the
 *    stored 8-bit values.
 *  - k' > k: each stored token keeps its k pairs (it was pruned with the k of
 *    its step) and slots k..k'-1 take value +0 at its lowest dims not kept.
 *  - k' == k: the pairs are copied.
 * Slots past k' are padding as always.  Tokens still in the dense buffer are not
 * touched: they are pruned with the new k when they leave it, so later calls on
 * the sequence pass k_active_dst / k_value_dst.
 *  seq_len_host[batch]  tokens cached per sequence (0 allowed);
 *  src, dst             descriptors with the same batch, heads, buffer_tokens and
 *                       dtype; dst's sparse_capacity may differ but must hold every
 *                       sequence's sparse tokens; dst must use src's ring arrays
 *                       (k_ring, v_ring) and page arrays that do not overlap src's,
 *                       sized with swan_cache_bytes for the new k.
 * Errors: SWAN_ERR_INVALID_ARG (mismatched descriptors, overlap, other rings,
 * k outside 1..head_dim), SWAN_ERR_CAPACITY.
 */
swan_status swan_change_k(const swan_cache* src, const int32_t* k_active_src,
                          const int32_t* k_value_src, const swan_cache* dst,
                          const int32_t* k_active_dst, const int32_t* k_value_dst,
                          const int32_t* seq_len_host, void* stream);

/*
 * Tuning of swan_decode_workspace_bytes, swan_decode_attention and
 * swan_decode_attention_noalloc on the calling thread (it holds until changed;
 * NULL restores the defaults).  None of it changes what is computed: the
 * softmax of Algorithm 1 runs over all cached tokens whatever the token axis is
 * cut into, and only the order of floating-point additions differs.  The
 * workspace size depends on the plan, so query it under the same tuning.
 * Every field: 0 selects the default.
 *  target_waves       sparse attention waves the split planner aims for over
 *                     the batch (default 2048, two per wave slot of the GPU;
 *                     twice that for a batch of several k_pad on the
 *                     one-query-head-per-wave path with fp16 storage, which
 *                     takes one launch with each sequence's waves specialised
 *                     on its own k_pad); each sequence's token splits follow
 *                     its share of the bytes, every split keeps at least one
 *                     page;
 *  short_split_pages  a short sequence (whose shrinking splits would be at most
 *                     half as many as its share asks for) is cut into equal
 *                     splits of this many pages (default 3); -1: shrinking
 *                     splits for every sequence;
 *  merge_pct          for a batch mixing k_pad on the other paths (several
 *                     query heads per wave, or fp32 storage): from the largest
 *                     k_pad down, a group of sequences joins the launch before
 *                     it when its k_pad is at least this percentage of that
 *                     launch's (default 66); -1: one launch per k_pad;
 *  side_streams       library streams (per thread and device) for those
 *                     launches, 1..3 (default 3); -1: all on the caller's stream.
 * Errors: SWAN_ERR_INVALID_ARG for a value outside these ranges (the thread's
 * tuning is then unchanged).
 */
typedef struct swan_decode_tuning {
  int32_t target_waves;       /* 0 or 1..1048576 */
  int32_t short_split_pages;  /* 0, -1 or 1..4096 */
  int32_t merge_pct;          /* 0, -1 or 1..100 */
  int32_t side_streams;       /* 0, -1 or 1..3 */
} swan_decode_tuning;
swan_status swan_set_decode_tuning(const swan_decode_tuning* tuning);

/*
 * Profiling hook.  While both are non-NULL, swan_decode_attention,
 * swan_decode_attention_noalloc and swan_decode_step on this thread record
 * start_event (a hipEvent_t) on their stream right before their sparse/buffer
 * attention launches and stop_event right after them, so that
 * hipEventElapsedTime gives the duration of those kernels alone.  Events made
 * with hipEventReleaseToDevice cost the stream the least (no system-scope
 * release at each record).  NULL, NULL (the default) disables it.  The events
 * stay owned by the caller.
 */
swan_status swan_set_profile_events(void* start_event, void* stop_event);

#ifdef __cplusplus
}
#endif

#endif /* SWAN_H */
